// Local objective of Eq. (3)-(5) on the frozen readout of Eq. (2).
//
// The head GEMM writes the logits of a row block: rows of z (readout of
// h_out) interleaved with rows of z' (readout of h_in, the stop-gradient
// consistency target) when alpha < 1; fp32, or fp16 in the bf16 path, where
// the GEMM's epilogue also leaves the fp32 statistics of pass 1 and the
// fp32 label logit z_y, and the fp16 values are z minus the fp32 maximum of
// their 64-column block.  One workgroup per token row then
//   pass 1: online max / sum-exp of z and z', plus the KL statistic
//           E = sum_v p_v (z_v - z'_v)   (reverse)   or
//           F = sum_v q_v (z'_v - z_v)   (forward),
//   pass 2: dL/dz_v = (1/|Omega|) [alpha (p_v - [v = y]) + (1 - alpha) g_v]
//           with g = p (z - z' - E) (reverse, the softmax Jacobian applied to
//           log p - log q) or g = p - q (forward),
// and writes the row's loss alpha CE + (1 - alpha) KL (0 outside Omega),
// CE = lse - z_y, KL_rev = E - lse + lse', KL_fwd = F - lse' + lse.
#include "common.h"

namespace zl {

constexpr int OT = 256;

__device__ inline bool label_ok(int y, int V) { return y >= 0 && y < V; }

__global__ void count_omega_kernel(const int32_t* __restrict__ labels, int T, int V,
                                   float* __restrict__ out) {
  __shared__ int red[OT / 64];
  int c = 0;
  for (int i = threadIdx.x; i < T; i += OT) c += label_ok(labels[i], V) ? 1 : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int i = 0; i < OT / 64; ++i) t += red[i];
    out[0] = (float)t;
  }
}

hipError_t launch_count_omega(const int32_t* labels, int T, int V, float* n_omega,
                              hipStream_t s) {
  hipLaunchKernelGGL(count_omega_kernel, dim3(1), dim3(OT), 0, s, labels, T, V, n_omega);
  return hipGetLastError();
}

struct Soft {  // running (max, sum exp(x - max), sum exp(x - max) * w)
  float m, s, e;
};

__device__ inline Soft soft_merge(Soft a, Soft b) {
  const float m = fmaxf(a.m, b.m);
  if (m == -INFINITY) return a;
  const float fa = __expf(a.m - m), fb = __expf(b.m - m);
  return {m, a.s * fa + b.s * fb, a.e * fa + b.e * fb};
}

__device__ inline Soft soft_add(Soft a, float x, float w) {
  if (x > a.m) {
    const float f = __expf(a.m - x);
    return {x, a.s * f + 1.f, a.e * f + w};
  }
  const float p = __expf(x - a.m);
  return {a.m, a.s + p, a.e + p * w};
}

// Four values at once: one rescale to their maximum, then four exponentials.
__device__ inline Soft soft_add4(Soft a, const float (&x)[4], const float (&w)[4]) {
  const float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
  if (mx > a.m) {
    const float f = __expf(a.m - mx);
    a = {mx, a.s * f, a.e * f};
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float p = __expf(x[k] - a.m);
    a.s += p;
    a.e += p * w[k];
  }
  return a;
}

__device__ inline Soft block_soft(Soft v, Soft* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    Soft t = {__shfl_xor(v.m, o, 64), __shfl_xor(v.s, o, 64), __shfl_xor(v.e, o, 64)};
    v = soft_merge(v, t);
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  Soft r = red[0];
  for (int i = 1; i < OT / 64; ++i) r = soft_merge(r, red[i]);
  return r;
}

// Rows are 16-byte aligned (ldz and lddz multiples of 8); 4 columns per
// thread and step, the last partial group of a row element by element.
__device__ inline void st_dz4(const ObjDesc& o, int64_t i, const float (&g)[4]) {
  if (o.dz_dtype == BF16) {
    uint2 u;
    u.x = (uint32_t)f32_to_bf16(g[0]) | ((uint32_t)f32_to_bf16(g[1]) << 16);
    u.y = (uint32_t)f32_to_bf16(g[2]) | ((uint32_t)f32_to_bf16(g[3]) << 16);
    *reinterpret_cast<uint2*>((bf16_t*)o.dz + i) = u;
  } else {
    *reinterpret_cast<float4*>((float*)o.dz + i) = make_float4(g[0], g[1], g[2], g[3]);
  }
}

// Logits as cached: fp32, or fp16 (ZT = uint16_t) in the bf16 path, where
// the cache holds z minus the maximum of its 64-column block and `st`
// points at the row's block statistics (the maximum in .x).
__device__ inline float ldz1(const float* p, int64_t v, const float4*) { return p[v]; }
__device__ inline float ldz1(const uint16_t* p, int64_t v, const float4* st) {
  return f16_to_f32(p[v]) + st[v >> 6].x;
}
__device__ inline void ldz4(const float* p, int64_t v, float (&x)[4], const float4*) {
  const float4 a = *reinterpret_cast<const float4*>(p + v);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
}
__device__ inline void ldz4(const uint16_t* p, int64_t v, float (&x)[4], const float4* st) {
  const uint2 a = *reinterpret_cast<const uint2*>(p + v);
  const float mx = st[v >> 6].x;  // four columns from v (v % 4 == 0) share a block
  x[0] = f16_to_f32((uint16_t)(a.x & 0xffff)) + mx;
  x[1] = f16_to_f32((uint16_t)(a.x >> 16)) + mx;
  x[2] = f16_to_f32((uint16_t)(a.y & 0xffff)) + mx;
  x[3] = f16_to_f32((uint16_t)(a.y >> 16)) + mx;
}

template <typename ZT>
__global__ void __launch_bounds__(OT) objective_rows_kernel(ObjDesc o) {
  __shared__ Soft red[OT / 64];
  const int i = blockIdx.x;
  const ZT* z = static_cast<const ZT*>(o.zc) + (int64_t)i * o.stacked * o.ldz;
  const ZT* zp = o.stacked == 2 ? z + o.ldz : nullptr;
  const int y = o.labels[i];
  const bool in_omega = label_ok(y, o.V);
  const float nomega = o.n_omega[0];
  const float inv = nomega > 0.f ? 1.f / nomega : 0.f;
  const bool rev = o.consis == 0;
  const int64_t orow = (int64_t)i * o.lddz;
  const int V4 = o.V & ~3;  // columns handled 4 at a time

  if (!in_omega) {
    const float zero[4] = {0.f, 0.f, 0.f, 0.f};
    for (int v = threadIdx.x * 4; v < o.Vpad; v += OT * 4) st_dz4(o, orow + v, zero);
    if (threadIdx.x == 0) o.row_loss[i] = 0.f;
    return;
  }

  // the row's 64-column block statistics (bf16 path; null in the fp32 path)
  const float4* stz = o.stats ? o.stats + (int64_t)i * o.stacked * o.ldst : nullptr;
  const float4* stq = o.stats && zp ? stz + o.ldst : nullptr;
  Soft sp = {-INFINITY, 0.f, 0.f}, sq = {-INFINITY, 0.f, 0.f};
  if (o.stats) {  // partials of 64-column blocks from the logit GEMM's epilogue
    const float4* st = stz;
    for (int cb = threadIdx.x; cb < o.nst; cb += OT) {
      const float4 p = st[cb];
      sp = soft_merge(sp, {p.x, p.y, p.z});
      if (zp) {
        const float4 q = st[o.ldst + cb];
        sq = soft_merge(sq, {q.x, q.y, q.z});
      }
    }
  }
  for (int v = o.stats ? V4 : threadIdx.x * 4; v < V4; v += OT * 4) {
    float a[4], b[4] = {0.f, 0.f, 0.f, 0.f};
    ldz4(z, v, a, stz);
    if (zp) ldz4(zp, v, b, stq);
    const float ab[4] = {a[0] - b[0], a[1] - b[1], a[2] - b[2], a[3] - b[3]};
    sp = soft_add4(sp, a, ab);  // e accumulates sum p (z - z') unnormalised
    if (zp) {
      const float ba[4] = {-ab[0], -ab[1], -ab[2], -ab[3]};
      sq = soft_add4(sq, b, ba);
    }
  }
  for (int v = V4 + threadIdx.x; v < (o.stats ? 0 : o.V); v += OT) {
    const float a = ldz1(z, v, stz);
    const float b = zp ? ldz1(zp, v, stq) : 0.f;
    sp = soft_add(sp, a, a - b);
    if (zp) sq = soft_add(sq, b, b - a);
  }
  sp = block_soft(sp, red);
  const float lse = sp.m + __logf(sp.s);
  float lse2 = 0.f, E = 0.f, F = 0.f;
  E = sp.e / sp.s;
  if (zp) {
    sq = block_soft(sq, red);
    lse2 = sq.m + __logf(sq.s);
    F = sq.e / sq.s;
  }
  const float zy = o.zy ? o.zy[i] : ldz1(z, y, stz);
  const float ce = lse - zy;
  float kl = 0.f;
  if (zp) kl = rev ? (E - lse + lse2) : (F - lse2 + lse);
  const float a = o.alpha;
  if (threadIdx.x == 0) o.row_loss[i] = a * ce + (zp ? (1.f - a) * kl : 0.f);

  // dL/dz of one column
  auto grad = [&](int v, float zv, float zpv) {
    const float p = __expf(zv - lse);
    float g = a * (p - (v == y ? 1.f : 0.f));
    if (zp) {
      if (rev) g += (1.f - a) * p * (zv - zpv - E);
      else g += (1.f - a) * (p - __expf(zpv - lse2));
    }
    return g * inv;
  };
  for (int v = threadIdx.x * 4; v < o.Vpad; v += OT * 4) {
    float g[4] = {0.f, 0.f, 0.f, 0.f};
    if (v < V4) {
      float a4[4], b4[4] = {0.f, 0.f, 0.f, 0.f};
      ldz4(z, v, a4, stz);
      if (zp) ldz4(zp, v, b4, stq);
#pragma unroll
      for (int k = 0; k < 4; ++k) g[k] = grad(v + k, a4[k], b4[k]);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (v + k < o.V) g[k] = grad(v + k, ldz1(z, v + k, stz), zp ? ldz1(zp, v + k, stq) : 0.f);
    }
    st_dz4(o, orow + v, g);
  }
}

hipError_t launch_objective_rows(const ObjDesc& o, hipStream_t s) {
  if (o.rows <= 0) return hipSuccess;
  if (o.z_dtype == F16) {
    if (!o.stats) return hipErrorInvalidValue;  // fp16 logits come with the GEMM's statistics
    hipLaunchKernelGGL(objective_rows_kernel<uint16_t>, dim3(o.rows), dim3(OT), 0, s, o);
  } else {
    hipLaunchKernelGGL(objective_rows_kernel<float>, dim3(o.rows), dim3(OT), 0, s, o);
  }
  return hipGetLastError();
}

__global__ void loss_reduce_kernel(const float* __restrict__ row_loss, int T,
                                   const float* __restrict__ n_omega, float* __restrict__ loss) {
  __shared__ float red[OT / 64];
  float s = 0.f;
  for (int i = threadIdx.x; i < T; i += OT) s += row_loss[i];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int i = 0; i < OT / 64; ++i) t += red[i];
    const float n = n_omega[0];
    loss[0] = n > 0.f ? t / n : 0.f;
  }
}

hipError_t launch_loss_reduce(const float* row_loss, int T, const float* n_omega, float* loss,
                              hipStream_t s) {
  hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(OT), 0, s, row_loss, T, n_omega, loss);
  return hipGetLastError();
}

}  // namespace zl
