// Row-wise and elementwise kernels of the chunk map (Eq. (1)) and of the
// frozen head's norm (Eq. (2)): RMSNorm / LayerNorm forward and backward,
// rotary embedding, SwiGLU, casts, deterministic two-stage reductions.
// All HBM-bound: one pass over each operand, coalesced along the row.
#include "common.h"

namespace zl {

constexpr int RT = 256;            // threads per row block

__device__ inline float ldf(const void* p, int dt, size_t i) {
  return dt == BF16 ? bf16_to_f32(((const bf16_t*)p)[i]) : ((const float*)p)[i];
}
__device__ inline void stf(void* p, int dt, size_t i, float v) {
  if (dt == BF16) ((bf16_t*)p)[i] = f32_to_bf16(v);
  else ((float*)p)[i] = v;
}

// ----------------------------------------------------------- norm forward
// One wave per output row; float4 loads; the row is read three times (sum,
// centred sum of squares, output) and stays in L1/L2 between the passes.
// Output row r reads source row: xb ? (r even: xa[row0 + r/2], odd:
// xb[row0 + r/2]) : xa[row0 + r].
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <int CM>
__global__ void __launch_bounds__(RT)
norm_fwd_kernel(int layernorm, const float* __restrict__ xa, const float* __restrict__ xb,
                int64_t ldx, int row0, const float* __restrict__ w, const float* __restrict__ b,
                void* __restrict__ y, int64_t ldy, int ydt, float* __restrict__ mean,
                float* __restrict__ rstd, int rows, int d, float eps) {
  const int r = blockIdx.x * (RT / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const float* x;
  if (xb) x = ((r & 1) ? xb : xa) + (int64_t)(row0 + (r >> 1)) * ldx;
  else x = xa + (int64_t)(row0 + r) * ldx;
  // the row is read once into registers (lane owns columns 256 k + 4 lane)
  float4 xv[CM];
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < CM; ++k) {
    const int c = k * 256 + lane * 4;
    xv[k] = c < d ? *reinterpret_cast<const float4*>(x + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    s += (xv[k].x + xv[k].y) + (xv[k].z + xv[k].w);
  }
  const float mu = layernorm ? wave_sum(s) / d : 0.f;
  float q = 0.f;
#pragma unroll
  for (int k = 0; k < CM; ++k) {
    const int c = k * 256 + lane * 4;
    if (c >= d) continue;
    const float a0 = xv[k].x - mu, a1 = xv[k].y - mu, a2 = xv[k].z - mu, a3 = xv[k].w - mu;
    q += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
  }
  const float rs = rsqrtf(wave_sum(q) / d + eps);
  if (lane == 0) {
    rstd[r] = rs;
    if (layernorm && mean) mean[r] = mu;
  }
#pragma unroll
  for (int k = 0; k < CM; ++k) {
    const int c = k * 256 + lane * 4;
    if (c >= d) continue;
    const float4 v = xv[k];
    const float4 g = *reinterpret_cast<const float4*>(w + c);
    float o0 = (v.x - mu) * rs * g.x, o1 = (v.y - mu) * rs * g.y;
    float o2 = (v.z - mu) * rs * g.z, o3 = (v.w - mu) * rs * g.w;
    if (layernorm) {
      const float4 bb = *reinterpret_cast<const float4*>(b + c);
      o0 += bb.x; o1 += bb.y; o2 += bb.z; o3 += bb.w;
    }
    const int64_t o = (int64_t)r * ldy + c;
    if (ydt == BF16) {
      *reinterpret_cast<ushort4*>((bf16_t*)y + o) =
          make_ushort4(f32_to_bf16(o0), f32_to_bf16(o1), f32_to_bf16(o2), f32_to_bf16(o3));
    } else {
      *reinterpret_cast<float4*>((float*)y + o) = make_float4(o0, o1, o2, o3);
    }
  }
}

static hipError_t norm_fwd_go(int layernorm, const float* xa, const float* xb, int64_t ldx,
                              int row0, const float* w, const float* b, void* y, int64_t ldy,
                              int ydt, float* mean, float* rstd, int rows, int d, float eps,
                              hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d <= 0 || d % 4 || d > 8192) return hipErrorInvalidValue;
  const dim3 grid((rows + 3) / 4), blk(RT);
  const int cm = (d + 255) / 256;
#define ZL_NF(CM) hipLaunchKernelGGL(norm_fwd_kernel<CM>, grid, blk, 0, s, layernorm, xa, xb, ldx, \
                                     row0, w, b, y, ldy, ydt, mean, rstd, rows, d, eps)
  if (cm <= 1) ZL_NF(1);
  else if (cm <= 2) ZL_NF(2);
  else if (cm <= 4) ZL_NF(4);
  else if (cm <= 8) ZL_NF(8);
  else if (cm <= 16) ZL_NF(16);
  else ZL_NF(32);
#undef ZL_NF
  return hipGetLastError();
}

hipError_t launch_norm_fwd(bool layernorm, const float* x, int64_t ldx, const float* w,
                           const float* b, void* y, int64_t ldy, int ydtype, float* mean,
                           float* rstd, int T, int d, float eps, hipStream_t s) {
  return norm_fwd_go((int)layernorm, x, nullptr, ldx, 0, w, b, y, ldy, ydtype, mean, rstd, T, d,
                     eps, s);
}

hipError_t launch_head_norm(bool layernorm, const float* xa, const float* xb, int64_t ldx,
                            int row0, int rows, const float* w, const float* b, void* y,
                            int ydtype, float* mean, float* rstd, int d, float eps,
                            hipStream_t s) {
  const int out_rows = xb ? 2 * rows : rows;
  return norm_fwd_go((int)layernorm, xa, xb, ldx, row0, w, b, y, (int64_t)d, ydtype, mean, rstd,
                     out_rows, d, eps, s);
}

// ---------------------------------------------------------- norm backward
// One 256-thread block per run of rows; thread t owns columns 4 (256 k + t)
// .. +3 (CM float4 groups), so a row is read once: dy and x stay in
// registers between the row reduction and dx.  Per row:
// g = dy * w, xhat = (x - mean) * rstd,
//   rms: dx = rstd * (g - xhat * mean(g * xhat))
//   ln:  dx = rstd * (g - mean(g) - xhat * mean(g * xhat))
// The row sums meet across the 4 waves in LDS (double-buffered, one
// barrier per row).  The weight-gradient partials sum(dy * xhat) (and
// sum(dy)) of the block's rows stay in registers and are written as one
// row of part_w / part_b per block: deterministic, no atomics.
int norm_bwd_blocks(int T) {
  int blocks = T / 16;  // about 16 rows per block
  if (blocks < 256) blocks = T < 256 ? T : 256;
  if (blocks > 2048) blocks = 2048;
  return blocks > 0 ? blocks : 1;  // number of partial rows
}

template <int CM, bool LN>
__global__ void __launch_bounds__(RT)
norm_bwd_kernel(const float* __restrict__ dy, int64_t lddy, const float* __restrict__ x,
                const float* __restrict__ w, const float* __restrict__ mean,
                const float* __restrict__ rstd, int rstride, const float* dres, float* dx,
                void* dx_act, int adt, float* __restrict__ part_w, float* __restrict__ part_b,
                int T, int d, int rpb, int nblk, int row_out0) {
  __shared__ float red[2][2][RT / 64];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const bool want_part = part_w != nullptr;
  float4 wv[CM], aw[CM], ab[CM];
#pragma unroll
  for (int k = 0; k < CM; ++k) {
    const int c = (k * RT + tid) * 4;
    wv[k] = c < d ? *reinterpret_cast<const float4*>(w + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    aw[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    ab[k] = aw[k];
  }
  const int r0 = blockIdx.x * rpb, r1 = min(T, r0 + rpb);
  int par = 0;
  for (int r = (blockIdx.x < nblk ? r0 : T); r < r1; ++r) {
    const float rs = rstd[(int64_t)r * rstride];
    const float mu = LN ? mean[(int64_t)r * rstride] : 0.f;
    const int ro = row_out0 + r;
    const float* dyr = dy + (int64_t)r * lddy;
    const float* xr = x + (int64_t)ro * d;
    float4 av[CM], hv[CM];
    float sg = 0.f, sgx = 0.f;
#pragma unroll
    for (int k = 0; k < CM; ++k) {
      const int c = (k * RT + tid) * 4;
      if (c >= d) { av[k] = make_float4(0.f, 0.f, 0.f, 0.f); hv[k] = av[k]; continue; }
      const float4 a = *reinterpret_cast<const float4*>(dyr + c);
      const float4 v = *reinterpret_cast<const float4*>(xr + c);
      const float4 g = wv[k];
      const float4 h = make_float4((v.x - mu) * rs, (v.y - mu) * rs, (v.z - mu) * rs, (v.w - mu) * rs);
      av[k] = a;
      hv[k] = h;
      const float g0 = a.x * g.x, g1 = a.y * g.y, g2 = a.z * g.z, g3 = a.w * g.w;
      sg += (g0 + g1) + (g2 + g3);
      sgx += (g0 * h.x + g1 * h.y) + (g2 * h.z + g3 * h.w);
      if (want_part) {
        aw[k].x += a.x * h.x; aw[k].y += a.y * h.y; aw[k].z += a.z * h.z; aw[k].w += a.w * h.w;
        if (LN) { ab[k].x += a.x; ab[k].y += a.y; ab[k].z += a.z; ab[k].w += a.w; }
      }
    }
    if (!dx) continue;
    sg = wave_sum(sg);
    sgx = wave_sum(sgx);
    if (lane == 0) {
      red[par][0][wave] = sg;
      red[par][1][wave] = sgx;
    }
    __syncthreads();
    float tg = 0.f, tgx = 0.f;
#pragma unroll
    for (int i = 0; i < RT / 64; ++i) {
      tg += red[par][0][i];
      tgx += red[par][1][i];
    }
    par ^= 1;
    const float mg = LN ? tg / d : 0.f;
    const float mgx = tgx / d;
#pragma unroll
    for (int k = 0; k < CM; ++k) {
      const int c = (k * RT + tid) * 4;
      if (c >= d) continue;
      const float4 a = av[k], h = hv[k], g = wv[k];
      float o[4] = {rs * (a.x * g.x - mg - h.x * mgx), rs * (a.y * g.y - mg - h.y * mgx),
                    rs * (a.z * g.z - mg - h.z * mgx), rs * (a.w * g.w - mg - h.w * mgx)};
      const int64_t off = (int64_t)ro * d + c;
      if (dres) {
        const float4 q = *reinterpret_cast<const float4*>(dres + off);
        o[0] += q.x; o[1] += q.y; o[2] += q.z; o[3] += q.w;
      }
      *reinterpret_cast<float4*>(dx + off) = make_float4(o[0], o[1], o[2], o[3]);
      if (dx_act) {
        if (adt == BF16)
          *reinterpret_cast<ushort4*>((bf16_t*)dx_act + off) =
              make_ushort4(f32_to_bf16(o[0]), f32_to_bf16(o[1]), f32_to_bf16(o[2]), f32_to_bf16(o[3]));
        else
          *reinterpret_cast<float4*>((float*)dx_act + off) = make_float4(o[0], o[1], o[2], o[3]);
      }
    }
  }
  if (want_part && blockIdx.x < nblk) {
#pragma unroll
    for (int k = 0; k < CM; ++k) {
      const int c = (k * RT + tid) * 4;
      if (c >= d) continue;
      *reinterpret_cast<float4*>(part_w + (int64_t)blockIdx.x * d + c) = aw[k];
      if (LN && part_b) *reinterpret_cast<float4*>(part_b + (int64_t)blockIdx.x * d + c) = ab[k];
    }
  }
}

template <int CM, bool LN>
static void norm_bwd_go(int blocks, hipStream_t s, const float* dy, int64_t lddy, const float* x,
                        const float* w, const float* mean, const float* rstd, int rstride,
                        const float* dres, float* dx, void* dx_act, int adt, float* part_w,
                        float* part_b, int T, int d, int rpb, int nb, int row_out0) {
  hipLaunchKernelGGL((norm_bwd_kernel<CM, LN>), dim3(blocks), dim3(RT), 0, s, dy, lddy, x, w,
                     mean, rstd, rstride, dres, dx, dx_act, adt, part_w, part_b, T, d, rpb, nb,
                     row_out0);
}

static hipError_t norm_bwd_launch(bool layernorm, const float* dy, int64_t lddy, const float* x,
                                  const float* w, const float* mean, const float* rstd,
                                  int rstride, const float* dres, float* dx, void* dx_act,
                                  int adt, float* part_w, float* part_b, int T, int d,
                                  int row_out0, int* nblk_out, hipStream_t s) {
  const int nb = norm_bwd_blocks(T);
  const int rpb = (T + nb - 1) / nb;
  if (nblk_out) *nblk_out = nb;
  if (d <= 0 || d % 4 || d > 8192) return hipErrorInvalidValue;
#define ZL_NB(CM, LN)                                                                       \
  norm_bwd_go<CM, LN>(nb, s, dy, lddy, x, w, mean, rstd, rstride, dres, dx, dx_act, adt,     \
                      part_w, part_b, T, d, rpb, nb, row_out0)
  const int cm = (d + 4 * RT - 1) / (4 * RT);
  if (layernorm) {
    if (cm <= 1) ZL_NB(1, true);
    else if (cm <= 2) ZL_NB(2, true);
    else if (cm <= 4) ZL_NB(4, true);
    else ZL_NB(8, true);
  } else {
    if (cm <= 1) ZL_NB(1, false);
    else if (cm <= 2) ZL_NB(2, false);
    else if (cm <= 4) ZL_NB(4, false);
    else ZL_NB(8, false);
  }
#undef ZL_NB
  return hipGetLastError();
}

hipError_t launch_norm_bwd(bool layernorm, const float* dy, const float* x, const float* w,
                           const float* mean, const float* rstd, const float* dres,
                           float* dx, void* dx_act, int act_dtype, float* part_w,
                           float* part_b, int T, int d, hipStream_t s, int* nblk_out) {
  return norm_bwd_launch(layernorm, dy, (int64_t)d, x, w, mean, rstd, 1, dres, dx, dx_act,
                         act_dtype, part_w, part_b, T, d, 0, nblk_out, s);
}

hipError_t launch_head_norm_bwd(bool layernorm, const float* dy, int64_t lddy, const float* x,
                                const float* w, const float* mean, const float* rstd,
                                int rstd_stride, float* dx, void* dx_act, int act_dtype,
                                int row0, int rows, int d, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  return norm_bwd_launch(layernorm, dy, lddy, x, w, mean, rstd, rstd_stride, nullptr, dx, dx_act,
                         act_dtype, nullptr, nullptr, rows, d, row0, nullptr, s);
}

// ------------------------------------------------------------- reductions
// out[j] = (accumulate ? out[j] : 0) + scale * sum_b part[b, j]; a block
// covers 64 columns with 4 row groups, each summing with 4 independent
// accumulators; the 4 group sums combine in a fixed order (deterministic).
// Rows b < nblk of part at part + b * rstride.  Block (x, y) sums rows
// [y gs, min(nblk, (y + 1) gs)) of columns 64 x .. 64 x + 63 in a fixed
// order; the last stage (final) writes out, an earlier one leaves its sum in
// place of the group's first row (read by the next stage), so the result is
// deterministic for a given nblk.
__global__ void __launch_bounds__(256) reduce_rows_kernel(float* part, int nblk, int64_t rstride,
                                                          int d, int gs, float* __restrict__ out,
                                                          float scale, int accumulate, int final) {
  __shared__ float red[4][64];
  const int j = blockIdx.x * 64 + (threadIdx.x & 63);
  const int grp = threadIdx.x >> 6;
  const int b0 = blockIdx.y * gs, b1 = min(nblk, b0 + gs);
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  if (j < d) {
    int b = b0 + grp;
    for (; b + 12 < b1; b += 16) {
      a0 += part[(int64_t)b * rstride + j];
      a1 += part[(int64_t)(b + 4) * rstride + j];
      a2 += part[(int64_t)(b + 8) * rstride + j];
      a3 += part[(int64_t)(b + 12) * rstride + j];
    }
    for (; b < b1; b += 4) a0 += part[(int64_t)b * rstride + j];
  }
  red[grp][threadIdx.x & 63] = (a0 + a1) + (a2 + a3);
  __syncthreads();
  if (grp == 0 && j < d) {
    const float t = ((red[0][threadIdx.x] + red[1][threadIdx.x]) + red[2][threadIdx.x]) + red[3][threadIdx.x];
    if (final) {
      const float v = scale * t;
      out[j] = accumulate ? out[j] + v : v;
    } else {
      part[(int64_t)b0 * rstride + j] = t;
    }
  }
}

hipError_t launch_reduce_rows(float* part, int nblk, int d, float* out, float scale,
                              int accumulate, hipStream_t s) {
  if (d <= 0) return hipSuccess;
  const int cb = (d + 63) / 64;
  int64_t stride = d;
  if (nblk > 256) {  // first stage: groups of 64 rows, many blocks
    constexpr int GS = 64;
    const int ng = (nblk + GS - 1) / GS;
    hipLaunchKernelGGL(reduce_rows_kernel, dim3(cb, ng), dim3(256), 0, s, part, nblk, stride, d,
                       GS, out, scale, accumulate, 0);
    nblk = ng;
    stride *= GS;
  }
  hipLaunchKernelGGL(reduce_rows_kernel, dim3(cb, 1), dim3(256), 0, s, part, nblk, stride, d, nblk,
                     out, scale, accumulate, 1);
  return hipGetLastError();
}

int colsum_blocks(int T) { return T < 256 ? (T > 0 ? T : 1) : 256; }

__global__ void colsum_kernel(const void* __restrict__ x, int64_t ldx, int dt, int T, int n,
                              int rpb, float* __restrict__ part) {
  const int r0 = blockIdx.y * rpb, r1 = min(T, r0 + rpb);
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < n; c += gridDim.x * blockDim.x) {
    float s0 = 0.f, s1 = 0.f;
    int r = r0;
    for (; r + 1 < r1; r += 2) {
      s0 += ldf(x, dt, (int64_t)r * ldx + c);
      s1 += ldf(x, dt, (int64_t)(r + 1) * ldx + c);
    }
    if (r < r1) s0 += ldf(x, dt, (int64_t)r * ldx + c);
    part[(int64_t)blockIdx.y * n + c] = s0 + s1;
  }
}

hipError_t launch_colsum_partial(const void* x, int64_t ldx, int dtype, int T, int n,
                                 float* part, int* nblk_out, hipStream_t s) {
  const int nblk = colsum_blocks(T);
  const int rpb = (T + nblk - 1) / nblk;
  *nblk_out = nblk;
  dim3 grid((n + 255) / 256, nblk);
  hipLaunchKernelGGL(colsum_kernel, grid, dim3(256), 0, s, x, ldx, dtype, T, n, rpb, part);
  return hipGetLastError();
}

// ------------------------------------------------------------ elementwise
__global__ void cast_kernel(const void* __restrict__ src, int sdt, void* __restrict__ dst,
                            int ddt, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    stf(dst, ddt, i, ldf(src, sdt, i));
}

hipError_t launch_cast(const void* src, int sdtype, void* dst, int ddtype, size_t n,
                       hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(cast_kernel, dim3((unsigned)blocks), dim3(256), 0, s, src, sdtype, dst,
                     ddtype, n);
  return hipGetLastError();
}

// mode 0: seq_lens (default S, clamped to [0, S]); mode 1: pos ids (default i % S)
__global__ void copy_i32_kernel(const int32_t* __restrict__ src, int32_t* __restrict__ dst, int n,
                                int mode, int S) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  if (mode == 0) {
    int v = src ? src[i] : S;
    dst[i] = v < 0 ? 0 : (v > S ? S : v);
  } else {
    dst[i] = src ? src[i] : (i % S);
  }
}

hipError_t launch_copy_i32(const int32_t* src, int32_t* dst, int n, int fill_default, int mode,
                           int S, hipStream_t s) {
  (void)fill_default;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n, mode,
                     S);
  return hipGetLastError();
}

// RoPE table: (cos, sin) of pos * theta^(-2j/hd), computed in double.
__global__ void rope_table_kernel(float2* table, int max_pos, int half, double theta) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= max_pos * half) return;
  const int p = i / half, j = i % half;
  const double inv = pow(theta, -(2.0 * j) / (2.0 * half));
  const double a = (double)p * inv;
  table[i] = make_float2((float)cos(a), (float)sin(a));
}

hipError_t launch_rope_table(float2* table, int max_pos, int half, double theta,
                             hipStream_t s) {
  const int n = max_pos * half;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_kernel, dim3((n + 255) / 256), dim3(256), 0, s, table, max_pos,
                     half, theta);
  return hipGetLastError();
}

// u'_j = u_j c - u_{j+h} s*sign ; u'_{j+h} = u_{j+h} c + u_j s*sign
__global__ void rope_kernel(void* __restrict__ qkv, int64_t ld, int dt,
                            const int32_t* __restrict__ pos, const float2* __restrict__ table,
                            int max_pos, int T, int nheads, int hd, float sign) {
  const int half = hd / 2;
  const int64_t n = (int64_t)T * nheads * half;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(i % half);
    const int64_t th = i / half;
    const int h = (int)(th % nheads);
    const int t = (int)(th / nheads);
    int p = pos[t];
    p = p < 0 ? 0 : (p >= max_pos ? max_pos - 1 : p);
    const float2 cs = table[(int64_t)p * half + j];
    const float sn = cs.y * sign;
    const int64_t o = (int64_t)t * ld + (int64_t)h * hd + j;
    const float a = ldf(qkv, dt, o), b = ldf(qkv, dt, o + half);
    stf(qkv, dt, o, a * cs.x - b * sn);
    stf(qkv, dt, o + half, b * cs.x + a * sn);
  }
}

hipError_t launch_rope(void* qkv, int64_t ld, int dtype, const int32_t* pos, const float2* table,
                       int max_pos, int T, int nheads_qk, int hd, int sign, hipStream_t s) {
  const int64_t n = (int64_t)T * nheads_qk * (hd / 2);
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(rope_kernel, dim3((unsigned)blocks), dim3(256), 0, s, qkv, ld, dtype, pos,
                     table, max_pos, T, nheads_qk, hd, (float)sign);
  return hipGetLastError();
}

// 8 consecutive elements per thread (16-byte bf16 / 2 x 16-byte fp32
// accesses); rows on the grid's y dimension (grid-stride beyond 65535).
__device__ inline void ld8(const void* p, int dt, int64_t i, float (&v)[8]) {
  if (dt == BF16) {
    const uint4 u = *reinterpret_cast<const uint4*>((const bf16_t*)p + i);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[2 * k] = bf16_to_f32((bf16_t)(w[k] & 0xffff));
      v[2 * k + 1] = bf16_to_f32((bf16_t)(w[k] >> 16));
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>((const float*)p + i);
    const float4 b = *reinterpret_cast<const float4*>((const float*)p + i + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}
__device__ inline void st8(void* p, int dt, int64_t i, const float (&v)[8]) {
  if (dt == BF16) {
    uint32_t w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      w[k] = (uint32_t)f32_to_bf16(v[2 * k]) | ((uint32_t)f32_to_bf16(v[2 * k + 1]) << 16);
    *reinterpret_cast<uint4*>((bf16_t*)p + i) = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
    *reinterpret_cast<float4*>((float*)p + i) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>((float*)p + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

__global__ void swiglu_fwd_kernel(const void* __restrict__ gu, int64_t ldgu,
                                  void* __restrict__ a, int64_t lda, int dt, int T, int ff) {
  const int j = (blockIdx.x * blockDim.x + threadIdx.x) * 8;
  if (j >= ff) return;
  for (int t = blockIdx.y; t < T; t += gridDim.y) {
    float g[8], u[8], o[8];
    ld8(gu, dt, (int64_t)t * ldgu + j, g);
    ld8(gu, dt, (int64_t)t * ldgu + ff + j, u);
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = g[k] / (1.f + __expf(-g[k])) * u[k];
    st8(a, dt, (int64_t)t * lda + j, o);
  }
}

hipError_t launch_swiglu_fwd(const void* gu, int64_t ldgu, void* a, int64_t lda, int dtype,
                             int T, int ff, hipStream_t s) {
  if (T <= 0 || ff <= 0) return hipSuccess;
  if (ff % 8 || ldgu % 8 || lda % 8) return hipErrorInvalidValue;
  const int bx = (ff / 8 + 255) / 256;
  const int by = T < 65535 ? T : 65535;
  hipLaunchKernelGGL(swiglu_fwd_kernel, dim3(bx, by), dim3(256), 0, s, gu, ldgu, a, lda, dtype,
                     T, ff);
  return hipGetLastError();
}

// Block-diagonal expansion of stacked low-rank factors (one thread per output
// element; the matrix is small: rows x nblk r).
__global__ void blockdiag_kernel(const void* __restrict__ src, void* __restrict__ dst, int dt,
                                 int rows, int r, int nblk, int b1, int b2) {
  const int64_t w = (int64_t)nblk * r, n = (int64_t)rows * w;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i / w;
    const int col = (int)(i % w);
    const int blk = row < b1 ? 0 : (row < b2 ? 1 : 2);
    stf(dst, dt, i, col / r == blk ? ldf(src, dt, row * r + col % r) : 0.f);
  }
}

hipError_t launch_blockdiag(const void* src, void* dst, int dtype, int rows, int r, int nblk,
                            int b1, int b2, hipStream_t s) {
  if (nblk < 1 || nblk > 3 || r < 1 || rows < 0 || b1 < 0 || b2 < b1 || b2 > rows)
    return hipErrorInvalidValue;
  const int64_t n = (int64_t)rows * nblk * r;
  if (n == 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(blockdiag_kernel, dim3((unsigned)blocks), dim3(256), 0, s, src, dst, dtype,
                     rows, r, nblk, b1, b2);
  return hipGetLastError();
}

}  // namespace zl
