// Causal GQA self-attention of the decoder layers inside f_k (Eq. (1)):
// scores q.k / sqrt(hd), key j visible to query i iff j <= i and
// j < seq_len[b]; q-head h reads kv-head h / (Hq / Hkv).  A query with no
// visible key outputs 0 and stores lse = -inf.
//
// This file holds the SIMT kernels: one thread per query (forward, dQ) or
// per key (dK, dV), K/V or Q/dO rows staged through LDS tiles, online
// softmax in fp32.  They serve the fp32 configuration and any head_dim the
// MFMA kernels (attention_mfma.hip) do not cover.
#include "common.h"

namespace zl {

constexpr int AT = 64;   // threads per block (one wave)
constexpr int KT = 32;   // rows per LDS tile

template <typename T>
__device__ inline float ld(const T* p, int64_t i) { return Elem<T>::load(p, i); }

template <typename T, int HD>
__global__ void __launch_bounds__(AT) attn_fwd_simt(AttnDesc a) {
  __shared__ float ks[KT][HD + 1], vs[KT][HD + 1];
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (a.Hq / a.Hkv);
  const int i = blockIdx.x * AT + threadIdx.x;
  const int L = a.seq_lens[b];
  const T* Q = (const T*)a.q;
  const T* K = (const T*)a.k;
  const T* Vv = (const T*)a.v;
  const int64_t rowb = (int64_t)b * a.S;
  float q[HD], o[HD];
  float m = -INFINITY, l = 0.f;
#pragma unroll
  for (int d = 0; d < HD; ++d) {
    q[d] = i < a.S ? ld(Q, (rowb + i) * a.ldq + (int64_t)h * HD + d) * a.scale : 0.f;
    o[d] = 0.f;
  }
  const int kend = min(min(blockIdx.x * AT + AT, a.S), L);
  for (int j0 = 0; j0 < kend; j0 += KT) {
    for (int e = threadIdx.x; e < KT * HD; e += AT) {
      const int r = e / HD, d = e % HD;
      const int j = j0 + r;
      float kv = 0.f, vv = 0.f;
      if (j < kend) {
        kv = ld(K, (rowb + j) * a.ldk + (int64_t)g * HD + d);
        vv = ld(Vv, (rowb + j) * a.ldv + (int64_t)g * HD + d);
      }
      ks[r][d] = kv;
      vs[r][d] = vv;
    }
    __syncthreads();
    for (int r = 0; r < KT; ++r) {
      const int j = j0 + r;
      if (j < kend && j <= i && i < a.S) {
        float s = 0.f;
#pragma unroll
        for (int d = 0; d < HD; ++d) s += q[d] * ks[r][d];
        const float mn = fmaxf(m, s);
        const float c = __expf(m - mn), p = __expf(s - mn);
        l = l * c + p;
#pragma unroll
        for (int d = 0; d < HD; ++d) o[d] = o[d] * c + p * vs[r][d];
        m = mn;
      }
    }
    __syncthreads();
  }
  if (i < a.S) {
    const float inv = l > 0.f ? 1.f / l : 0.f;
    T* O = (T*)a.o;
#pragma unroll
    for (int d = 0; d < HD; ++d) Elem<T>::store(O, (rowb + i) * a.ldo + (int64_t)h * HD + d, o[d] * inv);
    a.lse[((int64_t)b * a.Hq + h) * a.S + i] = l > 0.f ? m + __logf(l) : -INFINITY;
  }
}

// delta[b, h, i] = sum_d dO[i, h, d] * O[i, h, d]
template <typename T>
__global__ void attn_delta(AttnDesc a) {
  const int64_t n = (int64_t)a.B * a.Hq * a.S;
  const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (t >= n) return;
  const int i = (int)(t % a.S);
  const int h = (int)((t / a.S) % a.Hq);
  const int b = (int)(t / ((int64_t)a.S * a.Hq));
  const int64_t row = (int64_t)b * a.S + i;
  const T* O = (const T*)a.o;
  const T* dO = (const T*)a.dout;
  float s = 0.f;
  for (int d = 0; d < a.hd; ++d)
    s += ld(O, row * a.ldo + (int64_t)h * a.hd + d) * ld(dO, row * a.lddo + (int64_t)h * a.hd + d);
  a.delta[t] = s;
}

template <typename T, int HD>
__global__ void __launch_bounds__(AT) attn_dq_simt(AttnDesc a) {
  __shared__ float ks[KT][HD + 1], vs[KT][HD + 1];
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (a.Hq / a.Hkv);
  const int i = blockIdx.x * AT + threadIdx.x;
  const int L = a.seq_lens[b];
  const int64_t rowb = (int64_t)b * a.S;
  const T* Q = (const T*)a.q;
  const T* K = (const T*)a.k;
  const T* Vv = (const T*)a.v;
  const T* dO = (const T*)a.dout;
  float q[HD], dov[HD], dq[HD];
  float lse = -INFINITY, dl = 0.f;
  if (i < a.S) {
    lse = a.lse[((int64_t)b * a.Hq + h) * a.S + i];
    dl = a.delta[((int64_t)b * a.Hq + h) * a.S + i];
  }
#pragma unroll
  for (int d = 0; d < HD; ++d) {
    q[d] = i < a.S ? ld(Q, (rowb + i) * a.ldq + (int64_t)h * HD + d) * a.scale : 0.f;
    dov[d] = i < a.S ? ld(dO, (rowb + i) * a.lddo + (int64_t)h * HD + d) : 0.f;
    dq[d] = 0.f;
  }
  const int kend = min(min(blockIdx.x * AT + AT, a.S), L);
  for (int j0 = 0; j0 < kend; j0 += KT) {
    for (int e = threadIdx.x; e < KT * HD; e += AT) {
      const int r = e / HD, d = e % HD;
      const int j = j0 + r;
      float kv = 0.f, vv = 0.f;
      if (j < kend) {
        kv = ld(K, (rowb + j) * a.ldk + (int64_t)g * HD + d);
        vv = ld(Vv, (rowb + j) * a.ldv + (int64_t)g * HD + d);
      }
      ks[r][d] = kv;
      vs[r][d] = vv;
    }
    __syncthreads();
    for (int r = 0; r < KT; ++r) {
      const int j = j0 + r;
      if (j < kend && j <= i && i < a.S && lse != -INFINITY) {
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int d = 0; d < HD; ++d) {
          s += q[d] * ks[r][d];
          dp += dov[d] * vs[r][d];
        }
        const float p = __expf(s - lse);
        const float ds = p * (dp - dl);
#pragma unroll
        for (int d = 0; d < HD; ++d) dq[d] += ds * ks[r][d];
      }
    }
    __syncthreads();
  }
  if (i < a.S) {
    T* DQ = (T*)a.dq;
#pragma unroll
    for (int d = 0; d < HD; ++d)
      Elem<T>::store(DQ, (rowb + i) * a.lddq + (int64_t)h * HD + d, dq[d] * a.scale);
  }
}

template <typename T, int HD>
__global__ void __launch_bounds__(AT) attn_dkv_simt(AttnDesc a) {
  __shared__ float qs[KT][HD + 1], dos[KT][HD + 1];
  __shared__ float lses[KT], dls[KT];
  const int g = blockIdx.y, b = blockIdx.z;
  const int grp = a.Hq / a.Hkv;
  const int j = blockIdx.x * AT + threadIdx.x;
  const int L = a.seq_lens[b];
  const int64_t rowb = (int64_t)b * a.S;
  const T* Q = (const T*)a.q;
  const T* K = (const T*)a.k;
  const T* Vv = (const T*)a.v;
  const T* dO = (const T*)a.dout;
  const bool live = j < a.S && j < L;
  float k[HD], v[HD], dk[HD], dv[HD];
#pragma unroll
  for (int d = 0; d < HD; ++d) {
    k[d] = live ? ld(K, (rowb + j) * a.ldk + (int64_t)g * HD + d) : 0.f;
    v[d] = live ? ld(Vv, (rowb + j) * a.ldv + (int64_t)g * HD + d) : 0.f;
    dk[d] = 0.f;
    dv[d] = 0.f;
  }
  const int istart = blockIdx.x * AT;
  for (int hh = 0; hh < grp; ++hh) {
    const int h = g * grp + hh;
    for (int i0 = istart; i0 < a.S; i0 += KT) {
      for (int e = threadIdx.x; e < KT * HD; e += AT) {
        const int r = e / HD, d = e % HD;
        const int i = i0 + r;
        float qv = 0.f, dv_ = 0.f;
        if (i < a.S) {
          qv = ld(Q, (rowb + i) * a.ldq + (int64_t)h * HD + d) * a.scale;
          dv_ = ld(dO, (rowb + i) * a.lddo + (int64_t)h * HD + d);
        }
        qs[r][d] = qv;
        dos[r][d] = dv_;
      }
      if (threadIdx.x < KT) {
        const int i = i0 + threadIdx.x;
        lses[threadIdx.x] = i < a.S ? a.lse[((int64_t)b * a.Hq + h) * a.S + i] : -INFINITY;
        dls[threadIdx.x] = i < a.S ? a.delta[((int64_t)b * a.Hq + h) * a.S + i] : 0.f;
      }
      __syncthreads();
      if (live) {
        for (int r = 0; r < KT; ++r) {
          const int i = i0 + r;
          if (i < a.S && i >= j && lses[r] != -INFINITY) {
            float s = 0.f, dp = 0.f;
#pragma unroll
            for (int d = 0; d < HD; ++d) {
              s += qs[r][d] * k[d];
              dp += dos[r][d] * v[d];
            }
            const float p = __expf(s - lses[r]);
            const float ds = p * (dp - dls[r]);
#pragma unroll
            for (int d = 0; d < HD; ++d) {
              dv[d] += p * dos[r][d];
              dk[d] += ds * qs[r][d];  // qs already carries the scale
            }
          }
        }
      }
      __syncthreads();
    }
  }
  if (j < a.S) {
    T* DK = (T*)a.dk;
    T* DV = (T*)a.dv;
#pragma unroll
    for (int d = 0; d < HD; ++d) {
      Elem<T>::store(DK, (rowb + j) * a.lddk + (int64_t)g * HD + d, dk[d]);
      Elem<T>::store(DV, (rowb + j) * a.lddv + (int64_t)g * HD + d, dv[d]);
    }
  }
}

template <typename T, int HD>
static hipError_t fwd_simt(const AttnDesc& a, hipStream_t s) {
  dim3 grid((a.S + AT - 1) / AT, a.Hq, a.B);
  hipLaunchKernelGGL((attn_fwd_simt<T, HD>), grid, dim3(AT), 0, s, a);
  return hipGetLastError();
}

template <typename T, int HD>
static hipError_t bwd_simt(const AttnDesc& a, hipStream_t s) {
  const int64_t n = (int64_t)a.B * a.Hq * a.S;
  hipLaunchKernelGGL((attn_delta<T>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  dim3 gq((a.S + AT - 1) / AT, a.Hq, a.B);
  hipLaunchKernelGGL((attn_dq_simt<T, HD>), gq, dim3(AT), 0, s, a);
  dim3 gk((a.S + AT - 1) / AT, a.Hkv, a.B);
  hipLaunchKernelGGL((attn_dkv_simt<T, HD>), gk, dim3(AT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn_fwd_mfma(const AttnDesc& a, hipStream_t s, bool* handled);
hipError_t launch_attn_bwd_mfma(const AttnDesc& a, hipStream_t s, bool* handled);

#define ZL_HD_DISPATCH(FN, T)                      \
  switch (a.hd) {                                  \
    case 16: return FN<T, 16>(a, s);               \
    case 32: return FN<T, 32>(a, s);               \
    case 64: return FN<T, 64>(a, s);               \
    case 128: return FN<T, 128>(a, s);             \
    default: return hipErrorInvalidValue;          \
  }

hipError_t launch_attn_fwd(const AttnDesc& a, int dtype, hipStream_t s) {
  if (a.B <= 0 || a.S <= 0) return hipSuccess;
  if (dtype == BF16) {
    bool handled = false;
    hipError_t e = launch_attn_fwd_mfma(a, s, &handled);
    if (handled) return e;
    ZL_HD_DISPATCH(fwd_simt, bf16_t)
  }
  ZL_HD_DISPATCH(fwd_simt, float)
}

hipError_t launch_attn_bwd(const AttnDesc& a, int dtype, hipStream_t s, bool* rope_fused) {
  *rope_fused = false;
  if (a.B <= 0 || a.S <= 0) return hipSuccess;
  if (dtype == BF16) {
    bool handled = false;
    hipError_t e = launch_attn_bwd_mfma(a, s, &handled);
    if (handled) {
      *rope_fused = a.rope != nullptr;
      return e;
    }
    ZL_HD_DISPATCH(bwd_simt, bf16_t)
  }
  ZL_HD_DISPATCH(bwd_simt, float)
}

}  // namespace zl
