// GEMM kernels for every linear of the chunk map (Eq. (1)) and the frozen
// readout head (Eq. (2)), forward, data-gradient and weight-gradient forms.
//
// bf16: MFMA 16x16x32 or 32x32x16 (fp32 accumulate) on LDS tiles with
// 16-byte XOR-swizzled rows and an XCD-aware tile order so tiles sharing
// operand panels run on one L2.  The main path copies tiles global -> LDS
// with the buffer unit's direct-to-LDS loads and reads MN-major operands
// with LDS transpose reads; a register-staged path (8x8 in-register
// transposes) covers operands that do not meet the direct path's alignment.
// fp32: a plain LDS-tiled SIMT kernel (the fp32 configuration is small).
#include <stdio.h>

#include <cstring>
#include <type_traits>

#include "common.h"

#ifndef GEMM_IL  // main-loop schedule of the direct-to-LDS kernel
#define GEMM_IL 2
#endif

namespace zl {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// The two bf16 MFMA shapes (fp32 accumulate).  MF x MF output block, KS-deep
// k slice; every lane supplies 8 bf16 of A and of B.  Output register r of
// lane l holds row row(l, r), column l % MF.
template <int MF> struct Mma;
template <> struct Mma<32> {  // v_mfma_f32_32x32x16_bf16: A row l & 31, k 8 (l >> 5) .. +7
  using acc_t = f32x16_t;
  static constexpr int KS = 16, NR = 16;
  __device__ static inline acc_t run(bf16x8_t a, bf16x8_t b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static constexpr int row(int l, int r) { return 8 * (r >> 2) + 4 * (l >> 5) + (r & 3); }
};
template <> struct Mma<16> {  // v_mfma_f32_16x16x32_bf16: A row l & 15, k 8 (l >> 4) .. +7
  using acc_t = f32x4_t;
  static constexpr int KS = 32, NR = 4;
  __device__ static inline acc_t run(bf16x8_t a, bf16x8_t b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static constexpr int row(int l, int r) { return 4 * (l >> 4) + r; }
};

// f(std::integral_constant<int, i>) for i = B .. E-1: indices that are
// compile-time constants by construction, whatever the unroller decides
// (a register array indexed at run time would live in scratch memory).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// ---------------------------------------------------------------- epilogue
__device__ inline float silu_f(float g) { return g / (1.f + __expf(-g)); }

__device__ inline float gelu_f(float x) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  float t = tanhf(c * (x + 0.044715f * x * x * x));
  return 0.5f * x * (1.f + t);
}
__device__ inline float gelu_grad_f(float x) {
  const float c = 0.7978845608028654f;
  float t = tanhf(c * (x + 0.044715f * x * x * x));
  float dt = (1.f - t * t) * c * (1.f + 3.f * 0.044715f * x * x);
  return 0.5f * (1.f + t) + 0.5f * x * dt;
}

__device__ __forceinline__ float ld_act(const void* p, int dt, size_t i) {
  if (dt == F16) return f16_to_f32(((const uint16_t*)p)[i]);
  return dt == BF16 ? bf16_to_f32(((const bf16_t*)p)[i]) : ((const float*)p)[i];
}
__device__ __forceinline__ void st_act(void* p, int dt, size_t i, float v) {
  if (dt == F16) ((uint16_t*)p)[i] = f32_to_f16(v);
  else if (dt == BF16) ((bf16_t*)p)[i] = f32_to_bf16(v);
  else ((float*)p)[i] = v;
}

__device__ __forceinline__ void epilogue(const EpiArgs& e, int M, int N, int m, int n, float acc) {
  if (m >= M || n >= N) return;
  const size_t mo = (size_t)m;
  switch (e.kind) {
    case EPI_STORE:
    case EPI_STORE_DELTA: {
      float v = e.scale * acc + (e.bias ? e.bias[n] : 0.f);
      st_act(e.out, e.out_dtype, mo * e.ldo + n, v);
      break;
    }
    case EPI_RESID: {
      float v = e.resid[mo * e.ldr + n] + acc + (e.bias ? e.bias[n] : 0.f);
      ((float*)e.out)[mo * e.ldo + n] = v;
      break;
    }
    case EPI_GELU: {
      float h = acc + (e.bias ? e.bias[n] : 0.f);
      if (e.out_dtype == BF16) h = bf16_to_f32(f32_to_bf16(h));  // as stored
      st_act(e.out2, e.out_dtype, mo * e.ldo2 + n, h);
      st_act(e.out, e.out_dtype, mo * e.ldo + n, gelu_f(h));
      break;
    }
    case EPI_GRAD: {
      float* o = (float*)e.out + mo * e.ldo + n;
      float v = e.scale * acc;
      *o = e.accumulate ? *o + v : v;
      break;
    }
    case EPI_SWIGLU_BWD: {
      float g = ld_act(e.aux, e.out_dtype, mo * e.ldaux + n);
      float u = ld_act(e.aux, e.out_dtype, mo * e.ldaux + n + e.ff);
      float sg = __builtin_amdgcn_rcpf(1.f + __expf(-g));  // hardware reciprocal (1 ulp)
      float silu = g * sg;
      float dsilu = sg * (1.f + g * (1.f - sg));
      st_act(e.out, e.out_dtype, mo * e.ldo + n, acc * u * dsilu);
      st_act(e.out, e.out_dtype, mo * e.ldo + n + e.ff, acc * silu);
      break;
    }
    case EPI_GELU_BWD: {
      float h = ld_act(e.aux, e.out_dtype, mo * e.ldaux + n);
      st_act(e.out, e.out_dtype, mo * e.ldo + n, acc * gelu_grad_f(h));
      break;
    }
    case EPI_ROPE:  // rotation already applied by the staged epilogue
    case EPI_LOGITS:  // the staged epilogue adds the row statistics
      st_act(e.out, e.out_dtype, mo * e.ldo + n, acc);
      break;
  }
}

// EW consecutive columns n .. n+EW-1 of row m.  The vector path (vec: every
// operand 16-byte aligned, every row stride a multiple of 8, checked once
// per block) loads and stores them at once (16-byte accesses for bf16) with
// the same arithmetic as epilogue(); the column tail and unaligned operands
// take the scalar path.
constexpr int EW = 8;
__device__ __forceinline__ void ldv_f32(const float* p, float (&v)[EW]) {
#pragma unroll
  for (int k = 0; k < EW; k += 4) {
    const float4 f = *reinterpret_cast<const float4*>(p + k);
    v[k] = f.x; v[k + 1] = f.y; v[k + 2] = f.z; v[k + 3] = f.w;
  }
}
__device__ __forceinline__ void unpack_bf16x8(const uint4 u, float (&v)[EW]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = bf16_to_f32((bf16_t)(w[k] & 0xffff));
    v[2 * k + 1] = bf16_to_f32((bf16_t)(w[k] >> 16));
  }
}
__device__ __forceinline__ void ldv_act(const void* p, int dt, size_t i, float (&v)[EW]) {
  if (dt == BF16) {
    unpack_bf16x8(*reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(p) + i), v);
  } else {
    ldv_f32(static_cast<const float*>(p) + i, v);
  }
}
// dL/dg and dL/du of SwiGLU a = silu(g) u from da, and dL/dh of GELU
__device__ __forceinline__ void swiglu_bwd8(const float (&da)[EW], const float (&g)[EW],
                                            const float (&u)[EW], float (&dg)[EW], float (&du)[EW]) {
#pragma unroll
  for (int i = 0; i < EW; ++i) {
    const float sg = __builtin_amdgcn_rcpf(1.f + __expf(-g[i]));  // hardware reciprocal (1 ulp)
    const float silu = g[i] * sg;
    const float dsilu = sg * (1.f + g[i] * (1.f - sg));
    dg[i] = da[i] * u[i] * dsilu;
    du[i] = da[i] * silu;
  }
}
__device__ __forceinline__ void stv_act(void* p, int dt, size_t i, const float (&v)[EW]) {
  if (dt == BF16) {
    uint32_t w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      w[k] = (uint32_t)f32_to_bf16(v[2 * k]) | ((uint32_t)f32_to_bf16(v[2 * k + 1]) << 16);
    *reinterpret_cast<uint4*>(static_cast<bf16_t*>(p) + i) = make_uint4(w[0], w[1], w[2], w[3]);
  } else if (dt == F16) {
    uint32_t w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      w[k] = (uint32_t)f32_to_f16(v[2 * k]) | ((uint32_t)f32_to_f16(v[2 * k + 1]) << 16);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p) + i) = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
    float* q = static_cast<float*>(p) + i;
#pragma unroll
    for (int k = 0; k < EW; k += 4)
      *reinterpret_cast<float4*>(q + k) = make_float4(v[k], v[k + 1], v[k + 2], v[k + 3]);
  }
}

__device__ __forceinline__ bool epi_vec_ok(const EpiArgs& e) {
  const uintptr_t p = (uintptr_t)e.out | (uintptr_t)e.bias | (uintptr_t)e.resid |
                      (uintptr_t)e.out2 | (uintptr_t)e.aux;
  const int64_t l = e.ldo | e.ldr | e.ldo2 | e.ldaux | (int64_t)e.ff;
  return (p & 15) == 0 && (l & 7) == 0;
}

__device__ __forceinline__ void epilogue_v(const EpiArgs& e, int M, int N, int m, int n,
                                  const float (&a)[EW], bool vec) {
  if (m >= M) return;
  if (!vec || n + EW > N) {
#pragma unroll
    for (int i = 0; i < EW; ++i) epilogue(e, M, N, m, n + i, a[i]);
    return;
  }
  const size_t mo = (size_t)m;
  float v[EW], b[EW];
#pragma unroll
  for (int i = 0; i < EW; ++i) b[i] = 0.f;
  if (e.bias && (e.kind == EPI_STORE || e.kind == EPI_STORE_DELTA || e.kind == EPI_RESID ||
                 e.kind == EPI_GELU))
    ldv_f32(e.bias + n, b);
  switch (e.kind) {
    case EPI_STORE:
    case EPI_STORE_DELTA:
#pragma unroll
      for (int i = 0; i < EW; ++i) v[i] = e.scale * a[i] + b[i];
      stv_act(e.out, e.out_dtype, mo * e.ldo + n, v);
      break;
    case EPI_RESID: {
      float r[EW];
      ldv_f32(e.resid + mo * e.ldr + n, r);
#pragma unroll
      for (int i = 0; i < EW; ++i) v[i] = r[i] + a[i] + b[i];
      stv_act(e.out, F32, mo * e.ldo + n, v);
      break;
    }
    case EPI_GELU: {
      float h[EW];
#pragma unroll
      for (int i = 0; i < EW; ++i) {
        h[i] = a[i] + b[i];
        if (e.out_dtype == BF16) h[i] = bf16_to_f32(f32_to_bf16(h[i]));  // as stored
        v[i] = gelu_f(h[i]);
      }
      stv_act(e.out2, e.out_dtype, mo * e.ldo2 + n, h);
      stv_act(e.out, e.out_dtype, mo * e.ldo + n, v);
      break;
    }
    case EPI_GRAD: {
      float* o = static_cast<float*>(e.out) + mo * e.ldo + n;
#pragma unroll
      for (int i = 0; i < EW; ++i) v[i] = e.scale * a[i];
      if (e.accumulate) {
        float f[EW];
        ldv_f32(o, f);
#pragma unroll
        for (int i = 0; i < EW; ++i) v[i] = f[i] + v[i];
      }
      stv_act(o, F32, 0, v);
      break;
    }
    case EPI_SWIGLU_BWD: {
      float g[EW], u[EW], w[EW];
      ldv_act(e.aux, e.out_dtype, mo * e.ldaux + n, g);
      ldv_act(e.aux, e.out_dtype, mo * e.ldaux + n + e.ff, u);
      swiglu_bwd8(a, g, u, v, w);
      stv_act(e.out, e.out_dtype, mo * e.ldo + n, v);
      stv_act(e.out, e.out_dtype, mo * e.ldo + n + e.ff, w);
      break;
    }
    case EPI_GELU_BWD: {
      float h[EW];
      ldv_act(e.aux, e.out_dtype, mo * e.ldaux + n, h);
#pragma unroll
      for (int i = 0; i < EW; ++i) v[i] = a[i] * gelu_grad_f(h[i]);
      stv_act(e.out, e.out_dtype, mo * e.ldo + n, v);
      break;
    }
    case EPI_ROPE:  // rotation already applied by the staged epilogue
    case EPI_LOGITS:
      stv_act(e.out, e.out_dtype, mo * e.ldo + n, a);
      break;
  }
}

// Reductions over aligned groups of 8 lanes with DPP moves, no LDS
// traffic: the partner across lane bit 0, then bit 1 (quad permutations),
// then the mirrored lane of the other quad of the 8 (row_half_mirror).
// Every lane of the group ends with the same value.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float max8(float x) {
  x = fmaxf(x, dpp_f32<0xB1>(x));   // quad_perm [1, 0, 3, 2]
  x = fmaxf(x, dpp_f32<0x4E>(x));   // quad_perm [2, 3, 0, 1]
  return fmaxf(x, dpp_f32<0x141>(x));
}
__device__ __forceinline__ float sum8(float x) {
  x += dpp_f32<0xB1>(x);
  x += dpp_f32<0x4E>(x);
  return x + dpp_f32<0x141>(x);
}

// Online-softmax partials (max, sum exp(x - max), sum exp(x - max) w).
struct SoftPart { float m, s, e; };

// ------------------------------------------------------------- tile order
// Grouped (GROUP_M row panels) order, then remapped so that the blocks the
// dispatcher places on one XCD (round-robin over 8) take a contiguous range
// of the grouped order and share A/B panels in that XCD's L2.
__device__ inline void tile_coords(int b, int nbm, int nbn, int& tm, int& tn) {
  const int nb = nbm * nbn;
  if (nb >= 64) {
    const int per = nb / 8, rem = nb % 8;
    const int x = b % 8, idx = b / 8;
    b = (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + idx;
  }
#ifndef GEMM_GROUP_M  // 4 measured best in the 8B update (2, 6, 8 and 16 slower)
#define GEMM_GROUP_M 4
#endif
  const int GROUP_M = GEMM_GROUP_M;
  const int group = b / (GROUP_M * nbn);
  const int first_m = group * GROUP_M;
  const int gsz = min(nbm - first_m, GROUP_M);
  const int in_group = b % (GROUP_M * nbn);
  tm = first_m + in_group % gsz;
  tn = in_group / gsz;
}

// Epilogue through LDS, one 32-row block of every wave tile at a time: the
// accumulators are written with compile-time indices (so they stay in
// registers), then read back row-contiguously, which coalesces the global
// stores of the epilogue.  Callers end their main loop with a barrier.
template <int BM, int BN, int WM, int WN, int MF = 32>
__device__ __forceinline__ void store_tile(const typename Mma<MF>::acc_t (&acc)[BM / WM / MF][BN / WN / MF],
                                  unsigned char* smem, const GemmDesc& g, const EpiArgs& e,
                                  int m0, int n0, int wave, int lane) {
  using acc_t = typename Mma<MF>::acc_t;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / MF;
  const int wm = wave / WN, wn = wave % WN;
  constexpr int LDW = TN + 4;
  static_assert(WM * WN * 32 * LDW * 4 <= 160 * 1024, "epilogue tile exceeds LDS");
  float* ep = reinterpret_cast<float*>(smem) + wave * 32 * LDW;
  const bool vec = epi_vec_ok(e);
  // One 32-row block per call; the calls are spelled out (not a loop) so
  // that every acc index stays a compile-time constant however large the
  // epilogue grows (a rolled loop would move acc to scratch memory).
  // a0: the 32 rows' accumulators (MF 32), or those of their first 16 rows
  // with a1 those of the second 16 (MF 16)
  auto chunk = [&](const acc_t (&a0)[FN], const acc_t (&a1)[FN], const int i) __attribute__((always_inline)) {
#pragma unroll
    for (int h = 0; h < 32 / MF; ++h)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < Mma<MF>::NR; ++r)
          ep[(h * MF + Mma<MF>::row(lane, r)) * LDW + j * MF + (lane & (MF - 1))] = (h ? a1 : a0)[j][r];
    __syncthreads();
    const int mb = m0 + wm * TM + i * 32, nb = n0 + wn * TN;
    // EW consecutive columns per lane: a row of TN columns takes TN / EW lanes
    constexpr int QPR = TN / EW;
    static_assert(TN % EW == 0, "wave tile width must hold whole column groups");
    if (e.zstride) {
      // split-K partial: raw fp32 accumulators of split z (no epilogue)
      float* base = static_cast<float*>(e.out) + (size_t)blockIdx.z * e.zstride;
      for (int t = lane; t < 32 * QPR; t += 64) {
        const int row = t / QPR, col = (t % QPR) * EW;
        const int m = mb + row, n = nb + col;
        if (m >= g.M) continue;
        float* o = base + (size_t)m * e.ldo + n;
        if (n + EW <= g.N && (e.ldo & 3) == 0) {
#pragma unroll
          for (int k = 0; k < EW; k += 4)
            *reinterpret_cast<float4*>(o + k) = *reinterpret_cast<const float4*>(&ep[row * LDW + col + k]);
        } else {
          for (int k = 0; k < EW && n + k < g.N; ++k) o[k] = ep[row * LDW + col + k];
        }
      }
    } else if (e.kind == EPI_ROPE) {
      // wave tiles are head-aligned (nb % hd == 0, TN % hd == 0) and half =
      // hd / 2 is a multiple of EW, so the partner columns j +- hd/2 of a
      // column group are again EW consecutive columns of the staged row
      const int half = e.hd >> 1;
      for (int t = lane; t < 32 * QPR; t += 64) {
        const int row = t / QPR, col = (t % QPR) * EW;
        const int n = nb + col, m = mb + row;
        float v[EW];
#pragma unroll
        for (int k = 0; k < EW; k += 4) {
          const float4 x = *reinterpret_cast<const float4*>(&ep[row * LDW + col + k]);
          v[k] = x.x; v[k + 1] = x.y; v[k + 2] = x.z; v[k + 3] = x.w;
        }
        if (n < e.n_rot && m < g.M) {
          const int j = n % e.hd;
          const bool lo = j < half;
          const int pc = lo ? col + half : col - half;
          float pv[EW];
#pragma unroll
          for (int k = 0; k < EW; k += 4) {
            const float4 y = *reinterpret_cast<const float4*>(&ep[row * LDW + pc + k]);
            pv[k] = y.x; pv[k + 1] = y.y; pv[k + 2] = y.z; pv[k + 3] = y.w;
          }
          int p = e.pos[m];
          p = p < 0 ? 0 : (p >= e.max_pos ? e.max_pos - 1 : p);
          const float2* cs = e.rope + (int64_t)p * half + (lo ? j : j - half);
#pragma unroll
          for (int k = 0; k < EW; ++k)
            v[k] = lo ? v[k] * cs[k].x - pv[k] * cs[k].y : v[k] * cs[k].x + pv[k] * cs[k].y;
        }
        epilogue_v(e, g.M, g.N, m, n, v, vec);
      }
    } else if (e.kind == EPI_STORE_DELTA) {
      // the hd / EW lanes of one head's columns in a row sum dO (as stored)
      // times O, giving the attention backward's delta of (row, head)
      const int lph = e.hd / EW;
      auto head_sum = [&](const int m, const int n, const float (&v)[EW], const float (&o)[EW])
          __attribute__((always_inline)) {
        float ds = 0.f;
#pragma unroll
        for (int k = 0; k < EW; ++k) {
          const float d = e.out_dtype == BF16 ? bf16_to_f32(f32_to_bf16(e.scale * v[k]))
                                              : e.scale * v[k];
          ds += d * o[k];
        }
        for (int off = 1; off < lph; off <<= 1) ds += __shfl_xor(ds, off, 64);
        if ((lane & (lph - 1)) == 0 && m < g.M && n < g.N) {
          const int b = m / e.seq, sq = m - b * e.seq, h = n / e.hd;
          e.delta[((int64_t)b * e.nheads + h) * e.seq + sq] = ds;
        }
      };
      if (vec && e.out_dtype == BF16 && mb + 32 <= g.M && nb + TN <= g.N) {
        // interior rows, bf16: O of all of this lane's column groups is
        // loaded before any dO is stored (the compiler must assume the
        // stores may alias the loads, so loads placed between them would
        // each wait a memory round trip)
        constexpr int IT = 32 * QPR / 64;
        static_assert(IT * 64 == 32 * QPR, "column groups must divide over the lanes");
        uint4 oa[IT];
        static_for<0, IT>([&](auto ic) __attribute__((always_inline)) {
          constexpr int it = decltype(ic)::value;
          const int t = lane + 64 * it, m = mb + t / QPR, n = nb + (t % QPR) * EW;
          oa[it] = *reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(e.aux) +
                                                   (size_t)m * e.ldaux + n);
        });
        static_for<0, IT>([&](auto ic) __attribute__((always_inline)) {
          constexpr int it = decltype(ic)::value;
          const int t = lane + 64 * it, row = t / QPR, col = (t % QPR) * EW;
          const int m = mb + row, n = nb + col;
          float v[EW], o[EW];
#pragma unroll
          for (int k = 0; k < EW; k += 4) {
            const float4 x = *reinterpret_cast<const float4*>(&ep[row * LDW + col + k]);
            v[k] = x.x; v[k + 1] = x.y; v[k + 2] = x.z; v[k + 3] = x.w;
          }
          float w[EW], bi[EW];  // dO as the plain store of epilogue_v writes it
#pragma unroll
          for (int k = 0; k < EW; ++k) bi[k] = 0.f;
          if (e.bias) ldv_f32(e.bias + n, bi);
#pragma unroll
          for (int k = 0; k < EW; ++k) w[k] = e.scale * v[k] + bi[k];
          stv_act(e.out, BF16, (size_t)m * e.ldo + n, w);
          unpack_bf16x8(oa[it], o);
          head_sum(m, n, v, o);
        });
      } else {
        for (int t = lane; t < 32 * QPR; t += 64) {
          const int row = t / QPR, col = (t % QPR) * EW;
          const int m = mb + row, n = nb + col;
          float v[EW], o[EW];
#pragma unroll
          for (int k = 0; k < EW; k += 4) {
            const float4 x = *reinterpret_cast<const float4*>(&ep[row * LDW + col + k]);
            v[k] = x.x; v[k + 1] = x.y; v[k + 2] = x.z; v[k + 3] = x.w;
          }
          epilogue_v(e, g.M, g.N, m, n, v, vec);
          if (m < g.M && n < g.N) ldv_act(e.aux, e.out_dtype, (size_t)m * e.ldaux + n, o);
          else
#pragma unroll
            for (int k = 0; k < EW; ++k) o[k] = 0.f;
          head_sum(m, n, v, o);
        }
      }
    } else if (e.kind == EPI_LOGITS) {
      // 8 lanes cover a 64-column block of one row (64 % EW == 0, TN % 64 == 0)
      static_assert(TN % 64 == 0, "logit statistics need 64-column blocks");
      // The maximum of one row's 64-column block (every lane of the 8 gets it).
      auto block_max = [&](const int n, const float (&v)[EW]) __attribute__((always_inline)) {
        float mx = -INFINITY;
#pragma unroll
        for (int k = 0; k < EW; ++k) mx = n + k < g.N ? fmaxf(mx, v[k]) : mx;
        static_assert(64 / EW == 8, "a 64-column block spans 8 lanes");
        return max8(mx);
      };
      // The cached logits: an fp16 cache holds z minus its block maximum
      // (kept in fp32 in the statistics), so its rounding error is relative
      // to |z - max|, not to |z|: large confident logits keep p = exp(z -
      // lse) to fp16 precision where p matters.  An fp32 cache holds z.
      auto store_logits = [&](const int m, const int n, const float (&v)[EW], const float mx)
          __attribute__((always_inline)) {
        if (e.out_dtype == F16) {
          float r[EW];
#pragma unroll
          for (int k = 0; k < EW; ++k) r[k] = v[k] - mx;
          epilogue_v(e, g.M, g.N, m, n, r, vec);
        } else {
          epilogue_v(e, g.M, g.N, m, n, v, vec);
        }
      };
      // Softmax partials of one row's 64-column block: the block maximum,
      // then one exponential per logit (exp2 of a fused multiply-add).
      auto block_stats = [&](const int m, const int n, const float (&v)[EW], const float (&w)[EW],
                             const float mx) __attribute__((always_inline)) {
        constexpr float L2E = 1.4426950408889634f;
        SoftPart sp = {mx, 0.f, 0.f};
        if (mx != -INFINITY) {
          const float nm = -mx * L2E;
#pragma unroll
          for (int k = 0; k < EW; ++k) {
            const float p = n + k < g.N ? __builtin_amdgcn_exp2f(__builtin_fmaf(v[k], L2E, nm)) : 0.f;
            sp.s += p;
            sp.e += p * w[k];
          }
        }
        sp.s = sum8(sp.s);
        sp.e = sum8(sp.e);
        if ((lane & (64 / EW - 1)) == 0 && m < g.M && n < g.N)
          e.stats[(int64_t)m * e.ldst + n / 64] = make_float4(sp.m, sp.s, sp.e, 0.f);
      };
      // the label's logit of a z row, in fp32 (the cache may be fp16)
      auto label_logit = [&](const int m, const int n, const float (&v)[EW])
          __attribute__((always_inline)) {
        if (e.zy && m < g.M) {
          const int tok = e.pair ? m >> 1 : m;
          const int y = e.lab[tok];
#pragma unroll
          for (int k = 0; k < EW; ++k)
            if (y == n + k) e.zy[tok] = v[k];
        }
      };
      if (e.pair) {
        // z rows are even and their z' rows follow (mb is even): a lane takes
        // both rows of its columns, so each staged value is read once and
        // z - z' is formed once
        static_assert((16 * QPR) % 64 == 0, "row pairs must divide over the lanes");
        for (int t = lane; t < 16 * QPR; t += 64) {
          const int row = 2 * (t / QPR), col = (t % QPR) * EW;
          const int m = mb + row, n = nb + col;
          float v[EW], u[EW], w[EW], wn[EW];
#pragma unroll
          for (int k = 0; k < EW; k += 4) {
            const float4 x = *reinterpret_cast<const float4*>(&ep[row * LDW + col + k]);
            const float4 y = *reinterpret_cast<const float4*>(&ep[(row + 1) * LDW + col + k]);
            v[k] = x.x; v[k + 1] = x.y; v[k + 2] = x.z; v[k + 3] = x.w;
            u[k] = y.x; u[k + 1] = y.y; u[k + 2] = y.z; u[k + 3] = y.w;
          }
#pragma unroll
          for (int k = 0; k < EW; ++k) {
            w[k] = v[k] - u[k];
            wn[k] = -w[k];
          }
          const float mv = block_max(n, v), mu = block_max(n, u);
          store_logits(m, n, v, mv);
          store_logits(m + 1, n, u, mu);
          label_logit(m, n, v);
          block_stats(m, n, v, w, mv);
          block_stats(m + 1, n, u, wn, mu);
        }
      } else {
        for (int t = lane; t < 32 * QPR; t += 64) {
          const int row = t / QPR, col = (t % QPR) * EW;
          const int m = mb + row, n = nb + col;
          float v[EW];
#pragma unroll
          for (int k = 0; k < EW; k += 4) {
            const float4 x = *reinterpret_cast<const float4*>(&ep[row * LDW + col + k]);
            v[k] = x.x; v[k + 1] = x.y; v[k + 2] = x.z; v[k + 3] = x.w;
          }
          const float mv = block_max(n, v);
          store_logits(m, n, v, mv);
          label_logit(m, n, v);
          block_stats(m, n, v, v, mv);
        }
      }
    } else if (vec && e.out_dtype == BF16 && (e.kind == EPI_SWIGLU_BWD || e.kind == EPI_GELU_BWD) &&
               mb + 32 <= g.M && nb + TN <= g.N) {
      // Interior rows, bf16: the activation inputs of all of this lane's
      // column groups are loaded before any result is stored (the compiler
      // must assume the stores may alias the loads, so loads placed between
      // them would each wait a memory round trip).
      constexpr int IT = 32 * QPR / 64;
      static_assert(IT * 64 == 32 * QPR, "column groups must divide over the lanes");
      const bool two = e.kind == EPI_SWIGLU_BWD;
      uint4 xa[IT], xb[IT];
      static_for<0, IT>([&](auto ic) __attribute__((always_inline)) {
        constexpr int it = decltype(ic)::value;
        const int t = lane + 64 * it, m = mb + t / QPR, n = nb + (t % QPR) * EW;
        const bf16_t* ap = static_cast<const bf16_t*>(e.aux) + (size_t)m * e.ldaux + n;
        xa[it] = *reinterpret_cast<const uint4*>(ap);
        xb[it] = two ? *reinterpret_cast<const uint4*>(ap + e.ff) : make_uint4(0, 0, 0, 0);
      });
      static_for<0, IT>([&](auto ic) __attribute__((always_inline)) {
        constexpr int it = decltype(ic)::value;
        const int t = lane + 64 * it, row = t / QPR, col = (t % QPR) * EW;
        const size_t mo = (size_t)(mb + row);
        const int n = nb + col;
        float v[EW], x[EW], r[EW];
#pragma unroll
        for (int k = 0; k < EW; k += 4) {
          const float4 f = *reinterpret_cast<const float4*>(&ep[row * LDW + col + k]);
          v[k] = f.x; v[k + 1] = f.y; v[k + 2] = f.z; v[k + 3] = f.w;
        }
        unpack_bf16x8(xa[it], x);
        if (two) {
          float u[EW], w[EW];
          unpack_bf16x8(xb[it], u);
          swiglu_bwd8(v, x, u, r, w);
          stv_act(e.out, BF16, mo * e.ldo + n + e.ff, w);
        } else {
#pragma unroll
          for (int k = 0; k < EW; ++k) r[k] = v[k] * gelu_grad_f(x[k]);
        }
        stv_act(e.out, BF16, mo * e.ldo + n, r);
      });
    } else {
      for (int t = lane; t < 32 * QPR; t += 64) {
        const int row = t / QPR, col = (t % QPR) * EW;
        float v[EW];
#pragma unroll
        for (int k = 0; k < EW; k += 4) {
          const float4 x = *reinterpret_cast<const float4*>(&ep[row * LDW + col + k]);
          v[k] = x.x; v[k + 1] = x.y; v[k + 2] = x.z; v[k + 3] = x.w;
        }
        epilogue_v(e, g.M, g.N, mb + row, nb + col, v, vec);
      }
    }
    __syncthreads();
  };
  static_assert(FM >= 1 && FM <= 4, "32-row blocks per wave tile");
  constexpr int S = 32 / MF;  // accumulator row blocks per 32-row block
  chunk(acc[0], acc[S - 1], 0);
  if constexpr (FM > 1) chunk(acc[S], acc[2 * S - 1], 1);
  if constexpr (FM > 2) chunk(acc[2 * S], acc[3 * S - 1], 2);
  if constexpr (FM > 3) chunk(acc[3 * S], acc[4 * S - 1], 3);
}

// ------------------------------------------------------------ MFMA kernel
constexpr int BKT = 64;  // K-tile (elements)

__device__ inline int swz(int row) { return (row >> 1) & 7; }

// Transpose an 8x8 bf16 block held as 8 rows of 8 (uint4 = 4 x 2 bf16).
__device__ inline void transpose8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
  const uint32_t* iw = reinterpret_cast<const uint32_t*>(in);
  uint32_t* ow = reinterpret_cast<uint32_t*>(out);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t lo = iw[(2 * q) * 4 + j / 2];
      uint32_t hi = iw[(2 * q + 1) * 4 + j / 2];
      ow[j * 4 + q] = __builtin_amdgcn_perm(hi, lo, (j & 1) ? 0x07060302u : 0x05040100u);
    }
  }
}

// Per-thread staging of one operand tile (R rows of the MN dimension x 64 k).
template <int R, int NT, bool KMAJ>
struct Stage {
  // K-major: R*8 chunks of 16B; MN-major: R blocks of 8x8 (8 chunks each).
  static constexpr int ITEMS = KMAJ ? (R * 8 + NT - 1) / NT : (R + NT - 1) / NT;
  static constexpr int REGS = KMAJ ? ITEMS : ITEMS * 8;
  uint4 r[REGS];

  __device__ inline void load(const bf16_t* __restrict__ base, int64_t ld, int r0, int rmax,
                              int k0, int kvalid) {
    const int tid = threadIdx.x;
    if (KMAJ) {
#pragma unroll
      for (int i = 0; i < ITEMS; ++i) {
        const int c = tid + i * NT;
        const int row = c >> 3, kc = c & 7;
        const int gr = r0 + row, gk = k0 + kc * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (c < R * 8 && gr < rmax && gk < kvalid)
          v = *reinterpret_cast<const uint4*>(base + (int64_t)gr * ld + gk);
        r[i] = v;
      }
    } else {
#pragma unroll
      for (int i = 0; i < ITEMS; ++i) {
        const int b = tid + i * NT;
        const int kb = b & 7, mb = b >> 3;
        const int gm = r0 + mb * 8;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int gk = k0 + kb * 8 + t;
          uint4 v = make_uint4(0, 0, 0, 0);
          if (b < R && gm < rmax && gk < kvalid)
            v = *reinterpret_cast<const uint4*>(base + (int64_t)gk * ld + gm);
          r[i * 8 + t] = v;
        }
      }
    }
  }

  __device__ inline void store(bf16_t* __restrict__ lds) const {
    const int tid = threadIdx.x;
    if (KMAJ) {
#pragma unroll
      for (int i = 0; i < ITEMS; ++i) {
        const int c = tid + i * NT;
        if (c < R * 8) {
          const int row = c >> 3, kc = c & 7;
          *reinterpret_cast<uint4*>(lds + row * BKT + ((kc ^ swz(row)) * 8)) = r[i];
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < ITEMS; ++i) {
        const int b = tid + i * NT;
        if (b < R) {
          const int kb = b & 7, mb = b >> 3;
          uint4 in[8], out[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) in[t] = r[i * 8 + t];
          transpose8x8(in, out);
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int row = mb * 8 + j;
            *reinterpret_cast<uint4*>(lds + row * BKT + ((kb ^ swz(row)) * 8)) = out[j];
          }
        }
      }
    }
  }
};

template <int BM, int BN, int WM, int WN, bool AK, bool BKM>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_mfma_kernel(GemmDesc g, EpiArgs e) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* As = reinterpret_cast<bf16_t*>(smem);
  bf16_t* Bs = As + 2 * BM * BKT;

  const int nbm = (g.M + BM - 1) / BM, nbn = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_coords(blockIdx.x, nbm, nbn, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave / WN, wn = wave % WN;

  const bf16_t* A = reinterpret_cast<const bf16_t*>(g.A);
  const bf16_t* B = reinterpret_cast<const bf16_t*>(g.B);

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  Stage<BM, NT, AK> sa;
  Stage<BN, NT, BKM> sb;
  const int nk = (g.K + BKT - 1) / BKT;
  constexpr int NS = BKT / 16;  // k16 slices per tile

  // Per-lane LDS element offsets of each k16 slice (loop invariant).  The
  // swizzle depends on the row only through (row >> 1) & 7 and fragment rows
  // step by 32, so fragment i adds the immediate i * 32 * BKT.
  int offA[NS], offB[NS];
  {
    const int l = lane & 31, h = lane >> 5, sw = (l >> 1) & 7;
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      offA[q] = (wm * TM + l) * BKT + (((2 * q + h) ^ sw) * 8);
      offB[q] = (wn * TN + l) * BKT + (((2 * q + h) ^ sw) * 8);
    }
  }

  sa.load(A, g.lda, m0, g.M, 0, g.ka);
  sb.load(B, g.ldb, n0, g.N, 0, g.kb);
  sa.store(As);
  sb.store(Bs);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      sa.load(A, g.lda, m0, g.M, (kt + 1) * BKT, g.ka);
      sb.load(B, g.ldb, n0, g.N, (kt + 1) * BKT, g.kb);
    }
    const bf16_t* as = As + cur * BM * BKT;
    const bf16_t* bs = Bs + cur * BN * BKT;
    // fragments double-buffered across slices: slice q+1 is read from LDS
    // while the MFMAs of slice q run
    bf16x8_t af[2][FM], bfr[2][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) af[0][i] = *reinterpret_cast<const bf16x8_t*>(as + offA[0] + i * 32 * BKT);
#pragma unroll
    for (int j = 0; j < FN; ++j) bfr[0][j] = *reinterpret_cast<const bf16x8_t*>(bs + offB[0] + j * 32 * BKT);
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      const int cb = q & 1, nb = cb ^ 1;
      if (q + 1 < NS) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
          af[nb][i] = *reinterpret_cast<const bf16x8_t*>(as + offA[q + 1] + i * 32 * BKT);
#pragma unroll
        for (int j = 0; j < FN; ++j)
          bfr[nb][j] = *reinterpret_cast<const bf16x8_t*>(bs + offB[q + 1] + j * 32 * BKT);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cb][i], bfr[cb][j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      sa.store(As + (cur ^ 1) * BM * BKT);
      sb.store(Bs + (cur ^ 1) * BN * BKT);
    }
    __syncthreads();
  }
  // second K segment (same layouts), one tile at a time
  for (int k0 = 0; k0 < g.K2; k0 += BKT) {
    sa.load(reinterpret_cast<const bf16_t*>(g.A2), g.lda2, m0, g.M, k0, g.K2);
    sb.load(reinterpret_cast<const bf16_t*>(g.B2), g.ldb2, n0, g.N, k0, g.K2);
    sa.store(As);
    sb.store(Bs);
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[i] = *reinterpret_cast<const bf16x8_t*>(As + offA[q] + i * 32 * BKT);
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[j] = *reinterpret_cast<const bf16x8_t*>(Bs + offB[q] + j * 32 * BKT);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }

  store_tile<BM, BN, WM, WN>(acc, smem, g, e, m0, n0, wave, lane);
}

// ------------------------------------------------- direct-to-LDS MFMA kernel
// Operand tiles are copied global -> LDS by the buffer unit (16 bytes per
// lane, lane i's bytes land at M0 + 16 i; an offset at or above the
// resource's record count reads as zero), so no staging registers, no LDS
// store instructions and no transposes.  LDS layouts:
//   K-major operand  [row][64 k],  16-B chunk c of row r at c ^ ((r >> 1) & 7)
//   MN-major operand [k][R],       16-B chunk c of row k at c ^ xsk<MF>(k)
// and the DMA lane -> global mapping applies the inverse swizzle.  MN-major
// fragments are read with the LDS transpose read (ds_read_b64_tr_b16).
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
constexpr uint32_t DMA_OOB = 0x80000000u;  // record count; offsets >= it read as 0

__device__ inline i32x4_t buffer_rsrc(const void* base) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  i32x4_t r;
  r[0] = (int32_t)(uint32_t)p;
  r[1] = (int32_t)(uint32_t)(p >> 32);  // stride 0: raw byte addressing
  r[2] = (int32_t)DMA_OOB;
  r[3] = 0x00020000;
  return r;
}

// LDS-row swizzle of an MN-major tile: over any 4 consecutive k rows the
// values differ in bits 2-3 (distinct 64-byte bank groups for a half-wave
// transpose read) and in bits 1-2 (distinct 32-byte groups for 16 lanes).
__device__ inline int xs(int b) { return (0xCA60 >> (4 * b)) & 15; }
// The swizzle of LDS row k of an MN-major tile read as MF x MF fragments.
// A half-wave of 16x16 transpose reads covers k rows k0 .. k0 + 3 and
// k0 + 8 .. k0 + 11 (32 bytes each); folding bit 3 of k into the swizzle
// puts those 8 rows in 8 distinct 32-byte groups.
template <int MF>
__device__ inline int xsk(int k) { return MF == 16 ? xs(k & 3) ^ (k & 8) : xs(k & 3); }

extern "C" __device__ i32x4_t llvm_amdgcn_raw_buffer_load_v4i32(i32x4_t rsrc, uint32_t voffset,
                                                                 uint32_t soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.load.v4i32");
__device__ inline i32x4_t buffer_load16(i32x4_t rsrc, uint32_t voff) {
  return llvm_amdgcn_raw_buffer_load_v4i32(rsrc, voff, 0, 0);
}

__device__ inline void dma16(uint32_t lds_byte, uint32_t voff, i32x4_t rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_byte), "v"(voff), "s"(rsrc)
               : "memory");
}
__device__ inline void dma_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// K-major LDS rows of BK elements: 16-B chunk c of row r sits at
// c ^ ((r / 2) % (BK / 8)) for BK <= 64 (c ^ (r % 16) for BK 128).  A
// fragment read (16 consecutive rows, one chunk each, per 16 lanes) then
// takes 4 LDS cycles with no bank conflict, measured on gfx950 at BK 64 and
// 32; at BK 32 (64-byte rows) the earlier c ^ ((r / 4) % 4) took 8.
template <int BK>
__device__ inline int kswz(int row) { return (row / (BK <= 64 ? 2 : 128 / BK)) % (BK / 8); }

// One operand's BK-deep k tile, R rows of M (or N), copied by NT threads.
template <int R, int BK, int NT, bool KMAJ, int MF = 32>
struct DmaTile {
  static constexpr int ITEMS = R * BK / 8 / NT;  // 16-B chunks per thread
  static_assert(ITEMS >= 1 && ITEMS * NT == R * BK / 8, "tile chunks must divide over the threads");
  uint32_t off[ITEMS];  // byte offset at k0 = 0 from the tile origin, or DMA_OOB
  int kr[ITEMS];        // k of the chunk's first element within the tile
  uint32_t kstride;     // bytes per unit of k

  __device__ inline void init(int wave, int lane, int64_t ld, int rvalid) {
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      const int c = (wave * ITEMS + j) * 64 + lane;
      if (KMAJ) {
        constexpr int CR = BK / 8;
        const int row = c / CR, ch = (c % CR) ^ kswz<BK>(row);
        kr[j] = ch * 8;
        off[j] = row < rvalid ? (uint32_t)(row * ld) * 2u + (uint32_t)ch * 16u : DMA_OOB;
      } else {
        constexpr int CPR = R / 8;
        const int k = c / CPR, ch = (c % CPR) ^ xsk<MF>(k);
        kr[j] = k;
        off[j] = ch * 8 < rvalid ? (uint32_t)(k * ld) * 2u + (uint32_t)ch * 16u : DMA_OOB;
      }
    }
    kstride = KMAJ ? 2u : (uint32_t)ld * 2u;
  }
  __device__ inline uint32_t voff(int j, int k0, int kvalid) const {
    // a row outside the tile has off = DMA_OOB, and DMA_OOB plus any
    // in-range k advance (< 2^31) stays at or above the record count
    return k0 + kr[j] < kvalid ? off[j] + (uint32_t)k0 * kstride : DMA_OOB;
  }
  // Register path: the same chunks loaded into VGPRs (zero-filled in the
  // same way), then stored to the same contiguous LDS slots.
  __device__ inline void load(uint4 (&r)[ITEMS], int k0, int kvalid, i32x4_t rsrc) const {
#pragma unroll
    for (int j = 0; j < ITEMS; ++j)
      r[j] = __builtin_bit_cast(uint4, buffer_load16(rsrc, voff(j, k0, kvalid)));
  }
  __device__ inline void store(const uint4 (&r)[ITEMS], unsigned char* lds, int wave, int lane) const {
#pragma unroll
    for (int j = 0; j < ITEMS; ++j)
      *reinterpret_cast<uint4*>(lds + ((wave * ITEMS + j) * 64 + lane) * 16) = r[j];
  }
  __device__ inline void issue_one(int j, uint32_t lds_byte, int wave, int k0, int kvalid,
                                   i32x4_t rsrc) const {
    dma16(lds_byte + (uint32_t)(wave * ITEMS + j) * 1024u, voff(j, k0, kvalid), rsrc);
  }
  // Copy the tile starting at k0 into LDS at lds_byte.  Chunks at or past
  // kvalid (and rows outside the matrix) are zero-filled.
  __device__ inline void issue(uint32_t lds_byte, int wave, int k0, int kvalid, i32x4_t rsrc) const {
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      // a row outside the tile has off = DMA_OOB, and DMA_OOB plus any
      // in-range k advance (< 2^31) stays at or above the record count
      const uint32_t v = k0 + kr[j] < kvalid ? off[j] + (uint32_t)k0 * kstride : DMA_OOB;
      dma16(lds_byte + (uint32_t)(wave * ITEMS + j) * 1024u, v, rsrc);
    }
  }
};

// Per-lane LDS fragment addressing of one operand for the MF x MF MFMA
// (Mma<MF>): lane l supplies row l % MF and k 8 (l / MF) .. +7 of the
// KS-deep slice.  F fragments of MF rows each.
template <int R, int BK, int F, bool KMAJ, int MF = 32>
struct FragTile {
  static constexpr int KS = Mma<MF>::KS;
  static constexpr int NS = BK / KS;
  static constexpr int NO = KMAJ ? NS : F;
  int off[NO];  // element offsets: per slice (K-major) or per fragment (MN-major)

  __device__ inline void init(int wrow, int lane) {
    if (KMAJ) {
      // fragment rows step by MF, which keeps kswz (period 2 x BK/8 rows,
      // at most 16) unchanged: fragment i adds i * MF * BK
      const int l = lane & (MF - 1), h = lane / MF, sw = kswz<BK>(l);
#pragma unroll
      for (int q = 0; q < NS; ++q) off[q] = (wrow + l) * BK + ((((KS / 8) * q + h) ^ sw) * 8);
    } else if (MF == 32) {
      // transpose read: lane r of 16-lane group G addresses k row
      // 8 (G >> 1) + (r >> 2) (+ 16 q + 4 t) and the 4 elements at
      // m = wrow + 32 i + 16 (G & 1) + 4 (r & 3); it receives column
      // m = ... + r of those 4 k rows
      const int G = lane >> 4, r = lane & 15;
      const int kl = 8 * (G >> 1) + (r >> 2);
      const int P = (wrow >> 3) ^ (2 * (G & 1) + ((r >> 1) & 1)) ^ xs(r >> 2);
#pragma unroll
      for (int i = 0; i < F; ++i) off[i] = kl * R + ((P ^ (4 * i)) << 3) + 4 * (r & 1);
    } else {
      // transpose read: lane r of 16-lane group G addresses k row
      // 8 G + (r >> 2) (+ 32 q + 4 t) and the 4 elements at
      // m = wrow + 16 i + 4 (r & 3); it receives column m = ... + r of
      // those 4 k rows.  wrow is a multiple of 64, so the chunk index
      // (wrow >> 3) + 2 i + ((r >> 1) & 1) equals its XOR form.
      const int G = lane >> 4, r = lane & 15;
      const int kl = 8 * G + (r >> 2);
      const int P = (wrow >> 3) ^ ((r >> 1) & 1) ^ xsk<16>(kl);
#pragma unroll
      for (int i = 0; i < F; ++i) off[i] = kl * R + ((P ^ (2 * i)) << 3) + 4 * (r & 1);
    }
  }
  __device__ inline bf16x8_t read(const bf16_t* tile, int q, int i) const {
    if (KMAJ) {
      return *reinterpret_cast<const bf16x8_t*>(tile + off[q] + i * MF * BK);
    } else {
      const bf16_t* p = tile + off[i] + KS * q * R;
      const s16x4_t x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4_t*)(p));
      const s16x4_t y = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4_t*)(p + 4 * R));
      return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7));
    }
  }
};

// s_waitcnt with only the vector-memory count constrained (gfx9 encoding:
// vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// NST-stage pipeline: the tile NST - 1 steps ahead is in flight while the
// current one is multiplied; one barrier per BK-deep tile.  bl is the
// block's index among the tiles of its problem.
template <int BM, int BN, int WM, int WN, int BK, int NST, int DS, bool AK, bool BKM, bool RA, bool RB, int MF>
__device__ __forceinline__ void gemm_dma_body(const GemmDesc& g, const EpiArgs& e, const int bl,
                                              unsigned char* smem) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN;
  using M = Mma<MF>;
  using acc_t = typename M::acc_t;
  constexpr int FM = TM / MF, FN = TN / MF;
  constexpr int NS = BK / M::KS;
  // fragments of the next slice: double-buffered (MF 32), or refilled in
  // place right after their last use in the current slice (MF 16, whose
  // twice as many fragments would not fit twice beside the accumulators)
  constexpr int FB = MF == 32 ? 2 : 1;
  constexpr uint32_t ABYTES = BM * BK * 2, STAGE = (BM + BN) * BK * 2;
  using TA = DmaTile<BM, BK, NT, AK, MF>;
  using TB = DmaTile<BN, BK, NT, BKM, MF>;
  constexpr int PER_TILE = TA::ITEMS + TB::ITEMS;  // DMA instructions per wave per tile
  static_assert(NST >= 2 && (NST - 2) * PER_TILE < 64, "pipeline depth");
  static_assert(!(RA || RB) || NST == 2, "register staging uses two stages");
  static_assert(GEMM_IL == 2 || (DS >= 1 && DS < NS), "the tile copy is spread over slices before the last");
  static_assert(MF == 16 || NS % 2 == 0, "slice parity must repeat per tile");
  static_assert(MF == 32 || GEMM_IL, "16x16 fragments use the interleaved schedule");

  const int nbm = (g.M + BM - 1) / BM, nbn = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_coords(bl, nbm, nbn, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int wm = wave / WN, wn = wave % WN;

  // split K: this block's range [kbeg, kbeg + ksplit) of the reduction
  const int kz = blockIdx.z, kbeg = kz * g.ksplit;
  const int klen = min(g.K - kbeg, g.ksplit);
  const int ka = min(g.ka - kbeg, g.ksplit), kb = min(g.kb - kbeg, g.ksplit);
  const bf16_t* A = reinterpret_cast<const bf16_t*>(g.A) + (AK ? kbeg : (int64_t)kbeg * g.lda);
  const bf16_t* B = reinterpret_cast<const bf16_t*>(g.B) + (BKM ? kbeg : (int64_t)kbeg * g.ldb);
  const i32x4_t ra = buffer_rsrc(A + (AK ? (int64_t)m0 * g.lda : (int64_t)m0));
  const i32x4_t rb = buffer_rsrc(B + (BKM ? (int64_t)n0 * g.ldb : (int64_t)n0));
  TA da;
  TB db;
  da.init(wave, lane, g.lda, min(g.M - m0, BM));
  db.init(wave, lane, g.ldb, min(g.N - n0, BN));
  FragTile<BM, BK, FM, AK, MF> fa;
  FragTile<BN, BK, FN, BKM, MF> fb;
  fa.init(wm * TM, lane);
  fb.init(wn * TN, lane);

  acc_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < M::NR; ++r) acc[i][j][r] = 0.f;

  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>(smem);
  const int nk = (klen + BK - 1) / BK;
  // prologue: tiles 0 .. NST-2, or 0 .. NST-1 when each tile's copy is
  // issued as soon as its stage is released (tiles past K are zero-filled,
  // never used)
  constexpr int PRO = GEMM_IL == 2 ? NST : NST - 1;
#pragma unroll
  for (int t = 0; t < PRO; ++t) {
    da.issue(lds0 + t * STAGE, wave, t * BK, ka, ra);
    db.issue(lds0 + t * STAGE + ABYTES, wave, t * BK, kb, rb);
  }
  wait_vmcnt<(PRO - 1) * PER_TILE>();
  __syncthreads();
  // The fragments of the next KS-deep slice are read while the current
  // slice's MFMAs run (scheduling fences keep that order): into a second
  // register buffer (MF 32), or into each fragment's own registers right
  // after its last MFMA of the slice (MF 16).  The barrier that publishes
  // tile kt+1 sits before the MFMAs of tile kt's last slice, whose
  // fragments are already in registers, so slice 0 of tile kt+1 is read
  // while they run and the barrier also certifies that every wave is done
  // reading tile kt.
  bf16x8_t af[FB][FM], bfr[FB][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i) af[0][i] = fa.read(reinterpret_cast<const bf16_t*>(smem), 0, i);
#pragma unroll
  for (int j = 0; j < FN; ++j)
    bfr[0][j] = fb.read(reinterpret_cast<const bf16_t*>(smem) + BM * BK, 0, j);
  int rd = 0, wr = NST - 1;  // stage read this step, stage written this step
  uint4 rga[RA ? TA::ITEMS : 1], rgb[RB ? TB::ITEMS : 1];
  for (int kt = 0; kt < nk; ++kt) {
    const uint32_t dst = lds0 + wr * STAGE;
    const int k0n = (kt + NST - 1) * BK;
    if constexpr (RA) da.load(rga, k0n, ka, ra);
    if constexpr (RB) db.load(rgb, k0n, kb, rb);
    const int rn = rd + 1 == NST ? 0 : rd + 1;
    const bf16_t* as = reinterpret_cast<const bf16_t*>(smem + rd * STAGE);
    const bf16_t* an = reinterpret_cast<const bf16_t*>(smem + rn * STAGE);
#if GEMM_IL
    // Fine interleave: after each MFMA of slice q, the next slice's fragment
    // reads and this tile's share of the copy are issued in fixed places, so
    // the matrix pipe of a single wave per SIMD is never left waiting on an
    // issue burst.
    static_assert(!RA && !RB, "interleaved schedule uses direct-to-LDS copies");
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      const int cb = FB == 2 ? q & 1 : 0, nb = FB == 2 ? cb ^ 1 : 0;
      const bf16_t* src = q + 1 < NS ? as : an;
      const int qs = q + 1 < NS ? q + 1 : 0;
      if (q + 1 == NS) {
        wait_vmcnt<(NST - 2) * PER_TILE>();  // this wave's share of tile kt+1
        __syncthreads();                      // everyone's share; tile kt fully read
      }
      constexpr int NMF = FM * FN, NRD = FM + FN, TOT = TA::ITEMS + TB::ITEMS;
      // GEMM_IL == 2: tile kt + NST goes into stage rd right after the
      // barrier that releases it (last slice); else tile kt + NST - 1 into
      // stage wr over the first DS slices
      const bool early = GEMM_IL == 2;
      const bool dslice = early ? q + 1 == NS : q < DS;
      const int lo = !dslice ? 0 : early ? 0 : q * TOT / DS;
      const int hi = !dslice ? 0 : early ? TOT : (q + 1) * TOT / DS;
      const uint32_t ddst = early ? lds0 + rd * STAGE : dst;
      const int dk0 = early ? (kt + NST) * BK : k0n;
      const int span = hi > lo ? hi - lo : 1;
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < NMF; ++t) {
        acc[t / FN][t % FN] = M::run(af[cb][t / FN], bfr[cb][t % FN], acc[t / FN][t % FN]);
        if constexpr (FB == 2) {
#pragma unroll
          for (int r = 0; r < NRD; ++r) {
            if (r * NMF / NRD != t) continue;
            if (r < FM) af[nb][r] = fa.read(src, qs, r);
            else bfr[nb][r - FM] = fb.read(src + BM * BK, qs, r - FM);
          }
        } else {
          // rows i of A end at t = i FN + FN - 1; B columns are used
          // until the last row, the row the MFMAs run in order of
          const int ti = t / FN, tj = t % FN;
          if (ti + 1 == FM) bfr[0][tj] = fb.read(src + BM * BK, qs, tj);
          if (tj + 1 == FN) af[0][ti] = fa.read(src, qs, ti);
        }
#pragma unroll
        for (int u = 0; u < TOT; ++u) {
          if (u < lo || u >= hi || (u - lo) * NMF / span != t) continue;
          if (u < TA::ITEMS) da.issue_one(u, ddst, wave, dk0, ka, ra);
          else db.issue_one(u - TA::ITEMS, ddst + ABYTES, wave, dk0, kb, rb);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#else
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      const int cb = q & 1, nb = cb ^ 1;
      if (q + 1 < NS) {
#pragma unroll
        for (int i = 0; i < FM; ++i) af[nb][i] = fa.read(as, q + 1, i);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[nb][j] = fb.read(as + BM * BK, q + 1, j);
      } else {
        wait_vmcnt<(NST - 2) * PER_TILE>();  // this wave's share of tile kt+1
        if constexpr (RA) da.store(rga, smem + wr * STAGE, wave, lane);
        if constexpr (RB) db.store(rgb, smem + wr * STAGE + ABYTES, wave, lane);
        __syncthreads();                      // everyone's share; tile kt fully read
#pragma unroll
        for (int i = 0; i < FM; ++i) af[nb][i] = fa.read(an, 0, i);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[nb][j] = fb.read(an + BM * BK, 0, j);
      }
      // this slice's share of the copy of tile kt+NST-1: spreading the
      // copies keeps the vector-memory queue from stalling the MFMA issue
      if (q < DS) {
        constexpr int TOT = (RA ? 0 : TA::ITEMS) + (RB ? 0 : TB::ITEMS);
        const int lo = q * TOT / DS, hi = (q + 1) * TOT / DS;
#pragma unroll
        for (int t = 0; t < TOT; ++t) {
          if (t < lo || t >= hi) continue;
          const int ta = RA ? 0 : TA::ITEMS;
          if (t < ta) da.issue_one(t, dst, wave, k0n, ka, ra);
          else db.issue_one(t - ta, dst + ABYTES, wave, k0n, kb, rb);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = M::run(af[cb][i], bfr[cb][j], acc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
    }
#endif
    rd = rn;
    wr = wr + 1 == NST ? 0 : wr + 1;
  }
  dma_wait();  // the zero-fill copies past K must land before LDS is reused
  __syncthreads();
  if (g.K2 > 0 && kz == 0) {
    // second K segment (same layouts): one BK-deep tile at a time through
    // stage 0, copied and multiplied without overlap (K2 is a few tiles);
    // with split K the first split carries it
    const i32x4_t ra2 = buffer_rsrc(reinterpret_cast<const bf16_t*>(g.A2) +
                                    (AK ? (int64_t)m0 * g.lda2 : (int64_t)m0));
    const i32x4_t rb2 = buffer_rsrc(reinterpret_cast<const bf16_t*>(g.B2) +
                                    (BKM ? (int64_t)n0 * g.ldb2 : (int64_t)n0));
    da.init(wave, lane, g.lda2, min(g.M - m0, BM));
    db.init(wave, lane, g.ldb2, min(g.N - n0, BN));
    const bf16_t* as = reinterpret_cast<const bf16_t*>(smem);
    for (int k0 = 0; k0 < g.K2; k0 += BK) {
      da.issue(lds0, wave, k0, g.K2, ra2);
      db.issue(lds0 + ABYTES, wave, k0, g.K2, rb2);
      dma_wait();
      __syncthreads();
#pragma unroll
      for (int q = 0; q < NS; ++q) {
#pragma unroll
        for (int i = 0; i < FM; ++i) af[0][i] = fa.read(as, q, i);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[0][j] = fb.read(as + BM * BK, q, j);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = M::run(af[0][i], bfr[0][j], acc[i][j]);
      }
      __syncthreads();
    }
  }
  store_tile<BM, BN, WM, WN, MF>(acc, smem, g, e, m0, n0, wave, lane);
}

// One launch, one or two problems of the same layout: blocks below nb1 take
// (g, e), the rest (g2, e2) (two independent weight gradients share a launch
// so the last wave of one is filled by the other).  The problem is uniform
// per block; each branch inlines the body with its own descriptors.
template <int BM, int BN, int WM, int WN, int BK, int NST, int DS, bool AK, bool BKM, bool RA, bool RB, int MF>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_dma_kernel(GemmDesc g, EpiArgs e, GemmDesc g2, EpiArgs e2, int nb1) {
  extern __shared__ __align__(16) unsigned char smem[];
  if ((int)blockIdx.x < nb1)
    gemm_dma_body<BM, BN, WM, WN, BK, NST, DS, AK, BKM, RA, RB, MF>(g, e, blockIdx.x, smem);
  else
    gemm_dma_body<BM, BN, WM, WN, BK, NST, DS, AK, BKM, RA, RB, MF>(g2, e2, blockIdx.x - nb1, smem);
}

// ------------------------------------------------------------ SIMT (fp32)
template <bool AK, bool BKM>
__global__ void __launch_bounds__(256) gemm_simt_kernel(GemmDesc g, EpiArgs e) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  // segment 0: (A, B) over K; segment 1: (A2, B2) over K2
  for (int seg = 0; seg < 2; ++seg) {
  const float* A = reinterpret_cast<const float*>(seg ? g.A2 : g.A);
  const float* B = reinterpret_cast<const float*>(seg ? g.B2 : g.B);
  const int64_t lda = seg ? g.lda2 : g.lda, ldb = seg ? g.ldb2 : g.ldb;
  const int K = seg ? g.K2 : g.K, ka = seg ? g.K2 : g.ka, kb = seg ? g.K2 : g.kb;
  for (int k0 = 0; k0 < K; k0 += BK) {
    for (int idx = threadIdx.x; idx < BM * BK; idx += 256) {
      int r, k;
      if (AK) { r = idx / BK; k = idx % BK; } else { r = idx % BM; k = idx / BM; }
      const int gr = m0 + r, gk = k0 + k;
      float v = 0.f;
      if (gr < g.M && gk < ka) v = AK ? A[(int64_t)gr * lda + gk] : A[(int64_t)gk * lda + gr];
      As[k][r] = v;
    }
    for (int idx = threadIdx.x; idx < BN * BK; idx += 256) {
      int r, k;
      if (BKM) { r = idx / BK; k = idx % BK; } else { r = idx % BN; k = idx / BN; }
      const int gr = n0 + r, gk = k0 + k;
      float v = 0.f;
      if (gr < g.N && gk < kb) v = BKM ? B[(int64_t)gr * ldb + gk] : B[(int64_t)gk * ldb + gr];
      Bs[k][r] = v;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) epilogue(e, g.M, g.N, m0 + ty * 4 + i, n0 + tx * 4 + j, acc[i][j]);
}

// ------------------------------------------------------------------ launch
template <int BM, int BN, int WM, int WN, bool AK, bool BKM>
static hipError_t run_mfma(const GemmDesc& g, const EpiArgs& e, hipStream_t s) {
  auto kern = gemm_mfma_kernel<BM, BN, WM, WN, AK, BKM>;
  // LDS: the double-buffered operand tiles, reused by the epilogue's
  // 32-row fp32 staging of every wave tile
  const size_t lds_main = (size_t)2 * (BM + BN) * BKT * sizeof(bf16_t);
  const size_t lds_epi = (size_t)WM * WN * 32 * (BN / WN + 4) * sizeof(float);
  const size_t lds = lds_main > lds_epi ? lds_main : lds_epi;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute((const void*)kern,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int nb = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  hipLaunchKernelGGL(kern, dim3(nb), dim3(WM * WN * 64), lds, s, g, e);
  return hipGetLastError();
}

static const char* layout_tag(bool ak, bool bk) {
  return ak ? (bk ? "kk" : "kn") : (bk ? "mk" : "mn");
}

// Main-path configuration (compile-time; overridable for tuning builds)
#ifndef GEMM_BK
#define GEMM_BK 64
#endif
#ifndef GEMM_NST
#define GEMM_NST 2
#endif
#ifndef GEMM_BK_MN
#define GEMM_BK_MN 32
#endif
#ifndef GEMM_NST_MN
#define GEMM_NST_MN 3
#endif
// k-tile depth and stages per operand layout: both K-major (forward) BK 64
// with two stages; otherwise (an MN-major operand: data and weight
// gradients) BK 32 with three stages, measured faster in the 8B update
// MFMA shape per layout: 16x16x32 where an operand is K-major (6-8 %
// faster than 32x32x16 on the forward shapes, 2-3 % on the data-gradient
// ones), 32x32x16 when both are MN-major (weight gradients: 0.5 % faster)
#ifndef GEMM_MF
#define GEMM_MF 16
#endif
#ifndef GEMM_MF_MIX
#define GEMM_MF_MIX 16
#endif
#ifndef GEMM_MF_MN
#define GEMM_MF_MN 32
#endif
template <bool AK, bool BKM> struct KTile {
  static constexpr int BK = AK && BKM ? GEMM_BK : GEMM_BK_MN;
  static constexpr int NST = AK && BKM ? GEMM_NST : GEMM_NST_MN;
  static constexpr int MF = AK && BKM ? GEMM_MF : (AK || BKM ? GEMM_MF_MIX : GEMM_MF_MN);
};
#ifndef GEMM_DS
#define GEMM_DS 1
#endif
#ifndef GEMM_WM
#define GEMM_WM 4
#endif
#ifndef GEMM_WN
#define GEMM_WN 2
#endif
#ifndef GEMM_RA
#define GEMM_RA false
#endif
#ifndef GEMM_RB
#define GEMM_RB false
#endif


// Split-K reduction: C = sum over splits z = 0, 1, .. (in that order) of the
// fp32 partials, then the epilogue per element.
__global__ void __launch_bounds__(256) splitk_reduce_kernel(const float* __restrict__ part, int nz,
                                                            int M, int N, EpiArgs e) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t mn = (int64_t)M * N;
  if (i >= mn) return;
  float acc = 0.f;
  for (int z = 0; z < nz; ++z) acc += part[z * mn + i];
  epilogue(e, M, N, (int)(i / N), (int)(i % N), acc);
}

// Epilogues applied per element by the split-K reduction (the others need
// whole rows or column pairs of the staged tile).
static bool splitk_kind_ok(EpiKind k) {
  return k == EPI_STORE || k == EPI_RESID || k == EPI_GELU || k == EPI_GRAD ||
         k == EPI_SWIGLU_BWD || k == EPI_GELU_BWD;
}

template <int BM, int BN, int WM, int WN, int BK, int NST, bool AK, bool BKM>
static hipError_t run_dma(const GemmDesc& g, const EpiArgs& e, hipStream_t s, int nz = 1,
                          const GemmDesc* g2 = nullptr, const EpiArgs* e2 = nullptr) {
  auto kern = gemm_dma_kernel<BM, BN, WM, WN, BK, NST, GEMM_DS, AK, BKM, GEMM_RA, GEMM_RB, KTile<AK, BKM>::MF>;
  const size_t lds_main = (size_t)NST * (BM + BN) * BK * sizeof(bf16_t);
  const size_t lds_epi = (size_t)WM * WN * 32 * (BN / WN + 4) * sizeof(float);
  const size_t lds = lds_main > lds_epi ? lds_main : lds_epi;
  static_assert((size_t)NST * (BM + BN) * BK * 2 <= 160 * 1024, "pipeline exceeds LDS");
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute((const void*)kern,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int nb = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  const int nb2 = g2 ? ((g2->M + BM - 1) / BM) * ((g2->N + BN - 1) / BN) : 0;
  hipLaunchKernelGGL(kern, dim3(nb + nb2, 1, nz), dim3(WM * WN * 64), lds, s, g, e, g2 ? *g2 : g,
                     e2 ? *e2 : e, nb);
  return hipGetLastError();
}

// Splits of K for a GEMM of `tiles` output tiles: none from 3/4 of a wave
// of blocks (one per CU) up, else enough to give the chip about 256 blocks,
// each split at least 8 k-tiles deep, the partials within the workspace.
// Returns 1 for no split.
static int splitk_count(const GemmDesc& g, const EpiArgs& e, long tiles, int bk) {
  if (!g.part || !splitk_kind_ok(e.kind) || tiles > 192) return 1;
  int nz = (int)((256 + tiles - 1) / tiles);
  const int by_k = g.K / (8 * bk);
  if (nz > by_k) nz = by_k;
  const size_t mn = (size_t)g.M * g.N;
  if (mn && (size_t)nz * mn > g.part_elems) nz = (int)(g.part_elems / mn);
  return nz >= 2 ? nz : 1;
}

template <int BM, int BN, int WM, int WN, int BK, int NST, bool AK, bool BKM>
static hipError_t run_dma_split(const GemmDesc& g, const EpiArgs& e, hipStream_t s) {
  const long tiles = (long)((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  int nz = splitk_count(g, e, tiles, BK);
  GemmDesc gs = g;
  gs.ksplit = g.K;
  if (nz == 1) return run_dma<BM, BN, WM, WN, BK, NST, AK, BKM>(gs, e, s, 1);
  // K per split, a multiple of the k-tile, so every split but the last is whole
  gs.ksplit = ((g.K + nz - 1) / nz + BK - 1) / BK * BK;
  nz = (g.K + gs.ksplit - 1) / gs.ksplit;
  EpiArgs ep;
  memset(&ep, 0, sizeof(ep));
  ep.kind = EPI_STORE;
  ep.out = g.part;
  ep.ldo = g.N;
  ep.out_dtype = F32;
  ep.scale = 1.f;
  ep.zstride = (int64_t)g.M * g.N;
  hipError_t err = run_dma<BM, BN, WM, WN, BK, NST, AK, BKM>(gs, ep, s, nz);
  if (err != hipSuccess) return err;
  const int64_t mn = (int64_t)g.M * g.N;
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((mn + 255) / 256)), dim3(256), 0, s,
                     (const float*)g.part, nz, g.M, g.N, e);
  return hipGetLastError();
}

// The direct-to-LDS path copies whole 16-byte chunks with 32-bit buffer
// offsets from the tile origin: every chunk it reads must be either fully
// valid or fully outside (K-major: valid k a multiple of 8; MN-major: the
// M or N extent a multiple of 8), rows 16-byte aligned, and the largest
// offset below 2^31.
static bool dma_operand_ok(const void* p, int64_t ld, bool kmaj, int rows, int kvalid, int R) {
  if (reinterpret_cast<uintptr_t>(p) % 16 != 0 || ld % 8 != 0) return false;
  const int64_t lim = (int64_t)1 << 31;
  if (kmaj) return kvalid % 8 == 0 && ((int64_t)R * ld + kvalid + 64) * 2 < lim;
  return rows % 8 == 0 && ((int64_t)(kvalid + 64) * ld + R) * 2 < lim;
}

template <bool AK, bool BKM>
static hipError_t run_layout(const GemmDesc& g, const EpiArgs& e, int dtype, hipStream_t s,
                             const char** kname) {
  static const char* names[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
  static char buf[5][40];
  int which;
  hipError_t err;
  if (dtype == F32) {
    dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
    hipLaunchKernelGGL((gemm_simt_kernel<AK, BKM>), grid, dim3(256), 0, s, g, e);
    err = hipGetLastError();
    which = 0;
  } else {
    const long big = (long)((g.M + 255) / 256) * ((g.N + 255) / 256);
    // the RoPE and delta epilogues need head-aligned wave tiles of 128 columns
    bool large = big >= 240 || e.kind == EPI_ROPE || e.kind == EPI_STORE_DELTA;
    if (!large && dtype == BF16) {
      // A long reduction over few, nearly full large tiles (the head's data
      // gradient with K = V): large tiles split over K to fill the chip move
      // half the tile bytes per FLOP of 128 x 128 tiles, and each split stays
      // long enough to amortize its partials.
      const int nz = splitk_count(g, e, big, KTile<AK, BKM>::BK);
      large = nz >= 2 && big * nz >= 240 && g.K / nz >= 8192 &&
              (double)g.M * g.N >= 0.9 * (double)big * 65536.0;
    }
    const int R = large ? 256 : 128;
    const bool dma = dma_operand_ok(g.A, g.lda, AK, g.M, g.ka, R) &&
                     dma_operand_ok(g.B, g.ldb, BKM, g.N, g.kb, R) &&
                     (g.K2 <= 0 || (dma_operand_ok(g.A2, g.lda2, AK, g.M, g.K2, R) &&
                                    dma_operand_ok(g.B2, g.ldb2, BKM, g.N, g.K2, R)));
    if (dma) {
      constexpr int BKL = KTile<AK, BKM>::BK, NSTL = KTile<AK, BKM>::NST;
      if (large) { err = run_dma_split<256, 256, GEMM_WM, GEMM_WN, BKL, NSTL, AK, BKM>(g, e, s); which = 3; }
      else { err = run_dma_split<128, 128, 2, 2, BKL, NSTL, AK, BKM>(g, e, s); which = 4; }
    } else if (large) {
      if constexpr (AK && BKM) err = run_mfma<256, 256, 4, 2, AK, BKM>(g, e, s);
      else err = run_mfma<256, 256, 2, 2, AK, BKM>(g, e, s);
      which = 1;
    } else {
      err = run_mfma<128, 128, 2, 2, AK, BKM>(g, e, s);
      which = 2;
    }
  }
  if (kname) {
    if (!names[which]) {
      static const char* base[5] = {"gemm_simt_64x64", "gemm_mfma_256x256", "gemm_mfma_128x128",
                                    "gemm_dma_256x256", "gemm_dma_128x128"};
      snprintf(buf[which], sizeof(buf[which]), "%s_%s", base[which], layout_tag(AK, BKM));
      names[which] = buf[which];
    }
    *kname = names[which];
  }
  return err;
}

// Two GEMMs of one layout in one launch (256 x 256 direct-to-LDS tiles,
// no split K, no second K segment), else one after the other.
template <bool AK, bool BKM>
static hipError_t run_pair_layout(const GemmDesc& g1, const EpiArgs& e1, const GemmDesc& g2,
                                  const EpiArgs& e2, int dtype, hipStream_t s, bool* fused) {
  *fused = false;
  if (dtype != BF16 || g1.K2 != 0 || g2.K2 != 0) return hipSuccess;
  auto ok = [](const GemmDesc& g, const EpiArgs& e) {
    const long tiles = (long)((g.M + 255) / 256) * ((g.N + 255) / 256);
    constexpr int BKL = KTile<AK, BKM>::BK;
    return tiles >= 240 && e.kind != EPI_ROPE && e.kind != EPI_STORE_DELTA && e.kind != EPI_LOGITS &&
           splitk_count(g, e, tiles, BKL) == 1 && dma_operand_ok(g.A, g.lda, AK, g.M, g.ka, 256) &&
           dma_operand_ok(g.B, g.ldb, BKM, g.N, g.kb, 256);
  };
  if (!ok(g1, e1) || !ok(g2, e2)) return hipSuccess;
  constexpr int BKL = KTile<AK, BKM>::BK, NSTL = KTile<AK, BKM>::NST;
  GemmDesc a = g1, b = g2;
  a.ksplit = a.K;
  b.ksplit = b.K;
  *fused = true;
  return run_dma<256, 256, GEMM_WM, GEMM_WN, BKL, NSTL, AK, BKM>(a, e1, s, 1, &b, &e2);
}

hipError_t launch_gemm_pair(const GemmDesc& g1, const EpiArgs& e1, const GemmDesc& g2,
                            const EpiArgs& e2, int dtype, hipStream_t s, bool* fused,
                            const char** kname) {
  *fused = false;
  if (g1.a_kmajor != g2.a_kmajor || g1.b_kmajor != g2.b_kmajor || g1.M <= 0 || g1.N <= 0 ||
      g2.M <= 0 || g2.N <= 0)
    return hipSuccess;
  hipError_t err = hipSuccess;
  if (g1.a_kmajor && g1.b_kmajor) err = run_pair_layout<true, true>(g1, e1, g2, e2, dtype, s, fused);
  else if (g1.a_kmajor) err = run_pair_layout<true, false>(g1, e1, g2, e2, dtype, s, fused);
  else if (!g1.b_kmajor) err = run_pair_layout<false, false>(g1, e1, g2, e2, dtype, s, fused);
  else err = run_pair_layout<false, true>(g1, e1, g2, e2, dtype, s, fused);
  if (*fused && kname) {
    static char buf[4][48];
    const int w = (g1.a_kmajor ? 2 : 0) + (g1.b_kmajor ? 1 : 0);
    snprintf(buf[w], sizeof(buf[w]), "gemm_dma_256x256_%s", layout_tag(g1.a_kmajor, g1.b_kmajor));
    *kname = buf[w];
  }
  return err;
}

hipError_t launch_gemm(const GemmDesc& g, const EpiArgs& e, int dtype, hipStream_t s,
                       const char** kname) {
  if (kname) *kname = "gemm_empty";
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.K2 < 0 || (g.K2 > 0 && (!g.A2 || !g.B2))) return hipErrorInvalidValue;
  if (e.kind == EPI_ROPE && (dtype != BF16 || e.hd > 128 || 128 % e.hd != 0 || !e.pos || !e.rope))
    return hipErrorInvalidValue;
  if (e.kind == EPI_LOGITS && (dtype != BF16 || !e.stats || (e.out_dtype != F32 && e.out_dtype != F16) ||
                              (e.pair && g.M % 2) || (e.zy && !e.lab)))
    return hipErrorInvalidValue;
  if (e.kind == EPI_STORE_DELTA &&
      (dtype != BF16 || !e.delta || !e.aux || e.hd < EW || e.hd > 128 || 128 % e.hd ||
       e.seq < 1 || e.nheads < 1 || e.bias || (int64_t)e.nheads * e.hd != g.N || g.M % e.seq))
    return hipErrorInvalidValue;
  if (g.a_kmajor && g.b_kmajor) return run_layout<true, true>(g, e, dtype, s, kname);
  if (g.a_kmajor && !g.b_kmajor) return run_layout<true, false>(g, e, dtype, s, kname);
  if (!g.a_kmajor && !g.b_kmajor) return run_layout<false, false>(g, e, dtype, s, kname);
  return run_layout<false, true>(g, e, dtype, s, kname);
}

}  // namespace zl
