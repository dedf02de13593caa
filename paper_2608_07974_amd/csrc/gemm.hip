// GEMM kernels for every linear of the chunk map (Eq. (1)) and the frozen
// readout head (Eq. (2)), forward, data-gradient and weight-gradient forms.
//
// bf16: MFMA 32x32x16 (fp32 accumulate), LDS double-buffered tiles staged
// through registers, 16-byte XOR-swizzled LDS rows, 8x8 in-register
// transposes for operands whose contiguous dimension is not K, and an
// XCD-aware tile order so tiles sharing operand panels run on one L2.
// fp32: a plain LDS-tiled SIMT kernel (the fp32 configuration is small).
#include <stdio.h>

#include "common.h"

namespace zl {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

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

__device__ inline float ld_act(const void* p, int dt, size_t i) {
  return dt == BF16 ? bf16_to_f32(((const bf16_t*)p)[i]) : ((const float*)p)[i];
}
__device__ inline void st_act(void* p, int dt, size_t i, float v) {
  if (dt == BF16) ((bf16_t*)p)[i] = f32_to_bf16(v);
  else ((float*)p)[i] = v;
}

__device__ inline void epilogue(const EpiArgs& e, int M, int N, int m, int n, float acc) {
  if (m >= M || n >= N) return;
  const size_t mo = (size_t)m;
  switch (e.kind) {
    case EPI_STORE: {
      float v = acc + (e.bias ? e.bias[n] : 0.f);
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
      float sg = 1.f / (1.f + __expf(-g));
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
      st_act(e.out, e.out_dtype, mo * e.ldo + n, acc);
      break;
  }
}

// ------------------------------------------------------------- tile order
// Grouped (GROUP_M row panels) order, then remapped so that the blocks the
// dispatcher places on one XCD (round-robin over 8) take a contiguous range
// of the grouped order and share A/B panels in that XCD's L2.
__device__ inline void tile_coords(int nbm, int nbn, int& tm, int& tn) {
  const int nb = nbm * nbn;
  int b = blockIdx.x;
  if (nb >= 64) {
    const int per = nb / 8, rem = nb % 8;
    const int x = b % 8, idx = b / 8;
    b = (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + idx;
  }
  const int GROUP_M = 8;
  const int group = b / (GROUP_M * nbn);
  const int first_m = group * GROUP_M;
  const int gsz = min(nbm - first_m, GROUP_M);
  const int in_group = b % (GROUP_M * nbn);
  tm = first_m + in_group % gsz;
  tn = in_group / gsz;
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
  tile_coords(nbm, nbn, tm, tn);
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
#pragma unroll
    for (int s = 0; s < BKT / 16; ++s) {
      const int chunk = 2 * s + (lane >> 5);
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * TM + i * 32 + (lane & 31);
        af[i] = *reinterpret_cast<const bf16x8_t*>(as + row * BKT + ((chunk ^ swz(row)) * 8));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int row = wn * TN + j * 32 + (lane & 31);
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(bs + row * BKT + ((chunk ^ swz(row)) * 8));
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      sa.store(As + (cur ^ 1) * BM * BKT);
      sb.store(Bs + (cur ^ 1) * BN * BKT);
    }
    __syncthreads();
  }

  // Epilogue through LDS, one 32-row block of every wave tile at a time:
  // the accumulators are written with compile-time indices (so they stay in
  // registers), then read back row-contiguously, which coalesces the
  // global stores of the epilogue.
  constexpr int LDW = TN + 4;
  static_assert(WM * WN * 32 * LDW * 4 <= 2 * (BM + BN) * BKT * 2, "epilogue tile exceeds LDS");
  float* ep = reinterpret_cast<float*>(smem) + wave * 32 * LDW;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        ep[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * LDW + j * 32 + (lane & 31)] = acc[i][j][r];
    __syncthreads();
    const int mb = m0 + wm * TM + i * 32, nb = n0 + wn * TN;
    if (e.kind == EPI_ROPE) {
      // wave tiles are head-aligned (nb % hd == 0, TN % hd == 0), so the
      // partner column j +- hd/2 of a head lives in the same staged row
      const int half = e.hd >> 1;
      for (int t = lane; t < 32 * TN; t += 64) {
        const int row = t / TN, col = t % TN;
        const int n = nb + col, m = mb + row;
        float v = ep[row * LDW + col];
        if (n < e.n_rot && m < g.M) {
          const int j = n % e.hd;
          const bool lo = j < half;
          const float pv = ep[row * LDW + (lo ? col + half : col - half)];
          int p = e.pos[m];
          p = p < 0 ? 0 : (p >= e.max_pos ? e.max_pos - 1 : p);
          const float2 cs = e.rope[(int64_t)p * half + (lo ? j : j - half)];
          v = lo ? v * cs.x - pv * cs.y : v * cs.x + pv * cs.y;
        }
        epilogue(e, g.M, g.N, m, n, v);
      }
    } else {
      for (int t = lane; t < 32 * TN; t += 64) {
        const int row = t / TN, col = t % TN;
        epilogue(e, g.M, g.N, mb + row, nb + col, ep[row * LDW + col]);
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------ SIMT (fp32)
template <bool AK, bool BKM>
__global__ void __launch_bounds__(256) gemm_simt_kernel(GemmDesc g, EpiArgs e) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const float* A = reinterpret_cast<const float*>(g.A);
  const float* B = reinterpret_cast<const float*>(g.B);
  float acc[4][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += BK) {
    for (int idx = threadIdx.x; idx < BM * BK; idx += 256) {
      int r, k;
      if (AK) { r = idx / BK; k = idx % BK; } else { r = idx % BM; k = idx / BM; }
      const int gr = m0 + r, gk = k0 + k;
      float v = 0.f;
      if (gr < g.M && gk < g.ka) v = AK ? A[(int64_t)gr * g.lda + gk] : A[(int64_t)gk * g.lda + gr];
      As[k][r] = v;
    }
    for (int idx = threadIdx.x; idx < BN * BK; idx += 256) {
      int r, k;
      if (BKM) { r = idx / BK; k = idx % BK; } else { r = idx % BN; k = idx / BN; }
      const int gr = n0 + r, gk = k0 + k;
      float v = 0.f;
      if (gr < g.N && gk < g.kb) v = BKM ? B[(int64_t)gr * g.ldb + gk] : B[(int64_t)gk * g.ldb + gr];
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
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) epilogue(e, g.M, g.N, m0 + ty * 4 + i, n0 + tx * 4 + j, acc[i][j]);
}

// ------------------------------------------------------------------ launch
template <int BM, int BN, int WM, int WN, bool AK, bool BKM>
static hipError_t run_mfma(const GemmDesc& g, const EpiArgs& e, hipStream_t s) {
  auto kern = gemm_mfma_kernel<BM, BN, WM, WN, AK, BKM>;
  const size_t lds = (size_t)2 * (BM + BN) * BKT * sizeof(bf16_t);
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

template <bool AK, bool BKM>
static hipError_t run_layout(const GemmDesc& g, const EpiArgs& e, int dtype, hipStream_t s,
                             const char** kname) {
  static const char* names[3] = {nullptr, nullptr, nullptr};
  static char buf[3][40];
  int which;
  hipError_t err;
  if (dtype == F32) {
    dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
    hipLaunchKernelGGL((gemm_simt_kernel<AK, BKM>), grid, dim3(256), 0, s, g, e);
    err = hipGetLastError();
    which = 0;
  } else {
    const long big = (long)((g.M + 255) / 256) * ((g.N + 255) / 256);
    // the RoPE epilogue needs head-aligned wave tiles of 128 columns
    if (big >= 240 || e.kind == EPI_ROPE) { err = run_mfma<256, 256, 2, 2, AK, BKM>(g, e, s); which = 1; }
    else { err = run_mfma<128, 128, 2, 2, AK, BKM>(g, e, s); which = 2; }
  }
  if (kname) {
    if (!names[which]) {
      static const char* base[3] = {"gemm_simt_64x64", "gemm_mfma_256x256", "gemm_mfma_128x128"};
      snprintf(buf[which], sizeof(buf[which]), "%s_%s", base[which], layout_tag(AK, BKM));
      names[which] = buf[which];
    }
    *kname = names[which];
  }
  return err;
}

hipError_t launch_gemm(const GemmDesc& g, const EpiArgs& e, int dtype, hipStream_t s,
                       const char** kname) {
  if (kname) *kname = "gemm_empty";
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (e.kind == EPI_ROPE && (dtype != BF16 || e.hd > 128 || 128 % e.hd != 0 || !e.pos || !e.rope))
    return hipErrorInvalidValue;
  if (g.a_kmajor && g.b_kmajor) return run_layout<true, true>(g, e, dtype, s, kname);
  if (g.a_kmajor && !g.b_kmajor) return run_layout<true, false>(g, e, dtype, s, kname);
  if (!g.a_kmajor && !g.b_kmajor) return run_layout<false, false>(g, e, dtype, s, kname);
  return run_layout<false, true>(g, e, dtype, s, kname);
}

}  // namespace zl
