// Internal declarations shared by the HIP kernels and the C-ABI host code.
// Nothing here is part of the public interface in include/zl.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace zl {

// ------------------------------------------------------------------ types
typedef uint16_t bf16_t;  // storage type of bf16 values

// F16 only stores the bf16 path's logit cache (values of a few tens, where
// fp16 keeps 3 more mantissa bits than bf16).
enum DType { F32 = 0, BF16 = 1, F16 = 2 };

// Round to nearest even; finite values beyond the fp16 range saturate at
// +-65504 instead of becoming infinite (dL/dz of such a row is then inexact;
// the loss, taken from fp32 statistics, is not), NaN stays NaN.
__device__ inline uint16_t f32_to_f16(float f) {
  f = f > 65504.f ? 65504.f : (f < -65504.f ? -65504.f : f);
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}
__device__ inline float f16_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }

__host__ __device__ inline float bf16_to_f32(bf16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  __builtin_memcpy(&f, &u, 4);
  return f;
}

// Round to nearest, ties to even; NaN stays NaN.
__host__ __device__ inline bf16_t f32_to_bf16(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static inline float load(const float* p, size_t i) { return p[i]; }
  __device__ static inline void store(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16_t> {
  __device__ static inline float load(const bf16_t* p, size_t i) { return bf16_to_f32(p[i]); }
  __device__ static inline void store(bf16_t* p, size_t i, float v) { p[i] = f32_to_bf16(v); }
};

// ------------------------------------------------------------------- GEMM
// C[m, n] = sum_k A(m, k) * B(n, k) with
//   A(m, k) = a_kmajor ? A[m * lda + k] : A[k * lda + m]
//   B(n, k) = b_kmajor ? B[n * ldb + k] : B[k * ldb + n]
// Elements of A with k >= ka and of B with k >= kb read as zero (ragged K).
// Optional second K segment (K2 > 0): C[m, n] += sum_{k < K2} A2(m, k) B2(n, k)
// with A2, B2 in the layouts of A and B (row strides lda2, ldb2); it carries
// a low-rank term into the same accumulators.
// Contiguous dimensions must be multiples of 8 elements and 16-byte aligned.
struct GemmDesc {
  int M, N, K;
  int ka, kb;
  const void* A;
  int64_t lda;
  bool a_kmajor;
  const void* B;
  int64_t ldb;
  bool b_kmajor;
  int K2;
  const void* A2;
  int64_t lda2;
  const void* B2;
  int64_t ldb2;
  // Split-K workspace (bf16 direct-to-LDS path): with part != nullptr a GEMM
  // whose output has too few tiles to fill the chip may split K over the
  // grid's z dimension into fp32 partials [splits][M][N] (at most part_elems
  // floats), summed in split order by a second kernel that applies the
  // epilogue.  ksplit (K elements per split) is set by launch_gemm.
  float* part;
  size_t part_elems;
  int ksplit;
};

enum EpiKind {
  EPI_STORE = 0,       // out[m, n] = acc (+ bias[n]), out dtype = out_dtype
  EPI_RESID = 1,       // out32[m, n] = resid32[m, n] + acc (+ bias[n])
  EPI_GELU = 2,        // h[m, n] = acc + bias[n]; out[m, n] = gelu(h)  (act dtype)
  EPI_GRAD = 3,        // out32[m, n] = (accumulate ? out32 : 0) + scale * acc
  EPI_SWIGLU_BWD = 4,  // da = acc; g = aux[m, n], u = aux[m, n + ff];
                       // out[m, n] = da * u * silu'(g); out[m, n + ff] = da * silu(g)
  EPI_GELU_BWD = 5,    // out[m, n] = acc * gelu'(aux[m, n])
  EPI_ROPE = 6,        // EPI_STORE after rotating column pairs (j, j + hd/2) of
                       // every head in cols [0, n_rot) by pos[m] (rotate-half RoPE)
  EPI_LOGITS = 7,      // fp32 store, plus per row m and 64-column block cb the
                       // softmax partials stats[m * ldst + cb] = (max x,
                       // sum exp(x - max), sum exp(x - max) (x - x'), 0) over
                       // the block's columns < N, x' = row m ^ 1 (pair != 0)
                       // else 0.  MFMA (bf16) paths only.
  EPI_STORE_DELTA = 8, // EPI_STORE (act dtype) of dO, plus the attention
                       // backward's delta[(b * nheads + h) * seq + s] = sum over
                       // head h's hd columns of dO (as stored) * aux, aux = O,
                       // row m = b * seq + s.  MFMA (bf16) paths only.
};

struct EpiArgs {
  EpiKind kind;
  void* out;            // output base
  int64_t ldo;
  int out_dtype;        // F32 / BF16 for EPI_STORE, act dtype for GELU/bwd kinds
  const float* bias;    // [N] or nullptr
  const float* resid;   // EPI_RESID
  int64_t ldr;
  void* out2;           // EPI_GELU: pre-activation store (act dtype)
  int64_t ldo2;
  const void* aux;      // EPI_SWIGLU_BWD / EPI_GELU_BWD input (act dtype)
  int64_t ldaux;
  int ff;               // EPI_SWIGLU_BWD column offset of u / du
  float scale;          // EPI_GRAD, EPI_STORE (out = scale * acc + bias)
  int accumulate;       // EPI_GRAD
  float* delta;         // EPI_STORE_DELTA (also uses aux, ldaux, hd)
  int seq, nheads;
  float4* stats;        // EPI_LOGITS
  int64_t ldst;
  int pair;
  const int32_t* lab;   // EPI_LOGITS (optional): label of each token; the
  float* zy;            //   fp32 logit of the label, z[token, lab], goes to zy
  const int32_t* pos;   // EPI_ROPE: position of row m
  const float2* rope;   // EPI_ROPE: (cos, sin) table [max_pos, hd/2]
  int max_pos, hd, n_rot;
  int64_t zstride;      // split-K partials: raw fp32 store to out + z * zstride (set by launch_gemm)
};

// *kname (optional) receives a static name of the kernel instantiation used.
// EPI_ROPE is supported by the bf16 MFMA path only (hd <= 128).
hipError_t launch_gemm(const GemmDesc& g, const EpiArgs& e, int dtype, hipStream_t s,
                       const char** kname = nullptr);
// Two independent GEMMs in one launch when both take the 256 x 256
// direct-to-LDS path in the same layout (per-element epilogues, no split K
// or second segment): *fused = true.  Otherwise nothing is launched and
// *fused = false (the caller runs launch_gemm on each).
hipError_t launch_gemm_pair(const GemmDesc& g1, const EpiArgs& e1, const GemmDesc& g2,
                            const EpiArgs& e2, int dtype, hipStream_t s, bool* fused,
                            const char** kname = nullptr);

// --------------------------------------------------------------- row ops
// Norm forward over rows: y = norm(x) * w (+ b).  x fp32 [T, d] (row stride
// ldx); y in act dtype.  Writes rstd [T] (and mean [T] for LayerNorm).
hipError_t launch_norm_fwd(bool layernorm, const float* x, int64_t ldx, const float* w,
                           const float* b, void* y, int64_t ldy, int ydtype, float* mean,
                           float* rstd, int T, int d, float eps, hipStream_t s);
// Same, but rows of x are taken from x_rows[r] = x + src_row(r) * ldx where
// row r of the output is interleaved: output row 2i from xa row i, 2i+1 from
// xb row i (xb may be nullptr: then output row i from xa row i).
hipError_t launch_head_norm(bool layernorm, const float* xa, const float* xb, int64_t ldx,
                            int row0, int rows, const float* w, const float* b, void* y,
                            int ydtype, float* mean, float* rstd, int d, float eps,
                            hipStream_t s);
// Norm backward: dx = dres + norm_bwd(dy) (dres may be nullptr; dx may alias
// dres); also dx_act = act-dtype copy of dx when non-null.  Per-block
// partial sums of dy*xhat (and dy) go to part_w/part_b [nblk, d].  When dx
// is nullptr only the partials are formed.  Returns nblk via *nblk_out.
hipError_t launch_norm_bwd(bool layernorm, const float* dy, const float* x, const float* w,
                           const float* mean, const float* rstd, const float* dres,
                           float* dx, void* dx_act, int act_dtype, float* part_w,
                           float* part_b, int T, int d, hipStream_t s, int* nblk_out);
int norm_bwd_blocks(int T);
// Head-norm backward for a row block: dh[row0 + i] = norm_bwd(dy[i]) (head
// frozen, no weight gradient).  Also writes an act copy.
hipError_t launch_head_norm_bwd(bool layernorm, const float* dy, int64_t lddy, const float* x,
                                const float* w, const float* mean, const float* rstd,
                                int rstd_stride, float* dx, void* dx_act, int act_dtype,
                                int row0, int rows, int d, hipStream_t s);
// out[j] = (accumulate ? out[j] : 0) + scale * sum_b part[b, j]; part is
// scratch (a first stage may overwrite some of its rows).
hipError_t launch_reduce_rows(float* part, int nblk, int d, float* out, float scale,
                              int accumulate, hipStream_t s);
// Column sums of an act-dtype matrix [T, n] into partials [nblk, n].
hipError_t launch_colsum_partial(const void* x, int64_t ldx, int dtype, int T, int n,
                                 float* part, int* nblk_out, hipStream_t s);
int colsum_blocks(int T);

// ------------------------------------------------------------ elementwise
hipError_t launch_cast(const void* src, int sdtype, void* dst, int ddtype, size_t n,
                       hipStream_t s);
hipError_t launch_copy_i32(const int32_t* src, int32_t* dst, int n, int fill_default,
                           int mode, int S, hipStream_t s);
hipError_t launch_rope_table(float2* table, int max_pos, int half, double theta,
                             hipStream_t s);
// In-place rotary on the q and k column blocks of qkv [T, ld] (cols
// [0, (hq + hkv) * hd)), forward (sign = +1) or transpose (sign = -1).
hipError_t launch_rope(void* qkv, int64_t ld, int dtype, const int32_t* pos, const float2* table,
                       int max_pos, int T, int nheads_qk, int hd, int sign, hipStream_t s);
// Block-diagonal [rows, nblk * r] (act dtype, row stride nblk * r) from the
// stacked blocks src [rows, r]: rows [0, b1) form block 0, [b1, b2) block 1,
// [b2, rows) block 2 (nblk <= 3); row n of block j keeps src row n in
// columns j r .. j r + r - 1 and zeros elsewhere.
hipError_t launch_blockdiag(const void* src, void* dst, int dtype, int rows, int r, int nblk,
                            int b1, int b2, hipStream_t s);
hipError_t launch_swiglu_fwd(const void* gu, int64_t ldgu, void* a, int64_t lda, int dtype,
                             int T, int ff, hipStream_t s);

// -------------------------------------------------------------- attention
struct AttnDesc {
  int B, S, Hq, Hkv, hd;
  const void* q; const void* k; const void* v;  // [B*S, ld] with head h at cols h*hd
  int64_t ldq, ldk, ldv;
  void* o; int64_t ldo;                          // [B*S, ldo]
  float* lse;                                    // [B, Hq, S]
  const int32_t* seq_lens;                       // [B]
  // backward
  const void* dout; int64_t lddo;
  float* delta;                                  // [B, Hq, S]
  int delta_ready;                               // delta already formed (skip its kernel)
  void* dq; void* dk; void* dv; int64_t lddq, lddk, lddv;
  float scale;
  // optional inverse RoPE of dq / dk in the backward (rope != nullptr)
  const int32_t* pos; const float2* rope; int max_pos;
};
hipError_t launch_attn_fwd(const AttnDesc& a, int dtype, hipStream_t s);
// *rope_fused reports whether dq / dk already carry the inverse rotation.
hipError_t launch_attn_bwd(const AttnDesc& a, int dtype, hipStream_t s, bool* rope_fused);

// -------------------------------------------------------------- objective
struct ObjDesc {
  const void* zc;       // logits cache [rows_stacked, ldz]; row 2i = z, 2i+1 = z' (stacked)
  int64_t ldz;
  int z_dtype;          // F32, or F16 (with stats and zy)
  const float* zy;      // optional fp32 logit of each row's label (used for the loss)
  int stacked;          // 2 when z' rows are interleaved, else 1
  const int32_t* labels;  // [rows] for this row block
  int rows, V, Vpad;
  float alpha;
  int consis;
  const float* n_omega;   // device scalar |Omega|
  void* dz; int64_t lddz; int dz_dtype;  // [rows, Vpad]; pad columns zeroed
  float* row_loss;        // [rows]
  const float4* stats;    // optional EPI_LOGITS partials of zc's rows (row stride ldst,
  int64_t ldst;           // nst 64-column blocks): replace the statistics pass
  int nst;
};
hipError_t launch_count_omega(const int32_t* labels, int T, int V, float* n_omega,
                              hipStream_t s);
hipError_t launch_objective_rows(const ObjDesc& o, hipStream_t s);
// loss = sum(row_loss[0..T)) / max(n_omega, 1) with n_omega = 0 -> 0
hipError_t launch_loss_reduce(const float* row_loss, int T, const float* n_omega, float* loss,
                              hipStream_t s);

// -------------------------------------------------------------- optimizer
struct OptDesc {
  float* master; bf16_t* shadow; const float* grad; float* m; float* v;
  size_t n;
  int optimizer;
  float lr, beta1, beta2, eps, wd;
  float bc1, bc2;  // 1 - beta^t
};
hipError_t launch_optimizer(const OptDesc& o, hipStream_t s);
hipError_t launch_shadow(const float* master, bf16_t* shadow, size_t n, hipStream_t s);
// Zeroes rows [r0, r1) x columns [c0, c1) of a row-major fp32 matrix with row
// stride ld.
hipError_t launch_zero_block(float* p, int64_t ld, int64_t r0, int64_t r1, int64_t c0, int64_t c1,
                             hipStream_t s);

}  // namespace zl
