/*
 * zl_inspect.h -- read-only views into a chunk's workspace and direct calls
 * of single kernels, for verification against an independent reference.
 * Not needed to run an update; see zl.h for the update interface.
 */
#ifndef ZL_INSPECT_H
#define ZL_INSPECT_H

#include "zl.h"

#ifdef __cplusplus
extern "C" {
#endif

/* A device matrix [rows, cols] with row stride ld (elements), dtype ZL_F32 or
 * ZL_BF16.  Valid until the next call that rewrites the workspace. */
typedef struct zl_view {
  const void* ptr;
  int64_t rows, cols, ld;
  int dtype;
} zl_view;

/* View of an intermediate kept by the last zl_chunk_forward /
 * zl_local_objective (T = B * S tokens of that forward):
 *   "x"        layer in [0, L]: fp32 residual stream entering layer `layer`
 *              ("x", L) is h_out in fp32                           [T, d]
 *   "n1","n2"  normalised inputs of attention / MLP                [T, d]
 *   "qkv"      q|k|v projections (q, k after RoPE)                 [T, (hq+2hkv)*hd]
 *   "o"        attention output before the output projection      [T, hq*hd]
 *   "lse"      attention log-sum-exp, fp32                         [B*hq, S]
 *   "x2"       fp32 residual stream after attention                [T, d]
 *   "up"       llama: gate|up pre-activations [T, 2ff]; gpt2: fc pre-activation [T, ff]
 *   "act"      MLP activation entering the down projection        [T, ff]
 *   "rstd1","rstd2"  fp32 inverse norm scales                      [T, 1]
 *   "dh_out"   fp32 dL/dh_out after zl_local_objective            [T, d]
 *   "row_loss" fp32 per-token loss terms (0 outside Omega)        [T, 1]
 *   "n_omega"  fp32 |Omega|                                        [1, 1]
 * After zl_local_objective, of the head's last row block (R = min(T, 4096)
 * rows, or fewer when T is not a multiple of R; Vp = vocab rounded up to 8):
 *   "dz"       dL/dz in the activation dtype                       [R, Vp]
 *   "dnf"      fp32 dL/dz W_lm, the head's data gradient before its
 *              norm backward                                       [R, d]
 * After zl_chunk_backward, the operands of layer 0's weight gradients (the
 * backward's scratch, left by the last layer it processed), activation dtype:
 *   "dxa"      dL/d(layer output), the down projection's dy        [T, d]
 *   "dup"      dL/d(gate|up) (fc) pre-activations                   [T, 2ff or ff]
 *   "dxb"      dL/d(x2), the output projection's dy                [T, d]
 *   "do"       dL/d(attention output)                              [T, hq*hd]
 *   "dqkv"     dL/d(q|k|v projections), the rotation undone        [T, (hq+2hkv)*hd]
 *   "dn"       fp32 dL/d(n1) = dqkv W_qkv, the norm-1 backward's input [T, d]
 *              (layer 0 of a LoRA chunk skips it: then left by layer 1) 
 * Pointers are device pointers into the workspace; do not write them. */
zl_status zl_inspect(const zl_chunk* chunk, const char* name, int layer, zl_view* out);

/* C[m, n] = sum_k A(m, k) B(n, k) + sum_{k < K2} A2(m, k) B2(n, k), fp32
 * output with row stride ldc, where A(m, k) = a_kmajor ? A[m*lda + k] :
 * A[k*lda + m] and likewise for B, A2 (lda2) and B2 (ldb2) in the layouts of
 * A and B; the GEMM kernel used for every linear of the chunk (Eq. (1)), the
 * second segment carrying the LoRA term (K2 = 0: none, A2 and B2 unused),
 * and the head (Eq. (2)).  dtype ZL_BF16 (MFMA) or ZL_F32 (SIMT).
 * workspace (device, workspace_elems floats, or NULL): lets a bf16 GEMM
 * whose output has too few tiles to fill the GPU split K into fp32 partials
 * there, summed in a fixed order (the chunk's own GEMMs use a region of its
 * workspace for this); its contents are scratch. */
zl_status zl_kernel_gemm(int M, int N, int K, const void* A, int64_t lda, int a_kmajor,
                         const void* B, int64_t ldb, int b_kmajor, int K2, const void* A2,
                         int64_t lda2, const void* B2, int64_t ldb2, float* C, int64_t ldc,
                         float* workspace, size_t workspace_elems, int dtype, void* stream);

/* Causal GQA attention forward (backward = 0: o, lse) or backward
 * (backward = 1: dq, dk, dv and delta from q, k, v, o, lse, dout), the
 * kernels used inside each decoder layer.  q, k, v, dq, dk, dv share the row
 * stride ld_qkv; o and dout have row stride Hq * hd; lse, delta [B, Hq, S]. */
zl_status zl_kernel_attention(int B, int S, int Hq, int Hkv, int hd, const void* q,
                              const void* k, const void* v, int64_t ld_qkv,
                              const int32_t* seq_lens, void* o, float* lse, const void* dout,
                              void* dq, void* dk, void* dv, float* delta, int dtype,
                              int backward, void* stream);

/* The backward of zl_kernel_attention (backward = 1) for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): no delta argument; the softmax-backward
 * row term delta = rowsum(dout * o), B * Hq * S floats, is kept in a device
 * array of the library of at most 2^20 floats (4 MiB), one per GPU, held
 * until the process ends.  Larger B * Hq * S returns ZL_ERR_UNSUPPORTED
 * before any launch.  The call allocates nothing.  Calls on one GPU share
 * that array: calls that overlap on one GPU (different streams, or threads
 * without ordering) race.  dq, dk, dv are bit-identical to those of
 * zl_kernel_attention with a caller delta buffer. */
zl_status zl_kernel_attention_bwd_noalloc(int B, int S, int Hq, int Hkv, int hd, const void* q,
                                          const void* k, const void* v, int64_t ld_qkv,
                                          const int32_t* seq_lens, const void* o, const float* lse,
                                          const void* dout, void* dq, void* dk, void* dv, int dtype,
                                          void* stream);

/* Per-kernel timing of the chunk's own launches.  zl_profile_begin creates
 * `capacity` pairs of HIP events (host resources, no device memory) and,
 * until zl_profile_end, records one pair on the launch stream around each
 * kernel launch of zl_chunk_forward / zl_local_objective / zl_chunk_backward
 * / zl_optimizer_step (launches beyond capacity are not timed).
 * zl_profile_end waits for the recorded events and writes, per kernel name,
 * the number of launches, the summed duration and the summed algorithmic
 * work (FLOPs for GEMM and attention: 2*M*N*K and the causal pair count;
 * bytes for the streaming kernels: each operand read or written once).
 * *n on input is the capacity of `out`, on output the number of entries. */
typedef struct zl_profile_entry {
  char name[48];
  int64_t launches;
  double total_ms;
  double flops;
  double bytes;
} zl_profile_entry;

zl_status zl_profile_begin(zl_chunk* chunk, int capacity);
zl_status zl_profile_end(zl_chunk* chunk, zl_profile_entry* out, int* n);

/* Properties of HIP device `device` that throughput figures are priced
 * against: compute-unit count, peak shader clock (kHz) and the gfx
 * architecture name (NUL-terminated, truncated to arch_len - 1 bytes).
 * Any output pointer may be NULL.  ZL_ERR_HIP if the device query fails. */
zl_status zl_device_info(int device, int* cu_count, int* clock_khz, char* arch, int arch_len);

#ifdef __cplusplus
}
#endif
#endif /* ZL_INSPECT_H */
