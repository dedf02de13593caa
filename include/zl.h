/*
 * zl.h -- C ABI of the ZeroLock chunk-local update on one MI355X (gfx950).
 *
 * One model chunk (a run of consecutive decoder layers, Eq. (1) of Sec. II.A)
 * is updated from its own local objective:
 *   1. forward h_k = f_k(h_{k-1})                          (Eq. (1); in-stage S2)
 *   2. local objective on the frozen readout head          (Eq. (2)-(5); S3)
 *   3. backward inside the chunk only, input detached      (Remark 1; S3)
 *   4. gradient accumulation over an update window and the
 *      optimizer step (SGD of Eq. (6), or AdamW)           (S3, Sec. III-C)
 * The calls mirror the stage-execution interfaces of Sec. III-B: Input,
 * Forward-and-Output (zl_chunk_forward) and Local Update (zl_local_objective,
 * zl_chunk_backward, zl_optimizer_step), with hidden states as the only
 * exchanged state (Sec. III-A, technique III).
 *
 * Conventions
 *  - Every data pointer is a DEVICE pointer unless stated; `stream` is a
 *    hipStream_t (NULL = the default stream).  All calls are asynchronous on
 *    `stream` and never synchronise the host.
 *  - The caller owns every buffer.  After zl_chunk_create the library
 *    allocates no device memory: all scratch lives in the caller's workspace.
 *  - Arguments are checked on the host before any launch; a call that fails
 *    that check returns a negative zl_status and launches nothing, leaving
 *    parameters, optimizer state and call-order state unchanged.
 *    zl_last_error() then holds a human-readable reason (thread-local).
 *  - Device faults surface at the caller's next synchronisation.
 *  - No C++ exception crosses this interface.
 *  - A chunk handle must not be used from two threads at once, and calls on
 *    one handle must be issued on streams ordered with each other.
 */
#ifndef ZL_H
#define ZL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum zl_status {
  ZL_OK = 0,
  ZL_ERR_INVALID_ARG = -1, /* bad pointer, size, shape or config value       */
  ZL_ERR_UNSUPPORTED = -2, /* valid but not implemented (e.g. head_dim form) */
  ZL_ERR_HIP = -3,         /* a HIP runtime call or kernel launch failed      */
  ZL_ERR_STATE = -4,       /* call out of order (objective before forward...) */
  ZL_ERR_WORKSPACE = -5    /* workspace missing, misaligned or too small      */
} zl_status;

enum { ZL_ARCH_LLAMA = 0, /* RMSNorm, RoPE (rotate-half), GQA, SwiGLU        */
       ZL_ARCH_GPT2 = 1   /* LayerNorm, biases, GELU(tanh), no RoPE          */ };
enum { ZL_F32 = 0,        /* fp32 everywhere                                 */
       ZL_BF16 = 1        /* bf16 weights/activations, fp32 accumulate, fp32
                             master weights, gradients and optimizer state   */ };
enum { ZL_KL_REVERSE = 0, /* consistency KL(p_k || p_{k-1}), Eq. (5)         */
       ZL_KL_FORWARD = 1  /* consistency KL(p_{k-1} || p_k)                  */ };
enum { ZL_ADAMW = 0, ZL_SGD = 1 };

/* Chunk configuration, validated by zl_param_layout / zl_workspace_size /
 * zl_chunk_create.  alpha weights the task term against the consistency term
 * (Eq. (3), alpha in (0, 1]); alpha == 1 skips the readout of h_{k-1}.
 * max_batch * max_seq bounds the tokens of one micro-batch. */
typedef struct zl_config {
  int arch;          /* ZL_ARCH_*                                            */
  int n_layers;      /* layers in the chunk, >= 1                            */
  int d_model;       /* multiple of 64                                       */
  int n_heads;       /* query heads                                          */
  int n_kv_heads;    /* key/value heads; n_heads % n_kv_heads == 0           */
  int head_dim;      /* even, multiple of 8                                  */
  int d_ff;          /* MLP width, multiple of 64                            */
  int vocab;         /* head rows V (any value >= 2)                         */
  float norm_eps;    /* RMSNorm / LayerNorm epsilon                          */
  float rope_theta;  /* RoPE base (llama only)                               */
  int dtype;         /* ZL_F32 or ZL_BF16                                    */
  float alpha;       /* Eq. (3) weight, (0, 1]                               */
  int consis;        /* ZL_KL_REVERSE or ZL_KL_FORWARD                       */
  int optimizer;     /* ZL_ADAMW or ZL_SGD                                   */
  float lr, beta1, beta2, eps, weight_decay; /* AdamW (SGD uses lr only)     */
  int max_batch;     /* >= 1                                                 */
  int max_seq;       /* >= 1; also the RoPE position bound                   */
  int adapter_rank;  /* readout adapter width r (Sec. III-B, Local Update
                        interface (b)), 0 = static head only; else a multiple
                        of 16: h_out is read out as h' = h + gelu(h W1^T) W2^T
                        (W1 [r, d], W2 [d, r], GELU tanh form) through the
                        frozen norm and head; the consistency target from
                        h_in uses the static head.  W1 and W2 are trainable
                        (W2 = 0 makes the adapter the identity).             */
  int lora_rank;     /* LoRA rank r (Sec. II.A: Delta w_l = B_l A_l on the
                        frozen w_l, trained by Eq. (6)); 0 = the whole chunk
                        is trainable.  Else 1..256: every linear (llama wq wk
                        wv wo wg wu wd, gpt2 wqkv wo wfc wproj) computes
                        y = x W^T (+ b) + s (x A^T) B^T with s = lora_alpha /
                        r; W, norms and biases are frozen and read from
                        base_master / base_shadow; the trainable set is the
                        factors A [r, in], B [out, r] (and the readout
                        adapter).  The factors are stored r8 = r rounded up
                        to a multiple of 8 wide (A [r8, in], B [out, r8], the
                        shapes zl_param_layout reports); rows r.. of A and
                        columns r.. of B are padding, which zl_refresh_shadow
                        sets to zero and which then stays zero: its gradient
                        is exactly zero, so neither SGD nor AdamW moves it,
                        and the result is that of rank r.                  */
  float lora_alpha;  /* s = lora_alpha / lora_rank; > 0 when lora_rank > 0  */
} zl_config;

/* One trainable tensor inside the flat parameter buffers (zl_param_layout).
 * Per layer the order is
 *   llama: ln1_w[d], wq[hq*hd,d], wk[hkv*hd,d], wv[hkv*hd,d], wo[d,hq*hd],
 *          ln2_w[d], wg[ff,d], wu[ff,d], wd[d,ff]
 *   gpt2:  ln1_w[d], ln1_b[d], wqkv[(hq+2hkv)*hd,d], bqkv[..], wo[d,hq*hd],
 *          bo[d], ln2_w[d], ln2_b[d], wfc[ff,d], bfc[ff], wproj[d,ff], bproj[d]
 * With lora_rank r > 0 these are the frozen base tensors, laid out in the
 * base buffers as zl_param_layout of the same config with lora_rank = 0 and
 * adapter_rank = 0, and the trainable tensors are, per layer, the factors
 *   llama: wq_la[r,d], wk_la[r,d], wv_la[r,d], wq_lb[hq*hd,r],
 *          wk_lb[hkv*hd,r], wv_lb[hkv*hd,r], wo_la[r,hq*hd], wo_lb[d,r],
 *          wg_la[r,d], wu_la[r,d], wg_lb[ff,r], wu_lb[ff,r], wd_la[r,ff],
 *          wd_lb[d,r]
 *   gpt2:  wqkv_la[r,d], wqkv_lb[(hq+2hkv)*hd,r], wo_la, wo_lb, wfc_la,
 *          wfc_lb, wproj_la, wproj_lb
 * With adapter_rank r > 0 two more tensors follow the last layer, listed
 * with layer index n_layers: ad_w1[r,d], ad_w2[d,r].
 * Linear weights are row-major [out, in] (y = x W^T, as in Eq. (2)).  Offsets
 * are in elements and multiples of 64; wq/wk/wv (and wg/wu) are adjacent,
 * and so are their LoRA A factors and their B factors. */
typedef struct zl_tensor_desc {
  char name[16];
  int layer;
  int ndim;          /* 1 or 2                                               */
  int64_t shape[2];  /* shape[1] = 1 when ndim == 1                          */
  size_t offset;     /* element offset into master/shadow/grad/adam_m/adam_v */
  size_t numel;
} zl_tensor_desc;

/* Caller-owned buffers, all device memory, all n_params elements long unless
 * stated.  The library reads and writes them in place. */
typedef struct zl_buffers {
  float* master;            /* fp32 trainable parameters (read, updated)     */
  void* shadow;             /* bf16 copy of master (ZL_BF16), NULL for F32;
                               written by zl_refresh_shadow / optimizer step */
  float* grad;              /* fp32 gradient accumulator                     */
  float* adam_m;            /* fp32 first moment (ZL_ADAMW; NULL for SGD)    */
  float* adam_v;            /* fp32 second moment (ZL_ADAMW; NULL for SGD)   */
  const void* head_w;       /* frozen W_lm [vocab, d_model], dtype of config */
  const float* head_norm_w; /* frozen final-norm weight [d_model]            */
  const float* head_norm_b; /* frozen final-norm bias [d_model] (gpt2), else
                               NULL                                          */
  const float* base_master; /* lora_rank > 0: the frozen base tensors (fp32),
                               n_base elements laid out as zl_param_layout of
                               the config with lora_rank = adapter_rank = 0;
                               else NULL                                     */
  void* base_shadow;        /* lora_rank > 0 and ZL_BF16: bf16 copy of
                               base_master, written by zl_refresh_shadow;
                               else NULL                                     */
} zl_buffers;

typedef struct zl_chunk zl_chunk;

/* Parameter layout (host only).  Writes the total element count to *n_params
 * and, when descs != NULL, up to *n_descs descriptors (on return *n_descs is
 * the number of tensors).  Pass descs == NULL to query the count. */
zl_status zl_param_layout(const zl_config* cfg, size_t* n_params,
                          zl_tensor_desc* descs, int* n_descs);

/* Bytes of device workspace zl_chunk_create needs for cfg (host only). */
zl_status zl_workspace_size(const zl_config* cfg, size_t* bytes);

/* Creates a handle over caller-owned buffers and a workspace of at least
 * zl_workspace_size bytes, 256-byte aligned.  Launches one kernel on the
 * default stream that fills the rotary table inside the workspace, and
 * waits for it.  The handle keeps the pointers only; optimizer step count
 * starts at 0.  *out is set to NULL on failure. */
zl_status zl_chunk_create(const zl_config* cfg, const zl_buffers* bufs,
                          void* workspace, size_t ws_bytes, zl_chunk** out);
void zl_chunk_destroy(zl_chunk* chunk);

/* Writes the bf16 shadow from the fp32 master (round to nearest even), and
 * with lora_rank > 0 also base_shadow from base_master.  With a lora_rank
 * that is not a multiple of 8 it first zeroes the padding of the stored
 * factors in master (see zl_config.lora_rank).  Call after initialising or
 * loading master (or the base), in either dtype. */
zl_status zl_refresh_shadow(zl_chunk* chunk, void* stream);

/* Forward-and-Output (Sec. III-B; Eq. (1)).  h_in and h_out are [B, S, d]
 * row-major in the config dtype.  seq_lens [B] (NULL = all S) right-pads
 * each sequence: keys at j >= seq_lens[b] are masked, 0 <= seq_lens[b] <= S.
 * pos_ids [B, S] (NULL = 0..S-1) feed RoPE; values are clamped to
 * [0, max_seq).  h_in is never written; its values, seq_lens and pos_ids
 * are copied into the workspace on `stream`, so the caller may reuse them
 * once the stream has passed this call.  h_out is complete when the stream
 * reaches the end of this call -- the early-forwarding point of Sec. III-B
 * (downstream work may start there, before the local update).  Saves the
 * activations the backward needs.  1 <= B <= max_batch, 1 <= S <= max_seq. */
zl_status zl_chunk_forward(zl_chunk* chunk, const void* h_in,
                           const int32_t* seq_lens, const int32_t* pos_ids,
                           int B, int S, void* h_out, void* stream);

/* Local objective (Eq. (2)-(5)): readout z = Norm(h_out) W_lm^T of the
 * forward's output and, when alpha < 1, of its input (stop-gradient target,
 * recomputed here because stages exchange hidden states only), then
 *   L = alpha * mean_Omega CE + (1 - alpha) * mean_Omega KL
 * over the labelled set Omega = {labels != -100}; labels [B, S] int32 with
 * values in [0, vocab) or -100.  Writes L to *loss_out (one fp32, device)
 * and keeps dL/dh_out in the workspace.  |Omega| = 0 gives L = 0 and a zero
 * gradient.  Labels outside [0, vocab) other than -100 are treated as -100.
 * Requires a preceding zl_chunk_forward (else ZL_ERR_STATE). */
zl_status zl_local_objective(zl_chunk* chunk, const int32_t* labels,
                             float* loss_out, void* stream);

/* Backward inside the chunk (Remark 1): gradients of every trainable tensor
 * of the chunk, scaled by grad_scale, written (accumulate == 0) or added
 * (accumulate != 0) into grad.  No gradient to h_in is formed.  The first
 * backward after create or after an optimizer step always writes, whatever
 * `accumulate` says, so a window starts from zero without a clearing pass
 * (S3: gradients accumulate over the micro-batches of one update window).
 * Requires a preceding zl_local_objective (else ZL_ERR_STATE). */
zl_status zl_chunk_backward(zl_chunk* chunk, float grad_scale, int accumulate,
                            void* stream);

/* Optimizer step over all trainable tensors: AdamW with bias correction and
 * decoupled weight decay, or SGD (Eq. (6)).  Increments the step count
 * (first step is t = 1), refreshes the bf16 shadow, and marks the gradient
 * consumed (its contents are left as they are).  Requires at least one
 * zl_chunk_backward since the last step (else ZL_ERR_STATE). */
zl_status zl_optimizer_step(zl_chunk* chunk, void* stream);

/* forward -> objective -> backward(1, 0) -> optimizer step, on one stream:
 * one whole chunk-local update of one micro-batch window (m = 1). */
zl_status zl_chunk_update(zl_chunk* chunk, const void* h_in,
                          const int32_t* seq_lens, const int32_t* pos_ids,
                          const int32_t* labels, int B, int S, void* h_out,
                          float* loss_out, void* stream);

/* Optimizer step count, for checkpoint and resume of a stage (Sec. III-B,
 * failure recovery: parameters, optimizer state, progress). */
zl_status zl_get_step(const zl_chunk* chunk, int64_t* step);
zl_status zl_set_step(zl_chunk* chunk, int64_t step);

/* The configuration and buffer pointers the chunk was created with (copies;
 * the chunk keeps its own).  ZL_ERR_INVALID_ARG on NULL arguments. */
zl_status zl_chunk_get_config(const zl_chunk* chunk, zl_config* out);
zl_status zl_chunk_get_buffers(const zl_chunk* chunk, zl_buffers* out);
/* Number of trainable parameters (length of master / grad / adam_m / adam_v). */
zl_status zl_chunk_num_params(const zl_chunk* chunk, size_t* n_params);

const char* zl_status_string(zl_status s);
const char* zl_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ZL_H */
