/* ZeroLock single-GPU runtime: a pipeline of chunks with early forwarding,
 * and per-chunk checkpoint / resume.
 *
 * Pipeline (Sec. III-B, inter-stage runtime and in-stage execution; Fig. 1(b)).
 * K chunks run as stages 0 .. K-1, stage k on its own HIP stream.  Each
 * micro-batch passes through every stage as S1 (take the entry from the
 * stage's input buffer) -> S2 (chunk forward, output entry written, marked
 * ready) -> S3 (local objective, backward accumulating into the update
 * window, optimizer step after the window's last micro-batch).  Stage k+1's
 * S2 waits only for the readiness event of its own entry, so it overlaps
 * stage k's S3 (early forwarding: downstream work starts right after the
 * upstream forward, never waiting for the upstream backward).
 *
 * Entries.  Between stage k-1 and stage k (and before stage 0, and after
 * stage K-1) sits a ring of `depth` entries; `depth` is the in-flight depth:
 * at most `depth` micro-batches occupy a stage boundary.  An entry holds a
 * micro-batch's hidden state [B, S, d_model] and its metadata (labels,
 * position ids, sequence lengths), and binds two events: ready (written)
 * and free (its reading stage's backward, the last use of the input hidden
 * state, has run).  A writer waits on `free` before reusing an entry.
 * Entry memory is caller-owned device memory of zl_pipeline_entry_bytes.
 *
 * All calls are asynchronous except zl_pipeline_sync, the checkpoint calls
 * and zl_pipeline_destroy; errors are zl_status codes with detail in
 * zl_last_error(); arguments are validated before any work is enqueued.
 *
 * Checkpoint (Sec. III-B, failure recovery: each stage checkpoints its
 * trainable parameters, optimizer state and progress metadata on its own).
 * File format (little endian): a 256-byte header
 *   0   char[8]  magic "ZLCKPT01"
 *   8   uint32   header bytes (256)
 *   12  uint32   optimizer (ZL_ADAMW / ZL_SGD)
 *   16  int32    arch, n_layers, d_model, n_heads, n_kv_heads, head_dim,
 *                d_ff, vocab, dtype                       (9 x int32)
 *   52  uint32   payload tensors (3 for AdamW: master, m, v; 1 for SGD)
 *   56  uint64   n_params
 *   64  int64    optimizer step
 *   72  int64    progress: micro-batches consumed
 *   80  int64    progress: update windows completed
 *   88  uint64   FNV-1a 64 over the payload as 32-bit little-endian words
 *   96  zero padding to 256
 * followed by the payload: fp32 master [n_params], then (AdamW) adam_m and
 * adam_v [n_params] each.  The gradient is not saved: checkpoints are taken
 * at window boundaries, where it holds no pending contribution.
 */
#ifndef ZL_RUNTIME_H
#define ZL_RUNTIME_H

#include <stddef.h>
#include <stdint.h>

#include "zl.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct zl_pipeline zl_pipeline;

/* Device bytes of entry memory for K stages with in-flight depth `depth`,
 * sized for the first chunk's max_batch x max_seq x d_model (activation
 * dtype of the chunks).  ZL_ERR_INVALID_ARG if K < 1 or depth < 1. */
zl_status zl_pipeline_entry_bytes(const zl_chunk* first, int K, int depth, size_t* bytes);

/* chunks[0..K-1]: created chunks (same d_model, dtype, max_batch, max_seq);
 * streams[0..K-1]: distinct hipStream_t, one per stage; window: micro-batches
 * per update window m >= 1 (each micro-batch's gradient is scaled by 1/m,
 * the optimizer steps after the m-th); depth: in-flight entries per stage
 * boundary >= 1; entries: device memory of at least
 * zl_pipeline_entry_bytes(chunks[0], K, depth) bytes, 256-byte aligned.
 * The pipeline keeps pointers only; the caller keeps chunks, streams and
 * entry memory alive until zl_pipeline_destroy.  Creates HIP events
 * (no device memory).  The chunks must be idle (no call in flight). */
zl_status zl_pipeline_create(zl_chunk* const* chunks, int K, void* const* streams, int window,
                             int depth, void* entries, size_t entry_bytes, zl_pipeline** out);

/* Submit one micro-batch.  h0 [B, S, d_model] (activation dtype) is stage
 * 0's input; labels [B, S] (-100 = not in Omega), pos_ids [B, S] or NULL
 * (0 .. S-1), seq_lens [B] or NULL (S) as for zl_chunk_forward /
 * zl_local_objective.  They are copied into stage 0's input entry on stage
 * 0's stream: the caller keeps them unchanged until that stream has passed
 * this call (e.g. until zl_pipeline_sync).  losses: device float[K], stage
 * k's local loss of this micro-batch is written to losses[k] on stream k.
 * Returns the micro-batch's sequence number in *mb (may be NULL). */
zl_status zl_pipeline_submit(zl_pipeline* p, const void* h0, const int32_t* labels,
                             const int32_t* pos_ids, const int32_t* seq_lens, int B, int S,
                             float* losses, int64_t* mb);

/* Enqueue on `stream` (a hipStream_t): wait until the last stage has
 * written micro-batch `mb`'s output hidden state, then copy it [B, S,
 * d_model] (activation dtype) to device memory `dst`.  The output entry is
 * not reused before this copy has run.  ZL_ERR_INVALID_ARG if `mb` was not
 * submitted or its entry was already reused (`depth` later submissions). */
zl_status zl_pipeline_read_output(zl_pipeline* p, int64_t mb, void* dst, void* stream);

/* Block the host until every stage's stream has finished all submitted work. */
zl_status zl_pipeline_sync(zl_pipeline* p);

/* Progress: micro-batches submitted and update windows completed. */
zl_status zl_pipeline_progress(const zl_pipeline* p, int64_t* microbatches, int64_t* windows);

/* Write stage `stage`'s checkpoint (parameters, optimizer state, step and
 * the pipeline's progress) to `path`.  Only at a window boundary (the
 * submitted micro-batches are a multiple of the window), else ZL_ERR_STATE.
 * Waits for that stage's stream. */
zl_status zl_pipeline_checkpoint(zl_pipeline* p, int stage, const char* path);

void zl_pipeline_destroy(zl_pipeline* p);

/* Write a chunk's checkpoint with the given progress metadata.  Waits for
 * `stream`, then copies master (and adam_m, adam_v) to the file through a
 * bounded host staging buffer.  ZL_ERR_INVALID_ARG if the file cannot be
 * written, ZL_ERR_STATE if a forward/objective is pending (the gradient
 * window must be closed). */
zl_status zl_chunk_save(zl_chunk* chunk, const char* path, int64_t microbatches,
                        int64_t windows, void* stream);

/* Restore a chunk from a checkpoint: checks the header against the chunk's
 * configuration (architecture, shapes, dtype, optimizer, parameter count)
 * and the payload checksum, then writes master, adam_m, adam_v and the step,
 * refreshes the bf16 shadow and marks the gradient window closed.  Progress
 * is returned in *microbatches / *windows (may be NULL).  On any mismatch
 * ZL_ERR_INVALID_ARG and the chunk is unchanged. */
zl_status zl_chunk_load(zl_chunk* chunk, const char* path, int64_t* microbatches,
                        int64_t* windows, void* stream);

/* Header fields of a checkpoint file (host only; no device needed). */
typedef struct zl_checkpoint_info {
  int arch, n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, dtype, optimizer;
  uint64_t n_params;
  int64_t step, microbatches, windows;
  uint64_t checksum;
} zl_checkpoint_info;

/* Parse and validate a checkpoint's header and size (magic, header length,
 * tensor count, file length = header + payload).  ZL_ERR_INVALID_ARG if the
 * file is missing, short or malformed. */
zl_status zl_checkpoint_read_info(const char* path, zl_checkpoint_info* out);

#ifdef __cplusplus
}
#endif
#endif /* ZL_RUNTIME_H */
