// Single-GPU ZeroLock runtime: a pipeline of chunks with early forwarding
// over event-bound hidden-state entries, and per-chunk checkpoint / resume
// (Sec. III-B: inter-stage runtime, in-stage execution S1-S3, failure
// recovery).  Built on the public C ABI of the chunk.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <string.h>

#include <string>
#include <vector>

#include "../../include/zl.h"
#include "../../include/zl_runtime.h"
#include "internal.h"

using zl::set_error;

#define RT_HIP(call)                                                                        \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return set_error(ZL_ERR_HIP, std::string(#call) + ": " + hipGetErrorString(e_));      \
  } while (0)

#define RT_OK(call)                    \
  do {                                 \
    zl_status s_ = (call);             \
    if (s_ != ZL_OK) return s_;        \
  } while (0)

namespace {

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Byte layout of one entry: hidden state, labels, position ids, lengths.
struct EntryLayout {
  size_t h, lab, pos, seq, bytes;
  EntryLayout(const zl_config& c) {
    const size_t elt = c.dtype == ZL_BF16 ? 2 : 4;
    const size_t tok = (size_t)c.max_batch * c.max_seq;
    h = 0;
    lab = round_up(tok * c.d_model * elt, 256);
    pos = lab + round_up(tok * 4, 256);
    seq = pos + round_up(tok * 4, 256);
    bytes = seq + round_up((size_t)c.max_batch * 4, 256);
  }
};

}  // namespace

struct zl_pipeline {
  int K = 0, window = 1, depth = 1;
  std::vector<zl_chunk*> chunks;
  std::vector<hipStream_t> streams;
  zl_config cfg;
  EntryLayout lay{zl_config{}};
  char* entries = nullptr;
  // ring r (0 = stage 0 input, k = input of stage k, K = pipeline output),
  // slot j: events at index r * depth + j
  std::vector<hipEvent_t> ready, freed;
  std::vector<char> out_read;   // per output slot: a read_output copy is pending
  std::vector<int> out_B, out_S;  // per output slot: shape of its micro-batch
  int64_t submitted = 0;

  char* entry(int r, int j) const { return entries + ((size_t)r * depth + j) * lay.bytes; }
  hipEvent_t& rdy(int r, int j) { return ready[(size_t)r * depth + j]; }
  hipEvent_t& fre(int r, int j) { return freed[(size_t)r * depth + j]; }
};

extern "C" {

zl_status zl_pipeline_entry_bytes(const zl_chunk* first, int K, int depth, size_t* bytes) {
  if (!first || !bytes) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  if (K < 1 || depth < 1) return set_error(ZL_ERR_INVALID_ARG, "K and depth must be >= 1");
  zl_config c;
  RT_OK(zl_chunk_get_config(first, &c));
  *bytes = EntryLayout(c).bytes * (size_t)(K + 1) * depth;
  return ZL_OK;
}

zl_status zl_pipeline_create(zl_chunk* const* chunks, int K, void* const* streams, int window,
                             int depth, void* entries, size_t entry_bytes, zl_pipeline** out) {
  if (!chunks || !streams || !entries || !out) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  *out = nullptr;
  if (K < 1 || window < 1 || depth < 1)
    return set_error(ZL_ERR_INVALID_ARG, "K, window and depth must be >= 1");
  if (reinterpret_cast<uintptr_t>(entries) % 256)
    return set_error(ZL_ERR_INVALID_ARG, "entry memory must be 256-byte aligned");
  zl_config c0;
  for (int k = 0; k < K; ++k) {
    if (!chunks[k] || !streams[k]) return set_error(ZL_ERR_INVALID_ARG, "NULL chunk or stream");
    zl_config c;
    RT_OK(zl_chunk_get_config(chunks[k], &c));
    if (k == 0) c0 = c;
    if (c.d_model != c0.d_model || c.dtype != c0.dtype || c.max_batch != c0.max_batch ||
        c.max_seq != c0.max_seq)
      return set_error(ZL_ERR_INVALID_ARG,
                       "stage " + std::to_string(k) + ": d_model, dtype, max_batch and max_seq "
                       "must match stage 0");
    if (!zl::chunk_at_boundary(chunks[k]))
      return set_error(ZL_ERR_STATE, "stage " + std::to_string(k) + " has a call in flight");
    for (int i = 0; i < k; ++i)
      if (chunks[i] == chunks[k] || streams[i] == streams[k])
        return set_error(ZL_ERR_INVALID_ARG, "chunks and streams must be distinct per stage");
  }
  size_t need = 0;
  RT_OK(zl_pipeline_entry_bytes(chunks[0], K, depth, &need));
  if (entry_bytes < need)
    return set_error(ZL_ERR_WORKSPACE, "entry memory too small: need " + std::to_string(need));
  zl_pipeline* p = new zl_pipeline;
  p->K = K;
  p->window = window;
  p->depth = depth;
  p->cfg = c0;
  p->lay = EntryLayout(c0);
  p->entries = reinterpret_cast<char*>(entries);
  for (int k = 0; k < K; ++k) {
    p->chunks.push_back(chunks[k]);
    p->streams.push_back(reinterpret_cast<hipStream_t>(streams[k]));
  }
  p->out_read.assign(depth, 0);
  p->out_B.assign(depth, 0);
  p->out_S.assign(depth, 0);
  const size_t ne = (size_t)(K + 1) * depth;
  p->ready.assign(ne, nullptr);
  p->freed.assign(ne, nullptr);
  for (size_t i = 0; i < ne; ++i) {
    if (hipEventCreateWithFlags(&p->ready[i], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&p->freed[i], hipEventDisableTiming) != hipSuccess) {
      zl_pipeline_destroy(p);
      return set_error(ZL_ERR_HIP, "hipEventCreate failed");
    }
  }
  *out = p;
  return ZL_OK;
}

zl_status zl_pipeline_submit(zl_pipeline* p, const void* h0, const int32_t* labels,
                             const int32_t* pos_ids, const int32_t* seq_lens, int B, int S,
                             float* losses, int64_t* mb) {
  if (!p || !h0 || !labels || !losses) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  if (B < 1 || S < 1 || B > p->cfg.max_batch || S > p->cfg.max_seq)
    return set_error(ZL_ERR_INVALID_ARG, "B, S outside [1, max_batch] x [1, max_seq]");
  const int64_t i = p->submitted;
  const int j = (int)(i % p->depth);
  const bool reuse = i >= p->depth;
  const size_t elt = p->cfg.dtype == ZL_BF16 ? 2 : 4;
  const size_t hb = (size_t)B * S * p->cfg.d_model * elt, tb = (size_t)B * S * 4;
  const float scale = 1.f / (float)p->window;
  const bool first_of_window = i % p->window == 0;
  const bool last_of_window = i % p->window == p->window - 1;

  // S1 for stage 0: copy the micro-batch into its input entry
  {
    hipStream_t s0 = p->streams[0];
    char* e = p->entry(0, j);
    if (reuse) RT_HIP(hipStreamWaitEvent(s0, p->fre(0, j), 0));
    RT_HIP(hipMemcpyAsync(e + p->lay.h, h0, hb, hipMemcpyDeviceToDevice, s0));
    RT_HIP(hipMemcpyAsync(e + p->lay.lab, labels, tb, hipMemcpyDeviceToDevice, s0));
    if (pos_ids) RT_HIP(hipMemcpyAsync(e + p->lay.pos, pos_ids, tb, hipMemcpyDeviceToDevice, s0));
    if (seq_lens)
      RT_HIP(hipMemcpyAsync(e + p->lay.seq, seq_lens, (size_t)B * 4, hipMemcpyDeviceToDevice, s0));
    RT_HIP(hipEventRecord(p->rdy(0, j), s0));
  }
  for (int k = 0; k < p->K; ++k) {
    hipStream_t sk = p->streams[k];
    zl_chunk* c = p->chunks[k];
    char* in = p->entry(k, j);
    char* out = p->entry(k + 1, j);
    RT_HIP(hipStreamWaitEvent(sk, p->rdy(k, j), 0));  // S1: input entry written
    if (reuse && (k + 1 < p->K || p->out_read[j]))     // output entry's last reader done
      RT_HIP(hipStreamWaitEvent(sk, p->fre(k + 1, j), 0));
    const int32_t* sl = seq_lens ? reinterpret_cast<const int32_t*>(in + p->lay.seq) : nullptr;
    const int32_t* pi = pos_ids ? reinterpret_cast<const int32_t*>(in + p->lay.pos) : nullptr;
    // S2: forward, output entry (hidden state and metadata) marked ready
    RT_OK(zl_chunk_forward(c, in + p->lay.h, sl, pi, B, S, out + p->lay.h, sk));
    RT_HIP(hipMemcpyAsync(out + p->lay.lab, in + p->lay.lab, tb, hipMemcpyDeviceToDevice, sk));
    if (pos_ids)
      RT_HIP(hipMemcpyAsync(out + p->lay.pos, in + p->lay.pos, tb, hipMemcpyDeviceToDevice, sk));
    if (seq_lens)
      RT_HIP(hipMemcpyAsync(out + p->lay.seq, in + p->lay.seq, (size_t)B * 4,
                            hipMemcpyDeviceToDevice, sk));
    RT_HIP(hipEventRecord(p->rdy(k + 1, j), sk));
    // S3: local objective, backward into the window, step at its end
    RT_OK(zl_local_objective(c, reinterpret_cast<const int32_t*>(in + p->lay.lab), losses + k, sk));
    RT_OK(zl_chunk_backward(c, scale, first_of_window ? 0 : 1, sk));
    RT_HIP(hipEventRecord(p->fre(k, j), sk));  // the input entry's last use is done
    if (last_of_window) RT_OK(zl_optimizer_step(c, sk));
  }
  p->out_read[j] = 0;
  p->out_B[j] = B;
  p->out_S[j] = S;
  p->submitted = i + 1;
  if (mb) *mb = i;
  return ZL_OK;
}

zl_status zl_pipeline_read_output(zl_pipeline* p, int64_t mb, void* dst, void* stream) {
  if (!p || !dst) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  if (mb < 0 || mb >= p->submitted || mb < p->submitted - p->depth)
    return set_error(ZL_ERR_INVALID_ARG, "micro-batch not submitted or its entry was reused");
  const int j = (int)(mb % p->depth);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const size_t elt = p->cfg.dtype == ZL_BF16 ? 2 : 4;
  const size_t hb = (size_t)p->out_B[j] * p->out_S[j] * p->cfg.d_model * elt;
  RT_HIP(hipStreamWaitEvent(s, p->rdy(p->K, j), 0));
  RT_HIP(hipMemcpyAsync(dst, p->entry(p->K, j) + p->lay.h, hb, hipMemcpyDeviceToDevice, s));
  RT_HIP(hipEventRecord(p->fre(p->K, j), s));  // the last stage waits on this before reuse
  p->out_read[j] = 1;
  return ZL_OK;
}

zl_status zl_pipeline_sync(zl_pipeline* p) {
  if (!p) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  for (hipStream_t s : p->streams) RT_HIP(hipStreamSynchronize(s));
  return ZL_OK;
}

zl_status zl_pipeline_progress(const zl_pipeline* p, int64_t* microbatches, int64_t* windows) {
  if (!p) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  if (microbatches) *microbatches = p->submitted;
  if (windows) *windows = p->submitted / p->window;
  return ZL_OK;
}

zl_status zl_pipeline_checkpoint(zl_pipeline* p, int stage, const char* path) {
  if (!p || !path) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  if (stage < 0 || stage >= p->K) return set_error(ZL_ERR_INVALID_ARG, "stage out of range");
  if (p->submitted % p->window)
    return set_error(ZL_ERR_STATE, "checkpoints are taken at update-window boundaries");
  return zl_chunk_save(p->chunks[stage], path, p->submitted, p->submitted / p->window,
                       p->streams[stage]);
}

void zl_pipeline_destroy(zl_pipeline* p) {
  if (!p) return;
  for (hipStream_t s : p->streams) (void)hipStreamSynchronize(s);
  for (hipEvent_t e : p->ready)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : p->freed)
    if (e) (void)hipEventDestroy(e);
  delete p;
}

}  // extern "C"

// ------------------------------------------------------------- checkpoint
namespace {

constexpr char MAGIC[8] = {'Z', 'L', 'C', 'K', 'P', 'T', '0', '1'};
constexpr uint32_t HEADER_BYTES = 256;
constexpr size_t STAGE_BYTES = (size_t)64 << 20;  // host staging per copy

struct Header {  // the on-disk layout documented in zl_runtime.h
  char magic[8];
  uint32_t header_bytes;
  uint32_t optimizer;
  int32_t shape[9];  // arch, n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, dtype
  uint32_t tensors;
  uint64_t n_params;
  int64_t step, microbatches, windows;
  uint64_t checksum;
  unsigned char pad[HEADER_BYTES - 96];
};
static_assert(sizeof(Header) == HEADER_BYTES, "checkpoint header layout");
static_assert(offsetof(Header, tensors) == 52 && offsetof(Header, n_params) == 56 &&
                  offsetof(Header, checksum) == 88,
              "checkpoint header offsets");

// FNV-1a 64 over the payload's 32-bit little-endian words
struct Fnv {
  uint64_t h = 0xcbf29ce484222325ull;
  void add(const void* p, size_t n) {
    const uint32_t* w = reinterpret_cast<const uint32_t*>(p);
    for (size_t i = 0; i < n / 4; ++i) {
      h ^= w[i];
      h *= 0x100000001b3ull;
    }
  }
};

void fill_shape(const zl_config& c, int32_t* s) {
  const int32_t v[9] = {c.arch, c.n_layers, c.d_model, c.n_heads, c.n_kv_heads,
                        c.head_dim, c.d_ff, c.vocab, c.dtype};
  memcpy(s, v, sizeof(v));
}

const char* SHAPE_NAMES[9] = {"arch", "n_layers", "d_model", "n_heads", "n_kv_heads",
                              "head_dim", "d_ff", "vocab", "dtype"};

zl_status read_header(FILE* f, const char* path, Header* h, uint64_t* file_bytes) {
  if (fseek(f, 0, SEEK_END) != 0) return set_error(ZL_ERR_INVALID_ARG, "cannot seek " + std::string(path));
  const long len = ftell(f);
  rewind(f);
  if (len < (long)HEADER_BYTES || fread(h, 1, HEADER_BYTES, f) != HEADER_BYTES)
    return set_error(ZL_ERR_INVALID_ARG, std::string(path) + ": shorter than the header");
  if (memcmp(h->magic, MAGIC, 8) != 0 || h->header_bytes != HEADER_BYTES)
    return set_error(ZL_ERR_INVALID_ARG, std::string(path) + ": not a ZeroLock checkpoint");
  const uint32_t want = h->optimizer == ZL_ADAMW ? 3u : 1u;
  if ((h->optimizer != ZL_ADAMW && h->optimizer != ZL_SGD) || h->tensors != want)
    return set_error(ZL_ERR_INVALID_ARG, std::string(path) + ": bad optimizer / tensor count");
  const uint64_t expect = HEADER_BYTES + (uint64_t)h->tensors * h->n_params * 4;
  if ((uint64_t)len != expect)
    return set_error(ZL_ERR_INVALID_ARG, std::string(path) + ": file length " +
                                             std::to_string(len) + " != " + std::to_string(expect));
  *file_bytes = (uint64_t)len;
  return ZL_OK;
}

}  // namespace

extern "C" {

zl_status zl_chunk_save(zl_chunk* chunk, const char* path, int64_t microbatches, int64_t windows,
                        void* stream) {
  if (!chunk || !path) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  RT_HIP(hipStreamSynchronize(reinterpret_cast<hipStream_t>(stream)));
  if (!zl::chunk_at_boundary(chunk))
    return set_error(ZL_ERR_STATE, "a call or an unapplied gradient is pending");
  zl_config cfg;
  zl_buffers buf;
  size_t n = 0;
  int64_t step = 0;
  RT_OK(zl_chunk_get_config(chunk, &cfg));
  RT_OK(zl_chunk_get_buffers(chunk, &buf));
  RT_OK(zl_chunk_num_params(chunk, &n));
  RT_OK(zl_get_step(chunk, &step));
  Header h;
  memset(&h, 0, sizeof(h));
  memcpy(h.magic, MAGIC, 8);
  h.header_bytes = HEADER_BYTES;
  h.optimizer = (uint32_t)cfg.optimizer;
  fill_shape(cfg, h.shape);
  h.tensors = cfg.optimizer == ZL_ADAMW ? 3 : 1;
  h.n_params = n;
  h.step = step;
  h.microbatches = microbatches;
  h.windows = windows;
  FILE* f = fopen(path, "wb");
  if (!f) return set_error(ZL_ERR_INVALID_ARG, std::string("cannot open ") + path + " for writing");
  std::vector<char> host(n * 4 < STAGE_BYTES ? n * 4 : STAGE_BYTES);
  Fnv fnv;
  bool ok = fwrite(&h, 1, HEADER_BYTES, f) == HEADER_BYTES;
  const float* tens[3] = {buf.master, buf.adam_m, buf.adam_v};
  for (uint32_t t = 0; ok && t < h.tensors; ++t) {
    const char* src = reinterpret_cast<const char*>(tens[t]);
    for (size_t off = 0; ok && off < n * 4; off += host.size()) {
      const size_t len = n * 4 - off < host.size() ? n * 4 - off : host.size();
      if (hipMemcpy(host.data(), src + off, len, hipMemcpyDeviceToHost) != hipSuccess) {
        fclose(f);
        return set_error(ZL_ERR_HIP, "device-to-host copy of the chunk state failed");
      }
      fnv.add(host.data(), len);
      ok = fwrite(host.data(), 1, len, f) == len;
    }
  }
  h.checksum = fnv.h;
  ok = ok && fseek(f, 0, SEEK_SET) == 0 && fwrite(&h, 1, HEADER_BYTES, f) == HEADER_BYTES;
  ok = (fclose(f) == 0) && ok;
  if (!ok) return set_error(ZL_ERR_INVALID_ARG, std::string("write failed: ") + path);
  return ZL_OK;
}

zl_status zl_checkpoint_read_info(const char* path, zl_checkpoint_info* out) {
  if (!path || !out) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  FILE* f = fopen(path, "rb");
  if (!f) return set_error(ZL_ERR_INVALID_ARG, std::string("cannot open ") + path);
  Header h;
  uint64_t len = 0;
  const zl_status st = read_header(f, path, &h, &len);
  fclose(f);
  if (st != ZL_OK) return st;
  out->arch = h.shape[0];
  out->n_layers = h.shape[1];
  out->d_model = h.shape[2];
  out->n_heads = h.shape[3];
  out->n_kv_heads = h.shape[4];
  out->head_dim = h.shape[5];
  out->d_ff = h.shape[6];
  out->vocab = h.shape[7];
  out->dtype = h.shape[8];
  out->optimizer = (int)h.optimizer;
  out->n_params = h.n_params;
  out->step = h.step;
  out->microbatches = h.microbatches;
  out->windows = h.windows;
  out->checksum = h.checksum;
  return ZL_OK;
}

zl_status zl_chunk_load(zl_chunk* chunk, const char* path, int64_t* microbatches, int64_t* windows,
                        void* stream) {
  if (!chunk || !path) return set_error(ZL_ERR_INVALID_ARG, "NULL argument");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  zl_config cfg;
  zl_buffers buf;
  size_t n = 0;
  RT_OK(zl_chunk_get_config(chunk, &cfg));
  RT_OK(zl_chunk_get_buffers(chunk, &buf));
  RT_OK(zl_chunk_num_params(chunk, &n));
  FILE* f = fopen(path, "rb");
  if (!f) return set_error(ZL_ERR_INVALID_ARG, std::string("cannot open ") + path);
  Header h;
  uint64_t len = 0;
  zl_status st = read_header(f, path, &h, &len);
  int32_t shape[9];
  fill_shape(cfg, shape);
  for (int i = 0; st == ZL_OK && i < 9; ++i)
    if (shape[i] != h.shape[i])
      st = set_error(ZL_ERR_INVALID_ARG, std::string(path) + ": " + SHAPE_NAMES[i] + " " +
                                             std::to_string(h.shape[i]) + " != chunk's " +
                                             std::to_string(shape[i]));
  if (st == ZL_OK && (h.optimizer != (uint32_t)cfg.optimizer || h.n_params != n))
    st = set_error(ZL_ERR_INVALID_ARG, std::string(path) + ": optimizer or parameter count differs");
  if (st != ZL_OK) {
    fclose(f);
    return st;
  }
  // pass 1: verify the checksum before touching the chunk
  std::vector<char> host(n * 4 < STAGE_BYTES ? n * 4 : STAGE_BYTES);
  Fnv fnv;
  const uint64_t payload = len - HEADER_BYTES;
  for (uint64_t off = 0; off < payload; off += host.size()) {
    const size_t l = payload - off < host.size() ? (size_t)(payload - off) : host.size();
    if (fread(host.data(), 1, l, f) != l) {
      fclose(f);
      return set_error(ZL_ERR_INVALID_ARG, std::string(path) + ": short read");
    }
    fnv.add(host.data(), l);
  }
  if (fnv.h != h.checksum) {
    fclose(f);
    return set_error(ZL_ERR_INVALID_ARG, std::string(path) + ": payload checksum mismatch");
  }
  // pass 2: restore
  if (hipStreamSynchronize(s) != hipSuccess) {
    fclose(f);
    return set_error(ZL_ERR_HIP, "stream synchronize failed");
  }
  fseek(f, HEADER_BYTES, SEEK_SET);
  float* tens[3] = {buf.master, buf.adam_m, buf.adam_v};
  for (uint32_t t = 0; t < h.tensors; ++t) {
    char* dst = reinterpret_cast<char*>(tens[t]);
    for (size_t off = 0; off < n * 4; off += host.size()) {
      const size_t l = n * 4 - off < host.size() ? n * 4 - off : host.size();
      if (fread(host.data(), 1, l, f) != l ||
          hipMemcpy(dst + off, host.data(), l, hipMemcpyHostToDevice) != hipSuccess) {
        fclose(f);
        return set_error(ZL_ERR_HIP, std::string(path) + ": restore failed part-way");
      }
    }
  }
  fclose(f);
  RT_OK(zl_set_step(chunk, h.step));
  zl::chunk_close_window(chunk);
  RT_OK(zl_refresh_shadow(chunk, stream));
  if (microbatches) *microbatches = h.microbatches;
  if (windows) *windows = h.windows;
  return ZL_OK;
}

}  // extern "C"
