// Host side of the C ABI (include/zl.h): configuration checks, the flat
// parameter layout, the workspace plan, the call-order state machine and the
// launch sequences of the chunk-local update.
//
// Order of work inside one update (Sec. III-B, in-stage steps S1-S3):
//   forward    cast h_in -> X0 (fp32 residual stream); per layer:
//              norm1 -> QKV GEMM (+bias) -> RoPE -> attention -> O GEMM +
//              residual -> norm2 -> up GEMM (+GELU) [-> SwiGLU] -> down GEMM
//              + residual; cast X_L -> h_out (early-forward point)
//   objective  |Omega|; per row block of the head: head norm of h_out (and
//              h_in) -> logits GEMM -> row stats, loss rows, dL/dz ->
//              dz W_lm GEMM -> head-norm backward into dL/dh_out
//   backward   per layer, last to first: down dgrad (+SwiGLU/GELU bwd),
//              down wgrad, up dgrad, up wgrad, norm2 bwd, O dgrad, O wgrad,
//              attention bwd, RoPE bwd, QKV dgrad, QKV wgrad, norm1 bwd;
//              layer 0 forms no gradient into h_in (Remark 1)
//   step       AdamW / SGD over the flat buffers, bf16 shadow refresh
#include <math.h>
#include <string.h>

#include <string>
#include <vector>

#include "../../include/zl.h"
#include "../../include/zl_inspect.h"
#include "internal.h"
#include "common.h"

using namespace zl;

static thread_local std::string g_err;

static zl_status fail(zl_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define ZL_HIP(call)                                                              \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess)                                                         \
      return fail(ZL_ERR_HIP, std::string(#call) + ": " + hipGetErrorString(e_)); \
  } while (0)

// ----------------------------------------------------------------- layout
namespace {

constexpr size_t ALIGN_ELEMS = 64;
constexpr size_t ALIGN_BYTES = 256;

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct LayerOff {
  size_t ln1_w, ln1_b, w_qkv, b_qkv, w_o, b_o, ln2_w, ln2_b, w_up, b_up, w_down, b_down;
};

struct Dims {
  int arch, L, d, hq, hkv, hd, ff, V, dq, dkv, nqkv, nup;
  int ar;  // readout adapter width (0 = none)
  int lr;  // LoRA rank as stored: the configured rank rounded up to 8 (0 = full training)
  int lq;  // the configured LoRA rank (factor rows/columns lq .. lr-1 are zero padding)
  int nqa, nua;  // rows of the stacked A factors of the QKV and up projections
  float ls;      // LoRA scale lora_alpha / lq
  bool llama;
};

Dims dims_of(const zl_config& c) {
  Dims m;
  m.arch = c.arch;
  m.llama = c.arch == ZL_ARCH_LLAMA;
  m.L = c.n_layers;
  m.d = c.d_model;
  m.hq = c.n_heads;
  m.hkv = c.n_kv_heads;
  m.hd = c.head_dim;
  m.ff = c.d_ff;
  m.V = c.vocab;
  m.dq = m.hq * m.hd;
  m.dkv = m.hkv * m.hd;
  m.nqkv = m.dq + 2 * m.dkv;
  m.nup = m.llama ? 2 * m.ff : m.ff;
  m.ar = c.adapter_rank;
  m.lq = c.lora_rank;
  m.lr = (c.lora_rank + 7) / 8 * 8;
  m.nqa = m.llama ? 3 * m.lr : m.lr;
  m.nua = m.llama ? 2 * m.lr : m.lr;
  m.ls = m.lq ? c.lora_alpha / (float)m.lq : 0.f;
  return m;
}

zl_status check_config(const zl_config* c) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "config is NULL");
  if (c->arch != ZL_ARCH_LLAMA && c->arch != ZL_ARCH_GPT2)
    return fail(ZL_ERR_INVALID_ARG, "arch must be ZL_ARCH_LLAMA or ZL_ARCH_GPT2");
  if (c->n_layers < 1) return fail(ZL_ERR_INVALID_ARG, "n_layers must be >= 1");
  if (c->d_model < 64 || c->d_model % 64)
    return fail(ZL_ERR_INVALID_ARG, "d_model must be a positive multiple of 64");
  if (c->d_model > 8192) return fail(ZL_ERR_UNSUPPORTED, "d_model above 8192");
  if (c->arch == ZL_ARCH_GPT2 && c->d_model > 4096)
    return fail(ZL_ERR_UNSUPPORTED, "LayerNorm form above d_model 4096");
  if (c->n_heads < 1 || c->n_kv_heads < 1 || c->n_heads % c->n_kv_heads)
    return fail(ZL_ERR_INVALID_ARG, "n_heads must be a positive multiple of n_kv_heads");
  if (c->head_dim < 8 || c->head_dim % 8)
    return fail(ZL_ERR_INVALID_ARG, "head_dim must be a positive multiple of 8");
  if (c->head_dim != 16 && c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128)
    return fail(ZL_ERR_UNSUPPORTED, "head_dim must be 16, 32, 64 or 128");
  if (c->d_ff < 64 || c->d_ff % 64)
    return fail(ZL_ERR_INVALID_ARG, "d_ff must be a positive multiple of 64");
  if (c->vocab < 2) return fail(ZL_ERR_INVALID_ARG, "vocab must be >= 2");
  if (!(c->norm_eps > 0.f)) return fail(ZL_ERR_INVALID_ARG, "norm_eps must be > 0");
  if (c->arch == ZL_ARCH_LLAMA && !(c->rope_theta > 1.f))
    return fail(ZL_ERR_INVALID_ARG, "rope_theta must be > 1 for llama");
  if (c->dtype != ZL_F32 && c->dtype != ZL_BF16)
    return fail(ZL_ERR_INVALID_ARG, "dtype must be ZL_F32 or ZL_BF16");
  if (!(c->alpha > 0.f && c->alpha <= 1.f))
    return fail(ZL_ERR_INVALID_ARG, "alpha must be in (0, 1]");
  if (c->consis != ZL_KL_REVERSE && c->consis != ZL_KL_FORWARD)
    return fail(ZL_ERR_INVALID_ARG, "consis must be ZL_KL_REVERSE or ZL_KL_FORWARD");
  if (c->optimizer != ZL_ADAMW && c->optimizer != ZL_SGD)
    return fail(ZL_ERR_INVALID_ARG, "optimizer must be ZL_ADAMW or ZL_SGD");
  if (!(c->lr >= 0.f)) return fail(ZL_ERR_INVALID_ARG, "lr must be >= 0");
  if (c->optimizer == ZL_ADAMW) {
    if (!(c->beta1 >= 0.f && c->beta1 < 1.f) || !(c->beta2 >= 0.f && c->beta2 < 1.f))
      return fail(ZL_ERR_INVALID_ARG, "betas must be in [0, 1)");
    if (!(c->eps > 0.f)) return fail(ZL_ERR_INVALID_ARG, "eps must be > 0");
    if (!(c->weight_decay >= 0.f)) return fail(ZL_ERR_INVALID_ARG, "weight_decay must be >= 0");
  }
  if (c->max_batch < 1 || c->max_seq < 1)
    return fail(ZL_ERR_INVALID_ARG, "max_batch and max_seq must be >= 1");
  if ((int64_t)c->max_batch * c->max_seq > (int64_t)1 << 24)
    return fail(ZL_ERR_UNSUPPORTED, "max_batch * max_seq above 2^24 tokens");
  if (c->adapter_rank < 0 || c->adapter_rank % 16 || c->adapter_rank > 8192)
    return fail(ZL_ERR_INVALID_ARG, "adapter_rank must be 0 or a multiple of 16 up to 8192");
  if (c->lora_rank < 0 || c->lora_rank > 256)
    return fail(ZL_ERR_INVALID_ARG, "lora_rank must be in [0, 256]");
  if (c->lora_rank && !(c->lora_alpha > 0.f && isfinite(c->lora_alpha)))
    return fail(ZL_ERR_INVALID_ARG, "lora_alpha must be finite and > 0");
  return ZL_OK;
}

// LoRA factor offsets of one layer.  A factors of projections that share an
// input (q/k/v, gate/up) are adjacent, i.e. one stacked [nblk * r, in]
// matrix; so are their B factors ([sum of outs, r]).
struct LoraOff {
  size_t qkv_a, qkv_b, o_a, o_b, up_a, up_b, down_a, down_b;
};

struct Layout {
  std::vector<zl_tensor_desc> descs;  // trainable tensors
  std::vector<LayerOff> lay;  // layer tensors: trainable buffers, or the base buffers with LoRA
  std::vector<LoraOff> lora;  // lora_rank > 0
  size_t ad_w1 = 0, ad_w2 = 0;  // readout adapter (adapter_rank > 0)
  size_t n_params = 0;  // trainable elements
  size_t n_base = 0;    // base buffer elements (lora_rank > 0)
};

// Appends tensors to a flat buffer, each offset a multiple of ALIGN_ELEMS.
struct Packer {
  std::vector<zl_tensor_desc>* descs;
  size_t off = 0;
  size_t add(const char* name, int layer, int64_t r, int64_t cols, int ndim) {
    zl_tensor_desc t;
    memset(&t, 0, sizeof(t));
    strncpy(t.name, name, sizeof(t.name) - 1);
    t.layer = layer;
    t.ndim = ndim;
    t.shape[0] = r;
    t.shape[1] = cols;
    t.offset = off;
    t.numel = (size_t)r * cols;
    if (descs) descs->push_back(t);
    const size_t at = off;
    off = round_up(off + t.numel, ALIGN_ELEMS);
    return at;
  }
};

void layer_tensors(const Dims& m, Packer& pk, std::vector<LayerOff>& lay) {
  lay.resize(m.L);
  for (int l = 0; l < m.L; ++l) {
    LayerOff& o = lay[l];
    memset(&o, 0, sizeof(o));
    if (m.llama) {
      o.ln1_w = pk.add("ln1_w", l, m.d, 1, 1);
      o.w_qkv = pk.add("wq", l, m.dq, m.d, 2);
      pk.add("wk", l, m.dkv, m.d, 2);
      pk.add("wv", l, m.dkv, m.d, 2);
      o.w_o = pk.add("wo", l, m.d, m.dq, 2);
      o.ln2_w = pk.add("ln2_w", l, m.d, 1, 1);
      o.w_up = pk.add("wg", l, m.ff, m.d, 2);
      pk.add("wu", l, m.ff, m.d, 2);
      o.w_down = pk.add("wd", l, m.d, m.ff, 2);
    } else {
      o.ln1_w = pk.add("ln1_w", l, m.d, 1, 1);
      o.ln1_b = pk.add("ln1_b", l, m.d, 1, 1);
      o.w_qkv = pk.add("wqkv", l, m.nqkv, m.d, 2);
      o.b_qkv = pk.add("bqkv", l, m.nqkv, 1, 1);
      o.w_o = pk.add("wo", l, m.d, m.dq, 2);
      o.b_o = pk.add("bo", l, m.d, 1, 1);
      o.ln2_w = pk.add("ln2_w", l, m.d, 1, 1);
      o.ln2_b = pk.add("ln2_b", l, m.d, 1, 1);
      o.w_up = pk.add("wfc", l, m.ff, m.d, 2);
      o.b_up = pk.add("bfc", l, m.ff, 1, 1);
      o.w_down = pk.add("wproj", l, m.d, m.ff, 2);
      o.b_down = pk.add("bproj", l, m.d, 1, 1);
    }
  }
}

// Every factor's element count is a multiple of 64 (the stored rank and the
// widths are multiples of 8, d and ff of 64), so stacked factors are
// contiguous.  A rank that is not a multiple of 8 is stored padded to the
// next one (16-byte factor rows for the bf16 GEMMs): A [lr, in] with rows
// lq.. zero, B [out, lr] with columns lq.. zero.
void lora_tensors(const Dims& m, Packer& pk, std::vector<LoraOff>& lora) {
  const int r = m.lr;
  lora.resize(m.L);
  for (int l = 0; l < m.L; ++l) {
    LoraOff& o = lora[l];
    if (m.llama) {
      o.qkv_a = pk.add("wq_la", l, r, m.d, 2);
      pk.add("wk_la", l, r, m.d, 2);
      pk.add("wv_la", l, r, m.d, 2);
      o.qkv_b = pk.add("wq_lb", l, m.dq, r, 2);
      pk.add("wk_lb", l, m.dkv, r, 2);
      pk.add("wv_lb", l, m.dkv, r, 2);
      o.o_a = pk.add("wo_la", l, r, m.dq, 2);
      o.o_b = pk.add("wo_lb", l, m.d, r, 2);
      o.up_a = pk.add("wg_la", l, r, m.d, 2);
      pk.add("wu_la", l, r, m.d, 2);
      o.up_b = pk.add("wg_lb", l, m.ff, r, 2);
      pk.add("wu_lb", l, m.ff, r, 2);
      o.down_a = pk.add("wd_la", l, r, m.ff, 2);
      o.down_b = pk.add("wd_lb", l, m.d, r, 2);
    } else {
      o.qkv_a = pk.add("wqkv_la", l, r, m.d, 2);
      o.qkv_b = pk.add("wqkv_lb", l, m.nqkv, r, 2);
      o.o_a = pk.add("wo_la", l, r, m.dq, 2);
      o.o_b = pk.add("wo_lb", l, m.d, r, 2);
      o.up_a = pk.add("wfc_la", l, r, m.d, 2);
      o.up_b = pk.add("wfc_lb", l, m.ff, r, 2);
      o.down_a = pk.add("wproj_la", l, r, m.ff, 2);
      o.down_b = pk.add("wproj_lb", l, m.d, r, 2);
    }
  }
}

void build_layout(const zl_config& c, Layout& out) {
  const Dims m = dims_of(c);
  Packer pk{&out.descs};
  if (m.lr) {
    Packer base{nullptr};
    layer_tensors(m, base, out.lay);
    out.n_base = base.off;
    lora_tensors(m, pk, out.lora);
  } else {
    layer_tensors(m, pk, out.lay);
  }
  if (m.ar) {
    out.ad_w1 = pk.add("ad_w1", m.L, m.ar, m.d, 2);
    out.ad_w2 = pk.add("ad_w2", m.L, m.d, m.ar, 2);
  }
  out.n_params = pk.off;
}

// Workspace plan: byte offsets of every region, 256-byte aligned.
struct Plan {
  size_t total = 0;
  int Tmax = 0, R = 0, Vpad = 0, stk = 1;
  size_t rope, seqlens, pos;
  std::vector<size_t> X;  // L + 1
  std::vector<size_t> N1, RS1, MU1, QKV, O, LSE, X2, N2, RS2, MU2, UP, ACT;
  size_t DX, DXA, DXB, DUP, DN, DO, DQKV, DELTA, PART;
  size_t HN, HRS, HMU, ZC, HST, ZY, DZ, DNF, ROWLOSS, NOMEGA;
  int nst;  // 64-column blocks of a logit row (softmax partials, bf16 path)
  // readout adapter: act copy of h_out, pre-activation, activation, h',
  // dL/dh' (fp32 and act), dL/dU
  size_t AXO, AU, AG, AHP, ADHP, ADHPA, ADU;
  // LoRA: s x A^T of each projection per layer (act), the block-diagonal
  // B factors of the projection being computed (act), and s (dy B) (act)
  std::vector<size_t> LXQ, LXO, LXU, LXD;
  size_t LBD, LE;
  size_t part_elems;
  size_t SPK, spk_elems;  // split-K partials of the GEMMs
};

void build_plan(const zl_config& c, Plan& p) {
  const Dims m = dims_of(c);
  const size_t act = c.dtype == ZL_BF16 ? 2 : 4;
  const size_t T = (size_t)c.max_batch * c.max_seq;
  p.Tmax = (int)T;
  p.R = (int)(T < 4096 ? T : 4096);
  p.Vpad = (int)round_up((size_t)m.V, 8);
  p.stk = c.alpha < 1.f ? 2 : 1;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = round_up(off + (bytes ? bytes : 1), ALIGN_BYTES);
    return at;
  };
  p.rope = take(m.llama ? (size_t)c.max_seq * (m.hd / 2) * 8 : 0);
  p.seqlens = take((size_t)c.max_batch * 4);
  p.pos = take(T * 4);
  p.X.resize(m.L + 1);
  p.N1.resize(m.L); p.RS1.resize(m.L); p.MU1.resize(m.L); p.QKV.resize(m.L); p.O.resize(m.L);
  p.LSE.resize(m.L); p.X2.resize(m.L); p.N2.resize(m.L); p.RS2.resize(m.L); p.MU2.resize(m.L);
  p.UP.resize(m.L); p.ACT.resize(m.L);
  for (int l = 0; l < m.L; ++l) {
    p.X[l] = take(T * m.d * 4);
    p.N1[l] = take(T * m.d * act);
    p.RS1[l] = take(T * 4);
    p.MU1[l] = take(m.llama ? 0 : T * 4);
    p.QKV[l] = take(T * m.nqkv * act);
    p.O[l] = take(T * m.dq * act);
    p.LSE[l] = take(T * m.hq * 4);
    p.X2[l] = take(T * m.d * 4);
    p.N2[l] = take(T * m.d * act);
    p.RS2[l] = take(T * 4);
    p.MU2[l] = take(m.llama ? 0 : T * 4);
    p.UP[l] = take(T * m.nup * act);
    p.ACT[l] = take(T * m.ff * act);
  }
  p.X[m.L] = take(T * m.d * 4);
  p.DX = take(T * m.d * 4);
  p.DXA = take(T * m.d * act);
  p.DXB = take(T * m.d * act);
  p.DUP = take(T * m.nup * act);
  p.DN = take(T * m.d * 4);
  p.DO = take(T * m.dq * act);
  p.DQKV = take(T * m.nqkv * act);
  p.DELTA = take(T * m.hq * 4);
  size_t pe = (size_t)2 * norm_bwd_blocks((int)T) * m.d;
  size_t widest = m.nqkv > m.ff ? m.nqkv : m.ff;
  if (m.d > (int)widest) widest = m.d;
  const size_t pc = (size_t)colsum_blocks((int)T) * widest;
  p.part_elems = pe > pc ? pe : pc;
  p.PART = take(p.part_elems * 4);
  const size_t R = p.R, S2 = (size_t)p.stk * R;
  p.HN = take(S2 * m.d * act);
  p.HRS = take(S2 * 4);
  p.HMU = take(S2 * 4);
  p.ZC = take(S2 * p.Vpad * (act == 2 ? 2 : 4));  // fp16 logits in the bf16 path
  p.nst = (m.V + 63) / 64;
  p.HST = take(act == 2 ? S2 * p.nst * 16 : 0);
  p.ZY = take(act == 2 ? R * 4 : 0);
  p.DZ = take(R * p.Vpad * act);
  p.DNF = take(R * m.d * 4);
  p.ROWLOSS = take(T * 4);
  p.NOMEGA = take(4);
  const size_t ar = (size_t)m.ar;
  p.AXO = take(ar && act == 2 ? T * m.d * act : 0);
  p.AU = take(T * ar * act);
  p.AG = take(T * ar * act);
  p.AHP = take(ar ? T * m.d * 4 : 0);
  p.ADHP = take(ar ? T * m.d * 4 : 0);
  p.ADHPA = take(ar ? T * m.d * act : 0);
  p.ADU = take(T * ar * act);
  const size_t lr = (size_t)m.lr;
  p.LXQ.resize(m.L); p.LXO.resize(m.L); p.LXU.resize(m.L); p.LXD.resize(m.L);
  for (int l = 0; l < m.L; ++l) {
    p.LXQ[l] = take(T * m.nqa * act);
    p.LXO[l] = take(T * lr * act);
    p.LXU[l] = take(T * m.nua * act);
    p.LXD[l] = take(T * lr * act);
  }
  const size_t bd_q = (size_t)m.nqkv * m.nqa, bd_u = (size_t)m.nup * m.nua;
  p.LBD = take(lr && m.llama ? (bd_q > bd_u ? bd_q : bd_u) * act : 0);
  p.LE = take(T * m.nqa * act);
  // split-K partials (bf16 GEMMs whose outputs hold too few tiles to fill
  // the chip: the LoRA factor GEMMs); launch_gemm splits less if they do
  // not fit
  p.spk_elems = act == 2 ? (size_t)4 << 20 : 0;
  p.SPK = take(p.spk_elems * 4);
  p.total = off;
}

enum State { ST_IDLE = 0, ST_FORWARD = 1, ST_OBJECTIVE = 2 };

}  // namespace

struct zl_chunk {
  zl_config cfg;
  zl_buffers buf;
  Dims m;
  Layout layout;
  Plan plan;
  char* ws;
  int act;          // activation dtype (F32/BF16)
  int state;        // State
  bool has_grad;    // a backward ran since the last step
  bool grad_fresh;  // next backward overwrites the gradient
  int64_t step;
  int B, S, T;
  // profiling (zl_profile_begin / zl_profile_end)
  struct Rec { const char* name; double flops, bytes; };
  bool prof_on = false;
  std::vector<hipEvent_t> prof_ev;  // 2 per record
  std::vector<Rec> prof_rec;
  size_t prof_used = 0;

  int prof_start(hipStream_t s) {
    if (!prof_on || prof_used >= prof_rec.size()) return -1;
    const int i = (int)prof_used++;
    hipEventRecord(prof_ev[2 * i], s);
    return i;
  }
  void prof_cancel(int i) {  // the last prof_start recorded nothing worth keeping
    if (i >= 0 && (size_t)i + 1 == prof_used) --prof_used;
  }
  void prof_stop(int i, hipStream_t s, const char* name, double flops, double bytes) {
    if (i < 0) return;
    hipEventRecord(prof_ev[2 * i + 1], s);
    prof_rec[i] = {name, flops, bytes};
  }

  template <typename P> P* at(size_t off) const { return reinterpret_cast<P*>(ws + off); }
  // Layer tensors live in the trainable buffers, or in the frozen base
  // buffers with LoRA; the adapter and LoRA factors in the trainable ones.
  const void* W(size_t off) const {  // a layer weight matrix as the kernels consume it
    if (act == BF16)
      return reinterpret_cast<const bf16_t*>(m.lr ? buf.base_shadow : buf.shadow) + off;
    return V32(off);
  }
  const float* V32(size_t off) const { return (m.lr ? buf.base_master : buf.master) + off; }
  const void* WT(size_t off) const {  // a trainable matrix (adapter, LoRA factor)
    if (act == BF16) return reinterpret_cast<const bf16_t*>(buf.shadow) + off;
    return buf.master + off;
  }
  float* G(size_t off) const { return buf.grad + off; }
  size_t asz() const { return act == BF16 ? 2 : 4; }
  void* A(size_t base_off, size_t elem_off) const { return ws + base_off + elem_off * asz(); }
};

static hipStream_t S_(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ------------------------------------------------------------ GEMM helpers
static GemmDesc gdesc(int M, int N, int K, const void* A, int64_t lda, bool ak, const void* B,
                      int64_t ldb, bool bk) {
  GemmDesc g;
  g.M = M; g.N = N; g.K = K; g.ka = K; g.kb = K;
  g.A = A; g.lda = lda; g.a_kmajor = ak;
  g.B = B; g.ldb = ldb; g.b_kmajor = bk;
  g.K2 = 0; g.A2 = nullptr; g.lda2 = 0; g.B2 = nullptr; g.ldb2 = 0;
  g.part = nullptr; g.part_elems = 0; g.ksplit = K;
  return g;
}

static EpiArgs epi(EpiKind k, void* out, int64_t ldo, int dt) {
  EpiArgs e;
  memset(&e, 0, sizeof(e));
  e.kind = k; e.out = out; e.ldo = ldo; e.out_dtype = dt; e.scale = 1.f;
  return e;
}

// Launch wrappers that time the launch when profiling is on.
static hipError_t run_gemm(zl_chunk* c, hipStream_t s, const GemmDesc& g, const EpiArgs& e,
                           double k_alg = -1) {
  const int pi = c->prof_start(s);
  const char* kn = "gemm";
  GemmDesc gs = g;
  if (!gs.part) {
    gs.part = c->plan.spk_elems ? c->at<float>(c->plan.SPK) : nullptr;
    gs.part_elems = c->plan.spk_elems;
  }
  hipError_t err = launch_gemm(gs, e, c->act, s, &kn);
  c->prof_stop(pi, s, kn, 2.0 * g.M * g.N * ((k_alg < 0 ? g.K : k_alg) + g.K2), 0.0);
  return err;
}

// Two independent GEMMs: one launch when they share a kernel, else one
// after the other.
static hipError_t run_gemm_pair(zl_chunk* c, hipStream_t s, const GemmDesc& g1, const EpiArgs& e1,
                                const GemmDesc& g2, const EpiArgs& e2) {
  const int pi = c->prof_start(s);
  const char* kn = "gemm";
  GemmDesc a = g1, b = g2;
  a.part = b.part = c->plan.spk_elems ? c->at<float>(c->plan.SPK) : nullptr;
  a.part_elems = b.part_elems = c->plan.spk_elems;
  bool fused = false;
  hipError_t err = launch_gemm_pair(a, e1, b, e2, c->act, s, &fused, &kn);
  if (fused || err != hipSuccess) {
    c->prof_stop(pi, s, kn, 2.0 * g1.M * g1.N * (g1.K + g1.K2) + 2.0 * g2.M * g2.N * (g2.K + g2.K2),
                 0.0);
    return err;
  }
  c->prof_cancel(pi);
  err = run_gemm(c, s, g1, e1);
  return err == hipSuccess ? run_gemm(c, s, g2, e2) : err;
}

#define ZL_RUN(name, flops, bytes, call)                                             \
  do {                                                                              \
    const int pi_ = c->prof_start(s);                                               \
    hipError_t e_ = (call);                                                         \
    c->prof_stop(pi_, s, name, (double)(flops), (double)(bytes));                   \
    if (e_ != hipSuccess)                                                           \
      return fail(ZL_ERR_HIP, std::string(#call) + ": " + hipGetErrorString(e_));   \
  } while (0)

// ---------------------------------------------------------------- public
extern "C" {

const char* zl_status_string(zl_status s) {
  switch (s) {
    case ZL_OK: return "ZL_OK";
    case ZL_ERR_INVALID_ARG: return "ZL_ERR_INVALID_ARG";
    case ZL_ERR_UNSUPPORTED: return "ZL_ERR_UNSUPPORTED";
    case ZL_ERR_HIP: return "ZL_ERR_HIP";
    case ZL_ERR_STATE: return "ZL_ERR_STATE";
    case ZL_ERR_WORKSPACE: return "ZL_ERR_WORKSPACE";
  }
  return "unknown zl_status";
}

const char* zl_last_error(void) { return g_err.c_str(); }

zl_status zl_param_layout(const zl_config* cfg, size_t* n_params, zl_tensor_desc* descs,
                          int* n_descs) {
  zl_status st = check_config(cfg);
  if (st != ZL_OK) return st;
  if (!n_params) return fail(ZL_ERR_INVALID_ARG, "n_params is NULL");
  Layout L;
  build_layout(*cfg, L);
  *n_params = L.n_params;
  if (descs) {
    if (!n_descs) return fail(ZL_ERR_INVALID_ARG, "n_descs is NULL");
    if (*n_descs < (int)L.descs.size())
      return fail(ZL_ERR_INVALID_ARG, "descs array too small: need " +
                                          std::to_string(L.descs.size()));
    memcpy(descs, L.descs.data(), L.descs.size() * sizeof(zl_tensor_desc));
  }
  if (n_descs) *n_descs = (int)L.descs.size();
  return ZL_OK;
}

zl_status zl_workspace_size(const zl_config* cfg, size_t* bytes) {
  zl_status st = check_config(cfg);
  if (st != ZL_OK) return st;
  if (!bytes) return fail(ZL_ERR_INVALID_ARG, "bytes is NULL");
  Plan p;
  build_plan(*cfg, p);
  *bytes = p.total;
  return ZL_OK;
}

zl_status zl_chunk_create(const zl_config* cfg, const zl_buffers* bufs, void* workspace,
                          size_t ws_bytes, zl_chunk** out) {
  if (!out) return fail(ZL_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  zl_status st = check_config(cfg);
  if (st != ZL_OK) return st;
  if (!bufs) return fail(ZL_ERR_INVALID_ARG, "bufs is NULL");
  if (!bufs->master || !bufs->grad) return fail(ZL_ERR_INVALID_ARG, "master and grad required");
  if (cfg->dtype == ZL_BF16 && !bufs->shadow)
    return fail(ZL_ERR_INVALID_ARG, "bf16 mode needs a shadow buffer");
  if (cfg->optimizer == ZL_ADAMW && (!bufs->adam_m || !bufs->adam_v))
    return fail(ZL_ERR_INVALID_ARG, "AdamW needs adam_m and adam_v");
  if (!bufs->head_w || !bufs->head_norm_w)
    return fail(ZL_ERR_INVALID_ARG, "head_w and head_norm_w required");
  if (cfg->arch == ZL_ARCH_GPT2 && !bufs->head_norm_b)
    return fail(ZL_ERR_INVALID_ARG, "gpt2 needs head_norm_b");
  if (cfg->lora_rank && !bufs->base_master)
    return fail(ZL_ERR_INVALID_ARG, "LoRA mode needs base_master");
  if (cfg->lora_rank && cfg->dtype == ZL_BF16 && !bufs->base_shadow)
    return fail(ZL_ERR_INVALID_ARG, "LoRA in bf16 mode needs base_shadow");
  const uintptr_t al = (uintptr_t)bufs->master | (uintptr_t)bufs->grad |
                       (uintptr_t)bufs->head_w | (uintptr_t)(bufs->shadow) |
                       (uintptr_t)bufs->adam_m | (uintptr_t)bufs->adam_v |
                       (uintptr_t)bufs->base_master | (uintptr_t)bufs->base_shadow;
  if (al % 16) return fail(ZL_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
  Plan p;
  build_plan(*cfg, p);
  if (!workspace) return fail(ZL_ERR_WORKSPACE, "workspace is NULL");
  if ((uintptr_t)workspace % ALIGN_BYTES)
    return fail(ZL_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < p.total)
    return fail(ZL_ERR_WORKSPACE, "workspace too small: need " + std::to_string(p.total));
  zl_chunk* c = new (std::nothrow) zl_chunk();
  if (!c) return fail(ZL_ERR_INVALID_ARG, "out of host memory");
  c->cfg = *cfg;
  c->buf = *bufs;
  c->m = dims_of(*cfg);
  build_layout(*cfg, c->layout);
  c->plan = p;
  c->ws = reinterpret_cast<char*>(workspace);
  c->act = cfg->dtype == ZL_BF16 ? BF16 : F32;
  c->state = ST_IDLE;
  c->has_grad = false;
  c->grad_fresh = true;
  c->step = 0;
  c->B = c->S = c->T = 0;
  if (c->m.llama) {
    hipError_t e = launch_rope_table(c->at<float2>(p.rope), cfg->max_seq, c->m.hd / 2,
                                     (double)cfg->rope_theta, nullptr);
    if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
    if (e != hipSuccess) {
      delete c;
      return fail(ZL_ERR_HIP, std::string("rope table: ") + hipGetErrorString(e));
    }
  }
  *out = c;
  return ZL_OK;
}

void zl_chunk_destroy(zl_chunk* chunk) {
  if (!chunk) return;
  for (hipEvent_t e : chunk->prof_ev) hipEventDestroy(e);
  delete chunk;
}

zl_status zl_refresh_shadow(zl_chunk* c, void* stream) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "chunk is NULL");
  if (c->m.lq < c->m.lr) {
    // the padding of factors stored wider than their rank is zero: then its
    // gradient is exactly zero and no step moves it
    for (const zl_tensor_desc& t : c->layout.descs) {
      const size_t nl = strlen(t.name);
      if (nl < 3 || t.name[nl - 3] != '_' || t.name[nl - 2] != 'l') continue;
      const bool a = t.name[nl - 1] == 'a';
      const int64_t rows = t.shape[0], cols = t.shape[1];
      ZL_HIP(launch_zero_block(c->buf.master + t.offset, cols, a ? c->m.lq : 0, rows,
                               a ? 0 : c->m.lq, cols, S_(stream)));
    }
  }
  if (c->act != BF16) return ZL_OK;
  ZL_HIP(launch_shadow(c->buf.master, reinterpret_cast<bf16_t*>(c->buf.shadow),
                       c->layout.n_params, S_(stream)));
  if (c->m.lr)
    ZL_HIP(launch_shadow(c->buf.base_master, reinterpret_cast<bf16_t*>(c->buf.base_shadow),
                         c->layout.n_base, S_(stream)));
  return ZL_OK;
}

zl_status zl_get_step(const zl_chunk* c, int64_t* step) {
  if (!c || !step) return fail(ZL_ERR_INVALID_ARG, "NULL argument");
  *step = c->step;
  return ZL_OK;
}

zl_status zl_set_step(zl_chunk* c, int64_t step) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "chunk is NULL");
  if (step < 0) return fail(ZL_ERR_INVALID_ARG, "step must be >= 0");
  c->step = step;
  return ZL_OK;
}

}  // extern "C"

namespace zl {
zl_status set_error(zl_status s, const std::string& msg) { return fail(s, msg); }
bool chunk_at_boundary(const zl_chunk* c) { return c->state == ST_IDLE && !c->has_grad; }
void chunk_close_window(zl_chunk* c) {
  c->state = ST_IDLE;
  c->has_grad = false;
  c->grad_fresh = true;
}
}  // namespace zl

extern "C" {

zl_status zl_chunk_get_config(const zl_chunk* c, zl_config* out) {
  if (!c || !out) return fail(ZL_ERR_INVALID_ARG, "NULL argument");
  *out = c->cfg;
  return ZL_OK;
}

zl_status zl_chunk_get_buffers(const zl_chunk* c, zl_buffers* out) {
  if (!c || !out) return fail(ZL_ERR_INVALID_ARG, "NULL argument");
  *out = c->buf;
  return ZL_OK;
}

zl_status zl_chunk_num_params(const zl_chunk* c, size_t* n) {
  if (!c || !n) return fail(ZL_ERR_INVALID_ARG, "NULL argument");
  *n = c->layout.n_params;
  return ZL_OK;
}

// --------------------------------------------------------------- forward
zl_status zl_chunk_forward(zl_chunk* c, const void* h_in, const int32_t* seq_lens,
                           const int32_t* pos_ids, int B, int S, void* h_out, void* stream) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "chunk is NULL");
  if (!h_in || !h_out) return fail(ZL_ERR_INVALID_ARG, "h_in and h_out required");
  if (h_in == h_out) return fail(ZL_ERR_INVALID_ARG, "h_out must not alias h_in");
  if (B < 1 || S < 1 || B > c->cfg.max_batch || S > c->cfg.max_seq)
    return fail(ZL_ERR_INVALID_ARG, "B or S out of range");
  if (((uintptr_t)h_in | (uintptr_t)h_out) % 16)
    return fail(ZL_ERR_INVALID_ARG, "h_in and h_out must be 16-byte aligned");
  hipStream_t s = S_(stream);
  const Dims& m = c->m;
  const Plan& p = c->plan;
  const int T = B * S;
  const int act = c->act;
  const bool ln = !m.llama;
  const float eps = c->cfg.norm_eps;
  int32_t* sl = c->at<int32_t>(p.seqlens);
  int32_t* pos = c->at<int32_t>(p.pos);
  ZL_RUN("copy_inputs", 0, B * 8, launch_copy_i32(seq_lens, sl, B, 1, 0, S, s));
  ZL_RUN("copy_inputs", 0, (double)T * 8, launch_copy_i32(pos_ids, pos, T, 1, 1, S, s));
  ZL_RUN("cast", 0, (double)T * m.d * (4 + c->asz()), launch_cast(h_in, act, c->at<float>(p.X[0]), F32, (size_t)T * m.d, s));
  // LoRA (Delta w_l = B_l A_l of Sec. II.A on the frozen w_l): for the
  // projections reading x, xa = s x A^T over their stacked A factors
  // [na, in]; the projection's GEMM then takes xa and its B factors as a
  // second K segment, y = x W^T + xa B^T, in the same accumulators (before
  // bias, RoPE, activation or residual).  Projections sharing x (q/k/v,
  // gate/up) each see only their own block of xa: their B factors are
  // expanded block-diagonally to [out, na].
  const int r = m.lr;
  auto lora_fwd = [&](const void* x, int in, size_t a_off, int na, void* xa, size_t b_off,
                      int nblk, const int* widths, int out, GemmDesc& g) -> hipError_t {
    EpiArgs ea = epi(EPI_STORE, xa, na, act);
    ea.scale = m.ls;
    hipError_t err = run_gemm(c, s, gdesc(T, na, in, x, in, true, c->WT(a_off), in, true), ea);
    const void* b2 = c->WT(b_off);
    if (err == hipSuccess && nblk > 1) {
      void* bd = c->ws + p.LBD;
      const int b1 = widths[0], bnd2 = nblk > 2 ? widths[0] + widths[1] : out;
      const int pi = c->prof_start(s);
      err = launch_blockdiag(b2, bd, act, out, r, nblk, b1, bnd2, s);
      c->prof_stop(pi, s, "lora_blockdiag", 0, (double)out * (r + na) * c->asz());
      b2 = bd;
    }
    g.K2 = na; g.A2 = xa; g.lda2 = na; g.B2 = b2; g.ldb2 = na;
    return err;
  };
  const int w_qkv[3] = {m.dq, m.dkv, m.dkv}, w_up[2] = {m.ff, m.ff};
  const int n_qkv = m.llama ? 3 : 1, n_up = m.llama ? 2 : 1;
  for (int l = 0; l < m.L; ++l) {
    const LayerOff& o = c->layout.lay[l];
    const LoraOff* lo = r ? &c->layout.lora[l] : nullptr;
    float* X = c->at<float>(p.X[l]);
    float* X2 = c->at<float>(p.X2[l]);
    void* N1 = c->ws + p.N1[l];
    void* N2 = c->ws + p.N2[l];
    void* QKV = c->ws + p.QKV[l];
    void* O = c->ws + p.O[l];
    void* UP = c->ws + p.UP[l];
    void* ACT = c->ws + p.ACT[l];
    ZL_RUN("norm_fwd", 0, (double)T * m.d * (4 + c->asz()), launch_norm_fwd(ln, X, m.d, c->V32(o.ln1_w), ln ? c->V32(o.ln1_b) : nullptr, N1, m.d,
                           act, ln ? c->at<float>(p.MU1[l]) : nullptr, c->at<float>(p.RS1[l]),
                           T, m.d, eps, s));
    // bf16: RoPE is applied in the QKV GEMM epilogue (one rounding of q, k)
    const bool rope_in_gemm = m.llama && act == BF16 && m.hd <= 128;
    {
      EpiArgs e = epi(rope_in_gemm ? EPI_ROPE : EPI_STORE, QKV, m.nqkv, act);
      e.bias = ln ? c->V32(o.b_qkv) : nullptr;
      if (rope_in_gemm) {
        e.pos = pos; e.rope = c->at<float2>(p.rope); e.max_pos = c->cfg.max_seq;
        e.hd = m.hd; e.n_rot = (m.hq + m.hkv) * m.hd;
      }
      GemmDesc g = gdesc(T, m.nqkv, m.d, N1, m.d, true, c->W(o.w_qkv), m.d, true);
      if (r) ZL_HIP(lora_fwd(N1, m.d, lo->qkv_a, m.nqa, c->ws + p.LXQ[l], lo->qkv_b, n_qkv, w_qkv, m.nqkv, g));
      ZL_HIP(run_gemm(c, s, g, e));
    }
    if (m.llama && !rope_in_gemm)
      ZL_RUN("rope", 0, 2.0 * T * (m.hq + m.hkv) * m.hd * c->asz(),
             launch_rope(QKV, m.nqkv, act, pos, c->at<float2>(p.rope), c->cfg.max_seq, T,
                         m.hq + m.hkv, m.hd, +1, s));
    {
      AttnDesc a;
      memset(&a, 0, sizeof(a));
      a.B = B; a.S = S; a.Hq = m.hq; a.Hkv = m.hkv; a.hd = m.hd;
      a.q = QKV; a.k = c->A(p.QKV[l], m.dq); a.v = c->A(p.QKV[l], m.dq + m.dkv);
      a.ldq = a.ldk = a.ldv = m.nqkv;
      a.o = O; a.ldo = m.dq;
      a.lse = c->at<float>(p.LSE[l]);
      a.seq_lens = sl;
      a.scale = 1.f / sqrtf((float)m.hd);
      ZL_RUN("attn_fwd", 2.0 * B * m.hq * m.hd * (double)S * (S + 1), 0, launch_attn_fwd(a, act, s));
    }
    {
      EpiArgs e = epi(EPI_RESID, X2, m.d, F32);
      e.resid = X; e.ldr = m.d;
      e.bias = ln ? c->V32(o.b_o) : nullptr;
      GemmDesc g = gdesc(T, m.d, m.dq, O, m.dq, true, c->W(o.w_o), m.dq, true);
      if (r) ZL_HIP(lora_fwd(O, m.dq, lo->o_a, r, c->ws + p.LXO[l], lo->o_b, 1, nullptr, m.d, g));
      ZL_HIP(run_gemm(c, s, g, e));
    }
    ZL_RUN("norm_fwd", 0, (double)T * m.d * (4 + c->asz()), launch_norm_fwd(ln, X2, m.d, c->V32(o.ln2_w), ln ? c->V32(o.ln2_b) : nullptr, N2, m.d,
                           act, ln ? c->at<float>(p.MU2[l]) : nullptr, c->at<float>(p.RS2[l]),
                           T, m.d, eps, s));
    if (m.llama) {
      EpiArgs e = epi(EPI_STORE, UP, m.nup, act);
      GemmDesc g = gdesc(T, m.nup, m.d, N2, m.d, true, c->W(o.w_up), m.d, true);
      if (r) ZL_HIP(lora_fwd(N2, m.d, lo->up_a, m.nua, c->ws + p.LXU[l], lo->up_b, n_up, w_up, m.nup, g));
      ZL_HIP(run_gemm(c, s, g, e));
      ZL_RUN("swiglu_fwd", 0, 3.0 * T * m.ff * c->asz(), launch_swiglu_fwd(UP, m.nup, ACT, m.ff, act, T, m.ff, s));
    } else {
      EpiArgs e = epi(EPI_GELU, ACT, m.ff, act);
      e.out2 = UP; e.ldo2 = m.nup;
      e.bias = c->V32(o.b_up);
      GemmDesc g = gdesc(T, m.ff, m.d, N2, m.d, true, c->W(o.w_up), m.d, true);
      if (r) ZL_HIP(lora_fwd(N2, m.d, lo->up_a, m.nua, c->ws + p.LXU[l], lo->up_b, 1, nullptr, m.ff, g));
      ZL_HIP(run_gemm(c, s, g, e));
    }
    {
      EpiArgs e = epi(EPI_RESID, c->at<float>(p.X[l + 1]), m.d, F32);
      e.resid = X2; e.ldr = m.d;
      e.bias = ln ? c->V32(o.b_down) : nullptr;
      GemmDesc g = gdesc(T, m.d, m.ff, ACT, m.ff, true, c->W(o.w_down), m.ff, true);
      if (r) ZL_HIP(lora_fwd(ACT, m.ff, lo->down_a, r, c->ws + p.LXD[l], lo->down_b, 1, nullptr, m.d, g));
      ZL_HIP(run_gemm(c, s, g, e));
    }
  }
  ZL_RUN("cast", 0, (double)T * m.d * (4 + c->asz()), launch_cast(c->at<float>(p.X[m.L]), F32, h_out, act, (size_t)T * m.d, s));
  c->B = B; c->S = S; c->T = T;
  c->state = ST_FORWARD;
  return ZL_OK;
}

// ------------------------------------------------------------- objective
zl_status zl_local_objective(zl_chunk* c, const int32_t* labels, float* loss_out, void* stream) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "chunk is NULL");
  if (!labels || !loss_out) return fail(ZL_ERR_INVALID_ARG, "labels and loss_out required");
  if (c->state != ST_FORWARD && c->state != ST_OBJECTIVE)
    return fail(ZL_ERR_STATE, "zl_local_objective needs a preceding zl_chunk_forward");
  hipStream_t s = S_(stream);
  const Dims& m = c->m;
  const Plan& p = c->plan;
  const int T = c->T;
  const int act = c->act;
  const bool ln = !m.llama;
  const int stk = p.stk;
  float* nomega = c->at<float>(p.NOMEGA);
  ZL_RUN("count_omega", 0, (double)T * 4, launch_count_omega(labels, T, m.V, nomega, s));
  const float* hout = c->at<float>(p.X[m.L]);
  const float* hin = c->at<float>(p.X[0]);
  // readout adapter (Sec. III-B (b)): h_out is read out as
  // h' = h_out + gelu(h_out W1^T) W2^T; h_in keeps the static head
  float* dh_read = c->at<float>(p.DX);  // dL/d(read-out rows of h_out)
  void* dh_read_a = c->ws + p.DXA;
  if (m.ar) {
    const void* xo = hout;
    if (act == BF16) {
      ZL_RUN("cast", 0, (double)T * m.d * 6, launch_cast(hout, F32, c->ws + p.AXO, BF16, (size_t)T * m.d, s));
      xo = c->ws + p.AXO;
    }
    {
      EpiArgs e = epi(EPI_GELU, c->ws + p.AG, m.ar, act);
      e.out2 = c->ws + p.AU;
      e.ldo2 = m.ar;
      ZL_HIP(run_gemm(c, s, gdesc(T, m.ar, m.d, xo, m.d, true, c->WT(c->layout.ad_w1), m.d, true), e));
    }
    {
      EpiArgs e = epi(EPI_RESID, c->at<float>(p.AHP), m.d, F32);
      e.resid = hout;
      e.ldr = m.d;
      ZL_HIP(run_gemm(c, s, gdesc(T, m.d, m.ar, c->ws + p.AG, m.ar, true, c->WT(c->layout.ad_w2), m.ar,
                               true), e));
    }
    hout = c->at<float>(p.AHP);
    dh_read = c->at<float>(p.ADHP);
    dh_read_a = c->ws + p.ADHPA;
  }
  for (int r0 = 0; r0 < T; r0 += p.R) {
    const int rows = T - r0 < p.R ? T - r0 : p.R;
    ZL_RUN("head_norm", 0, (double)stk * rows * m.d * (4 + c->asz()), launch_head_norm(ln, hout, stk == 2 ? hin : nullptr, m.d, r0, rows,
                            c->buf.head_norm_w, c->buf.head_norm_b, c->ws + p.HN, act,
                            ln ? c->at<float>(p.HMU) : nullptr, c->at<float>(p.HRS), m.d,
                            c->cfg.norm_eps, s));
    {
      // bf16: the GEMM's epilogue also leaves per-row softmax partials of
      // 64-column blocks (z rows paired with their z' rows), which replace
      // the objective's statistics pass over the logits, and the fp32 logit
      // of each label; the cached logits are then fp16 (they only form
      // dL/dz)
      const bool fused = act == BF16;
      EpiArgs e = epi(fused ? EPI_LOGITS : EPI_STORE, c->ws + p.ZC, p.Vpad, fused ? F16 : F32);
      if (fused) {
        e.stats = c->at<float4>(p.HST);
        e.ldst = p.nst;
        e.pair = stk == 2;
        e.lab = labels + r0;
        e.zy = c->at<float>(p.ZY);
      }
      ZL_HIP(run_gemm(c, s, gdesc(stk * rows, m.V, m.d, c->ws + p.HN, m.d, true, c->buf.head_w, m.d,
                               true), e));
    }
    {
      ObjDesc o;
      o.zc = c->ws + p.ZC; o.ldz = p.Vpad; o.stacked = stk;
      o.z_dtype = act == BF16 ? F16 : F32;
      o.zy = act == BF16 ? c->at<float>(p.ZY) : nullptr;
      o.labels = labels + r0; o.rows = rows; o.V = m.V; o.Vpad = p.Vpad;
      o.alpha = c->cfg.alpha; o.consis = c->cfg.consis; o.n_omega = nomega;
      o.dz = c->ws + p.DZ; o.lddz = p.Vpad; o.dz_dtype = act;
      o.row_loss = c->at<float>(p.ROWLOSS) + r0;
      o.stats = act == BF16 ? c->at<float4>(p.HST) : nullptr;
      o.ldst = p.nst;
      o.nst = p.nst;
      ZL_RUN("objective_rows", 0, (double)rows * (stk * (act == BF16 ? 2.0 : 4.0) * m.V + c->asz() * p.Vpad), launch_objective_rows(o, s));
    }
    {
      GemmDesc g = gdesc(rows, m.d, p.Vpad, c->ws + p.DZ, p.Vpad, true, c->buf.head_w, m.d, false);
      g.kb = m.V;
      if (act == BF16) {
        // the logit cache is free once the objective has formed dZ: it
        // holds the split-K partials when rows x d is too few tiles
        g.part = c->at<float>(p.ZC);
        g.part_elems = (size_t)stk * p.R * p.Vpad * 2 / 4;
      }
      EpiArgs e = epi(EPI_STORE, c->at<float>(p.DNF), m.d, F32);
      ZL_HIP(run_gemm(c, s, g, e, (double)m.V));
    }
    ZL_RUN("head_norm_bwd", 0, (double)rows * m.d * (12 + c->asz()), launch_head_norm_bwd(ln, c->at<float>(p.DNF), m.d, hout, c->buf.head_norm_w,
                                ln ? c->at<float>(p.HMU) : nullptr, c->at<float>(p.HRS), stk,
                                dh_read, dh_read_a, act, r0, rows, m.d, s));
  }
  if (m.ar) {
    // dU = gelu'(U) (dh' W2), then dL/dh_out = dh' + dU W1
    {
      EpiArgs e = epi(EPI_GELU_BWD, c->ws + p.ADU, m.ar, act);
      e.aux = c->ws + p.AU;
      e.ldaux = m.ar;
      ZL_HIP(run_gemm(c, s, gdesc(T, m.ar, m.d, c->ws + p.ADHPA, m.d, true, c->WT(c->layout.ad_w2),
                               m.ar, false), e));
    }
    {
      EpiArgs e = epi(EPI_RESID, c->at<float>(p.DX), m.d, F32);
      e.resid = c->at<float>(p.ADHP);
      e.ldr = m.d;
      ZL_HIP(run_gemm(c, s, gdesc(T, m.d, m.ar, c->ws + p.ADU, m.ar, true, c->WT(c->layout.ad_w1), m.d,
                               false), e));
    }
    ZL_RUN("cast", 0, (double)T * m.d * (4 + c->asz()),
           launch_cast(c->at<float>(p.DX), F32, c->ws + p.DXA, act, (size_t)T * m.d, s));
  }
  ZL_RUN("loss_reduce", 0, (double)T * 4, launch_loss_reduce(c->at<float>(p.ROWLOSS), T, nomega, loss_out, s));
  c->state = ST_OBJECTIVE;
  return ZL_OK;
}

// -------------------------------------------------------------- backward
zl_status zl_chunk_backward(zl_chunk* c, float grad_scale, int accumulate, void* stream) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "chunk is NULL");
  if (c->state != ST_OBJECTIVE)
    return fail(ZL_ERR_STATE, "zl_chunk_backward needs a preceding zl_local_objective");
  if (!isfinite(grad_scale)) return fail(ZL_ERR_INVALID_ARG, "grad_scale must be finite");
  hipStream_t s = S_(stream);
  const Dims& m = c->m;
  const Plan& p = c->plan;
  const int T = c->T;
  const int act = c->act;
  const bool ln = !m.llama;
  const int acc = (accumulate && !c->grad_fresh) ? 1 : 0;
  float* DX = c->at<float>(p.DX);
  // MFMA copies of the residual-stream gradient: DXA from the norm-1 backward
  // (or the head) feeds the down projection, DXB from the norm-2 backward the
  // output projection, so the down weight gradient can wait for the QKV one
  void* DXA = c->ws + p.DXA;
  void* DXB = c->ws + p.DXB;
  void* DUP = c->ws + p.DUP;
  float* DN = c->at<float>(p.DN);
  void* DO = c->ws + p.DO;
  void* DQKV = c->ws + p.DQKV;
  float* PART = c->at<float>(p.PART);
  const size_t half_part = p.part_elems / 2;

  auto wgrad = [&](int M, int N, const void* A, int64_t lda, const void* Bm, int64_t ldb,
                   size_t goff) -> hipError_t {
    EpiArgs e = epi(EPI_GRAD, c->G(goff), N, F32);
    e.scale = grad_scale;
    e.accumulate = acc;
    return run_gemm(c, s, gdesc(M, N, T, A, lda, false, Bm, ldb, false), e);
  };
  // Two layer weight gradients in one launch: the tail wave of one is
  // filled with tiles of the other (both read buffers that stay unchanged
  // until the launch, and write disjoint gradients).
  auto wgrad2 = [&](int M1, int N1, const void* A1, int64_t lda1, const void* B1, int64_t ldb1,
                    size_t goff1, int M2, int N2, const void* A2, int64_t lda2, const void* B2,
                    int64_t ldb2, size_t goff2) -> hipError_t {
    EpiArgs e1 = epi(EPI_GRAD, c->G(goff1), N1, F32), e2 = epi(EPI_GRAD, c->G(goff2), N2, F32);
    e1.scale = e2.scale = grad_scale;
    e1.accumulate = e2.accumulate = acc;
    return run_gemm_pair(c, s, gdesc(M1, N1, T, A1, lda1, false, B1, ldb1, false), e1,
                         gdesc(M2, N2, T, A2, lda2, false, B2, ldb2, false), e2);
  };
  auto bias_grad = [&](const void* x, int dt, int n, size_t goff) -> hipError_t {
    int nblk = 0;
    int pi = c->prof_start(s);
    hipError_t e = launch_colsum_partial(x, n, dt, T, n, PART, &nblk, s);
    c->prof_stop(pi, s, "colsum", 0, (double)T * n * (dt == BF16 ? 2 : 4));
    if (e != hipSuccess) return e;
    pi = c->prof_start(s);
    e = launch_reduce_rows(PART, nblk, n, c->G(goff), grad_scale, acc, s);
    c->prof_stop(pi, s, "reduce_rows", 0, 0);
    return e;
  };

  // LoRA backward of projections y_j = x W_j^T + xa_j B_j^T (xa = s x A^T),
  // j over the column blocks of dy [T, out]: E_j = s dy_j B_j into LE
  // [T, na]; the data gradient dy W + E A takes (E, A) as its GEMM's second
  // K segment (when dx is needed); then dA = E^T x and dB_j = dy_j^T xa_j.
  // The frozen W_j get no gradient.
  const int r = m.lr;
  const size_t asz = c->asz();
  void* LE = c->ws + p.LE;
  auto lora_bwd_dx = [&](const void* dy, int out, size_t a_off, int na, size_t b_off,
                         const int* widths, int nblk, int in, bool need_dx,
                         GemmDesc& g) -> hipError_t {
    hipError_t err = hipSuccess;
    int col = 0;
    size_t boff = b_off;
    for (int j = 0; j < nblk && err == hipSuccess; ++j) {
      EpiArgs ee = epi(EPI_STORE, static_cast<char*>(LE) + (size_t)j * r * asz, na, act);
      ee.scale = m.ls;
      err = run_gemm(c, s, gdesc(T, r, widths[j], static_cast<const char*>(dy) + (size_t)col * asz,
                                 out, true, c->WT(boff), r, false), ee);
      col += widths[j];
      boff += (size_t)widths[j] * r;
    }
    if (need_dx) { g.K2 = na; g.A2 = LE; g.lda2 = na; g.B2 = c->WT(a_off); g.ldb2 = in; }
    return err;
  };
  auto lora_bwd_w = [&](const void* dy, int out, const void* x, int in, size_t a_off, int na,
                        const void* xa, size_t b_off, const int* widths, int nblk) -> hipError_t {
    hipError_t err = wgrad(na, in, LE, na, x, in, a_off);
    int col = 0;
    size_t boff = b_off;
    for (int j = 0; j < nblk && err == hipSuccess; ++j) {
      err = wgrad(widths[j], r, static_cast<const char*>(dy) + (size_t)col * asz, out,
                  static_cast<const char*>(xa) + (size_t)j * r * asz, na, boff);
      col += widths[j];
      boff += (size_t)widths[j] * r;
    }
    return err;
  };
  const int w_qkv[3] = {m.dq, m.dkv, m.dkv}, w_qkv1[1] = {m.nqkv};
  const int w_up[2] = {m.ff, m.ff}, w_up1[1] = {m.ff}, w_d[1] = {m.d};
  const int n_qkv = m.llama ? 3 : 1, n_up = m.llama ? 2 : 1;

  if (m.ar) {  // readout adapter weights: dW2 = dh'^T A, dW1 = dU^T h_out
    ZL_HIP(wgrad(m.d, m.ar, c->ws + p.ADHPA, m.d, c->ws + p.AG, m.ar, c->layout.ad_w2));
    const void* xo = act == BF16 ? (const void*)(c->ws + p.AXO) : (const void*)c->at<float>(p.X[m.L]);
    ZL_HIP(wgrad(m.ar, m.d, c->ws + p.ADU, m.ar, xo, m.d, c->layout.ad_w1));
  }
  for (int l = m.L - 1; l >= 0; --l) {
    const LayerOff& o = c->layout.lay[l];
    const LoraOff* lo = r ? &c->layout.lora[l] : nullptr;
    bool rope_fused = false;
    // down projection
    {
      EpiArgs e = epi(m.llama ? EPI_SWIGLU_BWD : EPI_GELU_BWD, DUP, m.nup, act);
      e.aux = c->ws + p.UP[l]; e.ldaux = m.nup; e.ff = m.ff;
      GemmDesc g = gdesc(T, m.ff, m.d, DXA, m.d, true, c->W(o.w_down), m.ff, false);
      if (r) ZL_HIP(lora_bwd_dx(DXA, m.d, lo->down_a, r, lo->down_b, w_d, 1, m.ff, true, g));
      ZL_HIP(run_gemm(c, s, g, e));
    }
    if (r) {
      ZL_HIP(lora_bwd_w(DXA, m.d, c->ws + p.ACT[l], m.ff, lo->down_a, r, c->ws + p.LXD[l],
                        lo->down_b, w_d, 1));
    } else if (ln) {  // the down weight gradient runs with the QKV one below
      ZL_HIP(bias_grad(DX, F32, m.d, o.b_down));
    }
    // up projection (gate|up or fc)
    {
      EpiArgs e = epi(EPI_STORE, DN, m.d, F32);
      GemmDesc g = gdesc(T, m.d, m.nup, DUP, m.nup, true, c->W(o.w_up), m.d, false);
      if (r)
        ZL_HIP(lora_bwd_dx(DUP, m.nup, lo->up_a, m.nua, lo->up_b, m.llama ? w_up : w_up1, n_up,
                           m.d, true, g));
      ZL_HIP(run_gemm(c, s, g, e));
    }
    if (r) {
      ZL_HIP(lora_bwd_w(DUP, m.nup, c->ws + p.N2[l], m.d, lo->up_a, m.nua, c->ws + p.LXU[l],
                        lo->up_b, m.llama ? w_up : w_up1, n_up));
    } else if (ln) {  // the up weight gradient runs with the output projection's below
      ZL_HIP(bias_grad(DUP, act, m.nup, o.b_up));
    }
    // norm 2
    {
      int nblk = 0;
      ZL_RUN("norm_bwd", 0, (double)T * m.d * (16 + c->asz()), launch_norm_bwd(ln, DN, c->at<float>(p.X2[l]), c->V32(o.ln2_w),
                             ln ? c->at<float>(p.MU2[l]) : nullptr, c->at<float>(p.RS2[l]), DX, DX,
                             DXB, act, r ? nullptr : PART, ln && !r ? PART + half_part : nullptr,
                             T, m.d, s, &nblk));
      if (!r) {
        ZL_RUN("reduce_rows", 0, 0, launch_reduce_rows(PART, nblk, m.d, c->G(o.ln2_w), grad_scale, acc, s));
        if (ln) ZL_RUN("reduce_rows", 0, 0, launch_reduce_rows(PART + half_part, nblk, m.d, c->G(o.ln2_b), grad_scale, acc, s));
      }
    }
    // output projection; in bf16 its epilogue also forms the attention
    // backward's delta = rowsum(dO * O) per head
    const bool delta_fused = act == BF16 && (m.hd == 64 || m.hd == 128);
    {
      EpiArgs e = epi(delta_fused ? EPI_STORE_DELTA : EPI_STORE, DO, m.dq, act);
      if (delta_fused) {
        e.aux = c->ws + p.O[l]; e.ldaux = m.dq; e.hd = m.hd;
        e.delta = c->at<float>(p.DELTA); e.seq = c->S; e.nheads = m.hq;
      }
      GemmDesc g = gdesc(T, m.dq, m.d, DXB, m.d, true, c->W(o.w_o), m.dq, false);
      if (r) ZL_HIP(lora_bwd_dx(DXB, m.d, lo->o_a, r, lo->o_b, w_d, 1, m.dq, true, g));
      ZL_HIP(run_gemm(c, s, g, e));
    }
    if (r) {
      ZL_HIP(lora_bwd_w(DXB, m.d, c->ws + p.O[l], m.dq, lo->o_a, r, c->ws + p.LXO[l], lo->o_b,
                        w_d, 1));
    } else {
      // up (dy = DUP, kept until the next layer's down data gradient) with
      // the output projection (dy = DXB)
      ZL_HIP(wgrad2(m.nup, m.d, DUP, m.nup, c->ws + p.N2[l], m.d, o.w_up,
                    m.d, m.dq, DXB, m.d, c->ws + p.O[l], m.dq, o.w_o));
      if (ln) ZL_HIP(bias_grad(DX, F32, m.d, o.b_o));
    }
    // attention
    {
      AttnDesc a;
      memset(&a, 0, sizeof(a));
      a.B = c->B; a.S = c->S; a.Hq = m.hq; a.Hkv = m.hkv; a.hd = m.hd;
      a.q = c->ws + p.QKV[l]; a.k = c->A(p.QKV[l], m.dq); a.v = c->A(p.QKV[l], m.dq + m.dkv);
      a.ldq = a.ldk = a.ldv = m.nqkv;
      a.o = c->ws + p.O[l]; a.ldo = m.dq;
      a.lse = c->at<float>(p.LSE[l]);
      a.seq_lens = c->at<int32_t>(p.seqlens);
      a.dout = DO; a.lddo = m.dq;
      a.delta = c->at<float>(p.DELTA);
      a.delta_ready = delta_fused ? 1 : 0;
      a.dq = DQKV; a.dk = c->A(p.DQKV, m.dq); a.dv = c->A(p.DQKV, m.dq + m.dkv);
      a.lddq = a.lddk = a.lddv = m.nqkv;
      a.scale = 1.f / sqrtf((float)m.hd);
      if (m.llama) {
        a.pos = c->at<int32_t>(p.pos); a.rope = c->at<float2>(p.rope); a.max_pos = c->cfg.max_seq;
      }
      ZL_RUN("attn_bwd", 4.0 * c->B * m.hq * m.hd * (double)c->S * (c->S + 1), 0,
             launch_attn_bwd(a, act, s, &rope_fused));
    }
    if (m.llama && !rope_fused)
      ZL_RUN("rope", 0, 2.0 * T * (m.hq + m.hkv) * m.hd * c->asz(),
             launch_rope(DQKV, m.nqkv, act, c->at<int32_t>(p.pos), c->at<float2>(p.rope),
                         c->cfg.max_seq, T, m.hq + m.hkv, m.hd, -1, s));
    // QKV projection.  With LoRA nothing below layer 0's QKV GEMMs is
    // trained, so its data gradient (feeding only norm-1 weight gradients
    // and h_in, which is detached) is skipped.
    const bool need_dn = !r || l > 0;
    {
      EpiArgs e = epi(EPI_STORE, DN, m.d, F32);
      GemmDesc g = gdesc(T, m.d, m.nqkv, DQKV, m.nqkv, true, c->W(o.w_qkv), m.d, false);
      if (r)
        ZL_HIP(lora_bwd_dx(DQKV, m.nqkv, lo->qkv_a, m.nqa, lo->qkv_b, m.llama ? w_qkv : w_qkv1,
                           n_qkv, m.d, need_dn, g));
      if (need_dn) ZL_HIP(run_gemm(c, s, g, e));
    }
    if (r) {
      ZL_HIP(lora_bwd_w(DQKV, m.nqkv, c->ws + p.N1[l], m.d, lo->qkv_a, m.nqa, c->ws + p.LXQ[l],
                        lo->qkv_b, m.llama ? w_qkv : w_qkv1, n_qkv));
    } else {
      // down (dy = DXA, rewritten only by the norm-1 backward below) with
      // QKV: 3.5 + 1.5 waves of tiles at 8B fill 5 waves instead of 4 + 2
      ZL_HIP(wgrad2(m.d, m.ff, DXA, m.d, c->ws + p.ACT[l], m.ff, o.w_down,
                    m.nqkv, m.d, DQKV, m.nqkv, c->ws + p.N1[l], m.d, o.w_qkv));
      if (ln) ZL_HIP(bias_grad(DQKV, act, m.nqkv, o.b_qkv));
    }
    // norm 1; layer 0 forms no gradient into h_in
    if (need_dn) {
      int nblk = 0;
      float* dx = l > 0 ? DX : nullptr;
      ZL_RUN("norm_bwd", 0, (double)T * m.d * (16 + c->asz()), launch_norm_bwd(ln, DN, c->at<float>(p.X[l]), c->V32(o.ln1_w),
                             ln ? c->at<float>(p.MU1[l]) : nullptr, c->at<float>(p.RS1[l]), dx, dx,
                             l > 0 ? DXA : nullptr, act, r ? nullptr : PART,
                             ln && !r ? PART + half_part : nullptr, T, m.d, s, &nblk));
      if (!r) {
        ZL_RUN("reduce_rows", 0, 0, launch_reduce_rows(PART, nblk, m.d, c->G(o.ln1_w), grad_scale, acc, s));
        if (ln) ZL_RUN("reduce_rows", 0, 0, launch_reduce_rows(PART + half_part, nblk, m.d, c->G(o.ln1_b), grad_scale, acc, s));
      }
    }
  }
  c->state = ST_IDLE;
  c->has_grad = true;
  c->grad_fresh = false;
  return ZL_OK;
}

// ------------------------------------------------------------- optimizer
zl_status zl_optimizer_step(zl_chunk* c, void* stream) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "chunk is NULL");
  if (!c->has_grad)
    return fail(ZL_ERR_STATE, "zl_optimizer_step needs a zl_chunk_backward since the last step");
  OptDesc o;
  o.master = c->buf.master;
  o.shadow = c->act == BF16 ? reinterpret_cast<bf16_t*>(c->buf.shadow) : nullptr;
  o.grad = c->buf.grad;
  o.m = c->buf.adam_m;
  o.v = c->buf.adam_v;
  o.n = c->layout.n_params;
  o.optimizer = c->cfg.optimizer == ZL_ADAMW ? 0 : 1;
  o.lr = c->cfg.lr; o.beta1 = c->cfg.beta1; o.beta2 = c->cfg.beta2;
  o.eps = c->cfg.eps; o.wd = c->cfg.weight_decay;
  const double t = (double)(c->step + 1);
  o.bc1 = (float)(1.0 - pow((double)c->cfg.beta1, t));
  o.bc2 = (float)(1.0 - pow((double)c->cfg.beta2, t));
  hipStream_t s = S_(stream);
  ZL_RUN("optimizer", 0, (double)o.n * (o.optimizer == 0 ? 28.0 : 12.0) + (o.shadow ? 2.0 * o.n : 0.0),
         launch_optimizer(o, s));
  c->step += 1;
  c->has_grad = false;
  c->grad_fresh = true;
  return ZL_OK;
}

zl_status zl_chunk_update(zl_chunk* c, const void* h_in, const int32_t* seq_lens,
                          const int32_t* pos_ids, const int32_t* labels, int B, int S,
                          void* h_out, float* loss_out, void* stream) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "chunk is NULL");
  if (!labels || !loss_out) return fail(ZL_ERR_INVALID_ARG, "labels and loss_out required");
  zl_status st = zl_chunk_forward(c, h_in, seq_lens, pos_ids, B, S, h_out, stream);
  if (st != ZL_OK) return st;
  st = zl_local_objective(c, labels, loss_out, stream);
  if (st != ZL_OK) return st;
  st = zl_chunk_backward(c, 1.f, 0, stream);
  if (st != ZL_OK) return st;
  return zl_optimizer_step(c, stream);
}

// ------------------------------------------------------------- inspection
zl_status zl_inspect(const zl_chunk* c, const char* name, int layer, zl_view* v) {
  if (!c || !name || !v) return fail(ZL_ERR_INVALID_ARG, "NULL argument");
  const Dims& m = c->m;
  const Plan& p = c->plan;
  const int T = c->T;
  const int act = c->act == BF16 ? ZL_BF16 : ZL_F32;
  auto set = [&](size_t off, int64_t rows, int64_t cols, int dt) {
    v->ptr = c->ws + off; v->rows = rows; v->cols = cols; v->ld = cols; v->dtype = dt;
    return ZL_OK;
  };
  const std::string n(name);
  if (n == "x") {
    if (layer < 0 || layer > m.L) return fail(ZL_ERR_INVALID_ARG, "layer out of range");
    return set(p.X[layer], T, m.d, ZL_F32);
  }
  if (n == "dh_out") return set(p.DX, T, m.d, ZL_F32);
  if (n == "row_loss") return set(p.ROWLOSS, T, 1, ZL_F32);
  if (n == "n_omega") return set(p.NOMEGA, 1, 1, ZL_F32);
  if (n == "dz" || n == "dnf") {
    if (T < 1) return fail(ZL_ERR_STATE, "no forward has run");
    const int last = (T - 1) / p.R * p.R;  // first row of the last row block
    const int rows = T - last;
    if (n == "dz") return set(p.DZ, rows, p.Vpad, act);
    return set(p.DNF, rows, m.d, ZL_F32);
  }
  if (n == "dxa") return set(p.DXA, T, m.d, act);
  if (n == "dxb") return set(p.DXB, T, m.d, act);
  if (n == "dup") return set(p.DUP, T, m.nup, act);
  if (n == "do") return set(p.DO, T, m.dq, act);
  if (n == "dqkv") return set(p.DQKV, T, m.nqkv, act);
  if (n == "dn") return set(p.DN, T, m.d, ZL_F32);
  if (layer < 0 || layer >= m.L) return fail(ZL_ERR_INVALID_ARG, "layer out of range");
  if (n == "n1") return set(p.N1[layer], T, m.d, act);
  if (n == "qkv") return set(p.QKV[layer], T, m.nqkv, act);
  if (n == "o") return set(p.O[layer], T, m.dq, act);
  if (n == "lse") return set(p.LSE[layer], (int64_t)c->B * m.hq, c->S, ZL_F32);
  if (n == "x2") return set(p.X2[layer], T, m.d, ZL_F32);
  if (n == "n2") return set(p.N2[layer], T, m.d, act);
  if (n == "up") return set(p.UP[layer], T, m.nup, act);
  if (n == "act") return set(p.ACT[layer], T, m.ff, act);
  if (n == "rstd1") return set(p.RS1[layer], T, 1, ZL_F32);
  if (n == "rstd2") return set(p.RS2[layer], T, 1, ZL_F32);
  return fail(ZL_ERR_INVALID_ARG, "unknown view name: " + n);
}

zl_status zl_profile_begin(zl_chunk* c, int capacity) {
  if (!c) return fail(ZL_ERR_INVALID_ARG, "chunk is NULL");
  if (capacity < 1 || capacity > (1 << 20)) return fail(ZL_ERR_INVALID_ARG, "bad capacity");
  while (c->prof_ev.size() < (size_t)capacity * 2) {
    hipEvent_t e;
    ZL_HIP(hipEventCreate(&e));
    c->prof_ev.push_back(e);
  }
  c->prof_rec.assign((size_t)capacity, zl_chunk::Rec{nullptr, 0, 0});
  c->prof_used = 0;
  c->prof_on = true;
  return ZL_OK;
}

zl_status zl_profile_end(zl_chunk* c, zl_profile_entry* out, int* n) {
  if (!c || !n) return fail(ZL_ERR_INVALID_ARG, "NULL argument");
  if (!c->prof_on) return fail(ZL_ERR_STATE, "profiling was not begun");
  c->prof_on = false;
  std::vector<zl_profile_entry> agg;
  for (size_t i = 0; i < c->prof_used; ++i) {
    const zl_chunk::Rec& r = c->prof_rec[i];
    if (!r.name) continue;
    ZL_HIP(hipEventSynchronize(c->prof_ev[2 * i + 1]));
    float ms = 0.f;
    ZL_HIP(hipEventElapsedTime(&ms, c->prof_ev[2 * i], c->prof_ev[2 * i + 1]));
    zl_profile_entry* e = nullptr;
    for (auto& a : agg)
      if (strncmp(a.name, r.name, sizeof(a.name)) == 0) e = &a;
    if (!e) {
      zl_profile_entry z;
      memset(&z, 0, sizeof(z));
      strncpy(z.name, r.name, sizeof(z.name) - 1);
      agg.push_back(z);
      e = &agg.back();
    }
    e->launches += 1;
    e->total_ms += ms;
    e->flops += r.flops;
    e->bytes += r.bytes;
  }
  const int cap = *n;
  *n = (int)agg.size();
  if (out) memcpy(out, agg.data(), sizeof(zl_profile_entry) * (size_t)(cap < *n ? cap : *n));
  c->prof_used = 0;
  return ZL_OK;
}

zl_status zl_device_info(int device, int* cu_count, int* clock_khz, char* arch, int arch_len) {
  hipDeviceProp_t prop;
  ZL_HIP(hipGetDeviceProperties(&prop, device));
  if (cu_count) *cu_count = prop.multiProcessorCount;
  if (clock_khz) *clock_khz = prop.clockRate;
  if (arch && arch_len > 0) {
    strncpy(arch, prop.gcnArchName, (size_t)arch_len - 1);
    arch[arch_len - 1] = 0;
  }
  return ZL_OK;
}

zl_status zl_kernel_gemm(int M, int N, int K, const void* A, int64_t lda, int a_kmajor,
                         const void* B, int64_t ldb, int b_kmajor, int K2, const void* A2,
                         int64_t lda2, const void* B2, int64_t ldb2, float* C, int64_t ldc,
                         float* workspace, size_t workspace_elems, int dtype, void* stream) {
  if (M < 0 || N < 0 || K < 0 || K2 < 0 || !A || !B || !C || (K2 > 0 && (!A2 || !B2)))
    return fail(ZL_ERR_INVALID_ARG, "bad gemm args");
  if (dtype != ZL_F32 && dtype != ZL_BF16) return fail(ZL_ERR_INVALID_ARG, "bad dtype");
  if (dtype == ZL_BF16) {
    const int64_t ca = a_kmajor ? K : M, cb = b_kmajor ? K : N;
    if (ca % 8 || cb % 8 || lda % 8 || ldb % 8 || ((uintptr_t)A | (uintptr_t)B) % 16)
      return fail(ZL_ERR_INVALID_ARG, "bf16 gemm needs 8-element contiguous dims and alignment");
    const int64_t ca2 = a_kmajor ? K2 : M, cb2 = b_kmajor ? K2 : N;
    if (K2 > 0 && (ca2 % 8 || cb2 % 8 || lda2 % 8 || ldb2 % 8 || ((uintptr_t)A2 | (uintptr_t)B2) % 16))
      return fail(ZL_ERR_INVALID_ARG, "bf16 gemm needs 8-element contiguous dims and alignment");
  }
  GemmDesc g = gdesc(M, N, K, A, lda, a_kmajor != 0, B, ldb, b_kmajor != 0);
  if (K2 > 0) { g.K2 = K2; g.A2 = A2; g.lda2 = lda2; g.B2 = B2; g.ldb2 = ldb2; }
  if (workspace && workspace_elems) {
    if ((uintptr_t)workspace % 16) return fail(ZL_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    g.part = workspace;
    g.part_elems = workspace_elems;
  }
  EpiArgs e = epi(EPI_STORE, C, ldc, F32);
  ZL_HIP(launch_gemm(g, e, dtype == ZL_BF16 ? BF16 : F32, S_(stream)));
  return ZL_OK;
}

zl_status zl_kernel_attention(int B, int S, int Hq, int Hkv, int hd, const void* q,
                              const void* k, const void* v, int64_t ld_qkv,
                              const int32_t* seq_lens, void* o, float* lse, const void* dout,
                              void* dq, void* dk, void* dv, float* delta, int dtype,
                              int backward, void* stream) {
  if (B < 1 || S < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || !q || !k || !v || !o || !lse || !seq_lens)
    return fail(ZL_ERR_INVALID_ARG, "bad attention args");
  if (hd != 16 && hd != 32 && hd != 64 && hd != 128)
    return fail(ZL_ERR_UNSUPPORTED, "head_dim must be 16, 32, 64 or 128");
  if (backward && (!dout || !dq || !dk || !dv || !delta))
    return fail(ZL_ERR_INVALID_ARG, "backward needs dout, dq, dk, dv and delta");
  AttnDesc a;
  memset(&a, 0, sizeof(a));
  a.B = B; a.S = S; a.Hq = Hq; a.Hkv = Hkv; a.hd = hd;
  a.q = q; a.k = k; a.v = v; a.ldq = a.ldk = a.ldv = ld_qkv;
  a.o = o; a.ldo = (int64_t)Hq * hd; a.lse = lse; a.seq_lens = seq_lens;
  a.dout = dout; a.lddo = (int64_t)Hq * hd; a.delta = delta;
  a.dq = dq; a.dk = dk; a.dv = dv; a.lddq = a.lddk = a.lddv = ld_qkv;
  a.scale = 1.f / sqrtf((float)hd);
  const int dt = dtype == ZL_BF16 ? BF16 : F32;
  bool fused = false;
  if (backward) ZL_HIP(launch_attn_bwd(a, dt, S_(stream), &fused));
  else ZL_HIP(launch_attn_fwd(a, dt, S_(stream)));
  return ZL_OK;
}

}  // extern "C"
