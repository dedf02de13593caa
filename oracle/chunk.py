"""The chunk-local update of one chunk k (Sec. II.A) and a global-BP reference.

chunk_update_ref runs, in the paper's order (in-stage steps S1-S3 of
Sec. III-B):
  1. forward h_k = f_k(h_{k-1}) through the chunk's layers (Eq. (1));
  2. the local objective on the frozen head (Eq. (2)-(5));
  3. backward inside the chunk only -- h_{k-1} is detached, so no gradient
     to it is formed (Remark 1; block-diagonal Jacobian of Sec. II.C);
  4. gradient accumulation over the update window and the optimizer step
     (Eq. (6) / AdamW).
In bf16 mode the 2-D weight matrices are rounded to bf16 (nearest-even) from
the fp32 master before use, as the device consumes its bf16 shadow; norm
weights and biases stay fp32; everything is then computed in fp64.
"""
from dataclasses import dataclass, field

import numpy as np

from . import blocks, ops
from .objective import local_objective_ref, head_norm_fwd, head_norm_bwd, log_softmax, IGNORE
from .optim import adamw_step_ref, sgd_step_ref


def bf16_round(x):
    """Round to the nearest bf16 value (ties to even), returned as float64."""
    a = np.ascontiguousarray(np.asarray(x, np.float64).astype(np.float32))
    bits = a.view(np.uint32).astype(np.uint64)
    keep_lsb = (bits >> np.uint64(16)) & np.uint64(1)
    rounded = ((bits + np.uint64(0x7FFF) + keep_lsb) >> np.uint64(16)) << np.uint64(16)
    out = (rounded & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(np.float32)
    return np.where(np.isnan(a), a, out).astype(np.float64)


@dataclass
class OracleConfig:
    arch: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    norm_eps: float = 1e-5
    rope_theta: float = 1e4
    dtype: str = "f32"
    alpha: float = 0.5
    consis: str = "reverse"
    optimizer: str = "adamw"
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.01
    adapter_rank: int = 0
    lora_rank: int = 0
    lora_alpha: float = 16.0
    # Reading r4 (the bf16 storage floor): when set, every intermediate that a
    # bf16 implementation keeps in bf16 between steps (norm outputs, q/k/v
    # after RoPE, the attention output, MLP pre-activations and activation,
    # the residual-stream gradient as a matrix operand, data gradients, the
    # head's normalised rows and dL/dz) is rounded to bf16 where it is
    # stored, the arithmetic staying fp64.  Off by default; it exists only to
    # measure how far bf16 storage alone moves each result.
    store_bf16: bool = False
    extra: dict = field(default_factory=dict)

    def st(self, x):
        """x as stored between steps: bf16-rounded under store_bf16."""
        return bf16_round(x) if self.store_bf16 else x

    @property
    def lora_scale(self):
        """s = lora_alpha / r of y = x W^T + s (x A^T) B^T."""
        return self.lora_alpha / self.lora_rank if self.lora_rank else 0.0

    @classmethod
    def from_shape(cls, shape, **kw):
        base = dict(arch=shape.arch, n_layers=shape.n_layers, d_model=shape.d_model,
                    n_heads=shape.n_heads, n_kv_heads=shape.n_kv_heads,
                    head_dim=shape.head_dim, d_ff=shape.d_ff, vocab=shape.vocab,
                    norm_eps=shape.norm_eps, rope_theta=shape.rope_theta, dtype=shape.dtype,
                    adapter_rank=getattr(shape, "adapter_rank", 0),
                    lora_rank=getattr(shape, "lora_rank", 0),
                    lora_alpha=getattr(shape, "lora_alpha", 16.0))
        base.update(kw)
        return cls(**base)


def _is_matrix(key, arr):
    return np.ndim(arr) == 2


def is_trainable(cfg, key):
    """With LoRA (Eq. (6)) only the low-rank factors and the readout adapter
    are trained; the base weights, norms and biases stay frozen."""
    if not cfg.lora_rank:
        return True
    name = key.split(".", 1)[1]
    return name.endswith("_la") or name.endswith("_lb") or name.startswith("ad_")


def effective_params(cfg, params):
    """fp64 copies of the parameters as the device consumes them."""
    out = {}
    for k, v in params.items():
        a = np.asarray(v, np.float64)
        if cfg.dtype == "bf16" and _is_matrix(k, a):
            a = bf16_round(a)
        out[k] = a
    return out


def _layer_fns(cfg):
    if cfg.arch == "llama":
        return blocks.llama_layer_fwd, blocks.llama_layer_bwd
    return blocks.gpt2_layer_fwd, blocks.gpt2_layer_bwd


def _input(cfg, h):
    h = np.asarray(h, np.float64)
    return bf16_round(h) if cfg.dtype == "bf16" else h


def chunk_forward_ref(cfg, params, h_in, seq_lens=None, pos_ids=None):
    """h_in [B, S, d] -> (h_out [B, S, d] fp64, caches)."""
    h_in = _input(cfg, h_in)
    B, S, d = h_in.shape
    seq_lens = np.full(B, S) if seq_lens is None else np.asarray(seq_lens)
    pos = np.tile(np.arange(S), (B, 1)) if pos_ids is None else np.asarray(pos_ids)
    ang = ops.rope_angles(pos, cfg.head_dim, cfg.rope_theta) if cfg.arch == "llama" else None
    P = effective_params(cfg, params)
    fwd, _ = _layer_fns(cfg)
    x = h_in.reshape(B * S, d)
    caches = []
    for l in range(cfg.n_layers):
        x, c = fwd(x, P, f"L{l}.", cfg, ang, seq_lens, B, S)
        caches.append(c)
    return x.reshape(B, S, d), dict(caches=caches, P=P, B=B, S=S, h_in=h_in)


def chunk_backward_ref(cfg, dh_out, fw, need_dx=False):
    """Backward through the chunk's layers; returns (dh_in or None, grads)."""
    _, bwd = _layer_fns(cfg)
    B, S = fw["B"], fw["S"]
    dx = np.asarray(dh_out, np.float64).reshape(B * S, -1)
    grads = {}
    for l in reversed(range(cfg.n_layers)):
        nd = need_dx or l > 0
        dx, G = bwd(dx, fw["P"], f"L{l}.", cfg, fw["caches"][l], need_dx=nd)
        grads.update({k: g for k, g in G.items() if is_trainable(cfg, k)})
    return (dx.reshape(B, S, -1) if dx is not None else None), grads


def chunk_grads_ref(cfg, params, h_in, labels, head_w, head_norm_w, head_norm_b=None,
                    seq_lens=None, pos_ids=None):
    """Forward, local objective, chunk-local backward.  No optimizer step."""
    h_out, fw = chunk_forward_ref(cfg, params, h_in, seq_lens, pos_ids)
    B, S, d = h_out.shape
    W = np.asarray(head_w, np.float64)
    if cfg.dtype == "bf16":
        W = bf16_round(W)
    adapter = None
    if cfg.adapter_rank:
        pre = f"L{cfg.n_layers}."
        adapter = (fw["P"][pre + "ad_w1"], fw["P"][pre + "ad_w2"])
    loss, dh, info = local_objective_ref(
        h_out.reshape(B * S, d), fw["h_in"].reshape(B * S, d), np.asarray(labels).reshape(-1),
        W, cfg.arch, np.asarray(head_norm_w, np.float64),
        None if head_norm_b is None else np.asarray(head_norm_b, np.float64),
        cfg.norm_eps, cfg.alpha, cfg.consis, adapter=adapter,
        store=cfg.st if cfg.store_bf16 else None)
    _, grads = chunk_backward_ref(cfg, dh.reshape(B, S, d), fw, need_dx=False)
    if adapter is not None:
        pre = f"L{cfg.n_layers}."
        grads[pre + "ad_w1"] = info["adapter_grads"]["w1"]
        grads[pre + "ad_w2"] = info["adapter_grads"]["w2"]
    return dict(loss=loss, grads=grads, h_out=h_out, dh_out=dh.reshape(B, S, d), info=info)


def optimizer_step_ref(cfg, params, grads, state):
    """Apply one step to every trainable tensor (frozen ones pass through);
    returns (params, state)."""
    t = state.get("t", 0) + 1
    newp, m, v = {}, {}, {}
    for k in params:
        if not is_trainable(cfg, k):
            newp[k] = params[k]
            continue
        if cfg.optimizer == "adamw":
            newp[k], m[k], v[k] = adamw_step_ref(
                params[k], grads[k], state["m"].get(k, 0.0), state["v"].get(k, 0.0), t,
                cfg.lr, cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay)
        else:
            newp[k] = sgd_step_ref(params[k], grads[k], cfg.lr)
            m[k] = np.asarray(state["m"].get(k, 0.0), np.float64) * np.ones_like(newp[k])
            v[k] = np.asarray(state["v"].get(k, 0.0), np.float64) * np.ones_like(newp[k])
    return newp, dict(m=m, v=v, t=t)


def init_opt_state():
    return dict(m={}, v={}, t=0)


def chunk_update_ref(cfg, params, state, microbatches, head_w, head_norm_w,
                     head_norm_b=None, grad_scale=None):
    """One update window: accumulate over micro-batches, then one step.

    microbatches: list of dicts with h_in, labels and optional seq_lens,
    pos_ids.  Each micro-batch's loss is its own Omega-mean; the window
    gradient is grad_scale * sum of the micro-batch gradients (grad_scale
    defaults to 1/m).
    """
    m = len(microbatches)
    scale = (1.0 / m) if grad_scale is None else grad_scale
    acc = None
    losses, outs = [], []
    for mb in microbatches:
        r = chunk_grads_ref(cfg, params, mb["h_in"], mb["labels"], head_w, head_norm_w,
                            head_norm_b, mb.get("seq_lens"), mb.get("pos_ids"))
        losses.append(r["loss"])
        outs.append(r)
        if acc is None:
            acc = {k: scale * g for k, g in r["grads"].items()}
        else:
            for k, g in r["grads"].items():
                acc[k] = acc[k] + scale * g
    newp, news = optimizer_step_ref(cfg, params, acc, state)
    return dict(params=newp, state=news, grads=acc, losses=losses, runs=outs)


def global_bp_ref(cfg, chunk_params, h0, labels, head_w, head_norm_w, head_norm_b=None,
                  seq_lens=None, pos_ids=None):
    """Ordinary backpropagation of the stacked chunks on the final head.

    Loss: token-mean cross-entropy of the last chunk's readout over Omega
    (the global objective L = L_task of Sec. II.B).  Returns the loss and the
    gradient of every chunk's parameters.
    """
    x = h0
    fws = []
    for P in chunk_params:
        x, fw = chunk_forward_ref(cfg, P, x, seq_lens, pos_ids)
        fws.append(fw)
    B, S, d = x.shape
    W = np.asarray(head_w, np.float64)
    if cfg.dtype == "bf16":
        W = bf16_round(W)
    hn_w = np.asarray(head_norm_w, np.float64)
    hn_b = None if head_norm_b is None else np.asarray(head_norm_b, np.float64)
    n, c = head_norm_fwd(x.reshape(B * S, d), cfg.arch, hn_w, hn_b, cfg.norm_eps)
    z = n @ W.T
    lab = np.asarray(labels).reshape(-1)
    idx = np.nonzero(lab != IGNORE)[0]
    logp = log_softmax(z)
    dz = np.zeros_like(z)
    loss = 0.0
    if len(idx):
        loss = float(-np.mean(logp[idx, lab[idx]]))
        p = np.exp(logp[idx])
        p[np.arange(len(idx)), lab[idx]] -= 1.0
        dz[idx] = p / len(idx)
    dx = head_norm_bwd(dz @ W, cfg.arch, c).reshape(B, S, d)
    all_grads = [None] * len(chunk_params)
    for k in reversed(range(len(chunk_params))):
        dx, all_grads[k] = chunk_backward_ref(cfg, dx, fws[k], need_dx=True)
    return dict(loss=loss, grads=all_grads, h_out=x)
