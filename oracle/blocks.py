"""One decoder layer, forward and backward (the pieces of f_k in Eq. (1)).

Llama form: pre-RMSNorm, RoPE'd GQA causal attention, residual, pre-RMSNorm,
SwiGLU MLP, residual.  GPT-2 form: pre-LayerNorm with biases everywhere,
GELU(tanh) MLP, no rotary (positions live in the embedding, outside the
chunk).
"""
import numpy as np

from . import ops


def _split_heads(y, B, S, H, hd):
    return y.reshape(B, S, H, hd)


def _lora(P, pre, name):
    """(A, B) of the low-rank update of linear `name` (Eq. (6): LoRA on the
    frozen w_l), or None when the linear has none."""
    a = P.get(pre + name + "_la")
    return None if a is None else (a, P[pre + name + "_lb"])


def _lin(x, P, pre, name, cfg, bias=None):
    """y = x W^T (+ b) + s (x A^T) B^T, s = lora_alpha / r, W frozen."""
    y = ops.linear_fwd(x, P[pre + name], None if bias is None else P[pre + bias])
    ab = _lora(P, pre, name)
    if ab is not None:
        y = y + cfg.st(cfg.lora_scale * (x @ ab[0].T)) @ ab[1].T
    return y


def _lin_bwd(dy, x, P, pre, name, cfg, G, bias=None):
    """dx of _lin; gradients of W (and b) into G, and of A, B when present:
    dx = dy W + s (dy B) A, dA = s (dy B)^T x, dB = s dy^T (x A^T)."""
    if bias is None:
        dx, G[pre + name] = ops.linear_bwd(dy, x, P[pre + name])
    else:
        dx, G[pre + name], G[pre + bias] = ops.linear_bwd(dy, x, P[pre + name], True)
    ab = _lora(P, pre, name)
    if ab is not None:
        A, Bm = ab
        s = cfg.lora_scale
        e = cfg.st(s * (dy @ Bm))
        dx = dx + e @ A
        G[pre + name + "_la"] = e.T @ x
        G[pre + name + "_lb"] = dy.T @ cfg.st(s * (x @ A.T))
    return dx


def llama_layer_fwd(x, P, pre, cfg, ang, seq_lens, B, S):
    """x [T, d] -> x_out [T, d]; returns (x_out, cache)."""
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    st = cfg.st  # identity unless the bf16 storage floor is measured
    n1, c_n1 = ops.rmsnorm_fwd(x, P[pre + "ln1_w"], cfg.norm_eps)
    n1 = st(n1)
    q = _split_heads(_lin(n1, P, pre, "wq", cfg), B, S, Hq, hd)
    k = _split_heads(_lin(n1, P, pre, "wk", cfg), B, S, Hkv, hd)
    v = st(_split_heads(_lin(n1, P, pre, "wv", cfg), B, S, Hkv, hd))
    qr = st(ops.rope_fwd(q, ang))
    kr = st(ops.rope_fwd(k, ang))
    o, c_att = ops.attention_fwd(qr, kr, v, seq_lens, st if cfg.store_bf16 else None)
    o2 = st(o.reshape(B * S, Hq * hd))
    x2 = x + _lin(o2, P, pre, "wo", cfg)
    n2, c_n2 = ops.rmsnorm_fwd(x2, P[pre + "ln2_w"], cfg.norm_eps)
    n2 = st(n2)
    g = st(_lin(n2, P, pre, "wg", cfg))
    u = st(_lin(n2, P, pre, "wu", cfg))
    a = st(ops.swiglu_fwd(g, u))
    x3 = x2 + _lin(a, P, pre, "wd", cfg)
    cache = dict(x=x, n1=n1, c_n1=c_n1, c_att=c_att, o2=o2, n2=n2, c_n2=c_n2,
                 g=g, u=u, a=a, ang=ang, B=B, S=S)
    return x3, cache


def llama_layer_bwd(dx3, P, pre, cfg, cache, need_dx=True):
    """Backward of llama_layer_fwd; returns (dx or None, grads dict)."""
    B, S = cache["B"], cache["S"]
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    st = cfg.st  # identity unless the bf16 storage floor is measured
    G = {}
    da = _lin_bwd(st(dx3), cache["a"], P, pre, "wd", cfg, G)
    dg, du = ops.swiglu_bwd(da, cache["g"], cache["u"])
    dg, du = st(dg), st(du)
    dn2_g = _lin_bwd(dg, cache["n2"], P, pre, "wg", cfg, G)
    dn2_u = _lin_bwd(du, cache["n2"], P, pre, "wu", cfg, G)
    dx2_n, G[pre + "ln2_w"] = ops.rmsnorm_bwd(dn2_g + dn2_u, cache["c_n2"])
    dx2 = dx3 + dx2_n
    do2 = st(_lin_bwd(st(dx2), cache["o2"], P, pre, "wo", cfg, G))
    dqr, dkr, dv = ops.attention_bwd(do2.reshape(B, S, Hq, hd), cache["c_att"])
    dq = st(ops.rope_bwd(dqr, cache["ang"]).reshape(B * S, Hq * hd))
    dk = st(ops.rope_bwd(dkr, cache["ang"]).reshape(B * S, Hkv * hd))
    dv = st(dv.reshape(B * S, Hkv * hd))
    n1 = cache["n1"]
    dn1_q = _lin_bwd(dq, n1, P, pre, "wq", cfg, G)
    dn1_k = _lin_bwd(dk, n1, P, pre, "wk", cfg, G)
    dn1_v = _lin_bwd(dv, n1, P, pre, "wv", cfg, G)
    dx_n, G[pre + "ln1_w"] = ops.rmsnorm_bwd(dn1_q + dn1_k + dn1_v, cache["c_n1"])
    dx = dx2 + dx_n if need_dx else None
    return dx, G


def gpt2_layer_fwd(x, P, pre, cfg, ang, seq_lens, B, S):
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    dq, dkv = Hq * hd, Hkv * hd
    st = cfg.st  # identity unless the bf16 storage floor is measured
    n1, c_n1 = ops.layernorm_fwd(x, P[pre + "ln1_w"], P[pre + "ln1_b"], cfg.norm_eps)
    n1 = st(n1)
    qkv = st(_lin(n1, P, pre, "wqkv", cfg, "bqkv"))
    q = _split_heads(qkv[:, :dq], B, S, Hq, hd)
    k = _split_heads(qkv[:, dq:dq + dkv], B, S, Hkv, hd)
    v = _split_heads(qkv[:, dq + dkv:], B, S, Hkv, hd)
    o, c_att = ops.attention_fwd(q, k, v, seq_lens, st if cfg.store_bf16 else None)
    o2 = st(o.reshape(B * S, dq))
    x2 = x + _lin(o2, P, pre, "wo", cfg, "bo")
    n2, c_n2 = ops.layernorm_fwd(x2, P[pre + "ln2_w"], P[pre + "ln2_b"], cfg.norm_eps)
    n2 = st(n2)
    hfc = st(_lin(n2, P, pre, "wfc", cfg, "bfc"))
    a = st(ops.gelu_fwd(hfc))
    x3 = x2 + _lin(a, P, pre, "wproj", cfg, "bproj")
    cache = dict(x=x, n1=n1, c_n1=c_n1, c_att=c_att, o2=o2, n2=n2, c_n2=c_n2,
                 hfc=hfc, a=a, B=B, S=S)
    return x3, cache


def gpt2_layer_bwd(dx3, P, pre, cfg, cache, need_dx=True):
    B, S = cache["B"], cache["S"]
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    st = cfg.st  # identity unless the bf16 storage floor is measured
    G = {}
    da = _lin_bwd(st(dx3), cache["a"], P, pre, "wproj", cfg, G, "bproj")
    dh = st(ops.gelu_bwd(da, cache["hfc"]))
    dn2 = _lin_bwd(dh, cache["n2"], P, pre, "wfc", cfg, G, "bfc")
    dx2_n, G[pre + "ln2_w"], G[pre + "ln2_b"] = ops.layernorm_bwd(dn2, cache["c_n2"])
    dx2 = dx3 + dx2_n
    do2 = st(_lin_bwd(st(dx2), cache["o2"], P, pre, "wo", cfg, G, "bo"))
    dq, dk, dv = ops.attention_bwd(do2.reshape(B, S, Hq, hd), cache["c_att"])
    dqkv = st(np.concatenate([dq.reshape(B * S, -1), dk.reshape(B * S, -1),
                              dv.reshape(B * S, -1)], axis=1))
    dn1 = _lin_bwd(dqkv, cache["n1"], P, pre, "wqkv", cfg, G, "bqkv")
    dx_n, G[pre + "ln1_w"], G[pre + "ln1_b"] = ops.layernorm_bwd(dn1, cache["c_n1"])
    dx = dx2 + dx_n if need_dx else None
    return dx, G
