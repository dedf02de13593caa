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


def llama_layer_fwd(x, P, pre, cfg, ang, seq_lens, B, S):
    """x [T, d] -> x_out [T, d]; returns (x_out, cache)."""
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    n1, c_n1 = ops.rmsnorm_fwd(x, P[pre + "ln1_w"], cfg.norm_eps)
    q = _split_heads(ops.linear_fwd(n1, P[pre + "wq"]), B, S, Hq, hd)
    k = _split_heads(ops.linear_fwd(n1, P[pre + "wk"]), B, S, Hkv, hd)
    v = _split_heads(ops.linear_fwd(n1, P[pre + "wv"]), B, S, Hkv, hd)
    qr = ops.rope_fwd(q, ang)
    kr = ops.rope_fwd(k, ang)
    o, c_att = ops.attention_fwd(qr, kr, v, seq_lens)
    o2 = o.reshape(B * S, Hq * hd)
    x2 = x + ops.linear_fwd(o2, P[pre + "wo"])
    n2, c_n2 = ops.rmsnorm_fwd(x2, P[pre + "ln2_w"], cfg.norm_eps)
    g = ops.linear_fwd(n2, P[pre + "wg"])
    u = ops.linear_fwd(n2, P[pre + "wu"])
    a = ops.swiglu_fwd(g, u)
    x3 = x2 + ops.linear_fwd(a, P[pre + "wd"])
    cache = dict(x=x, n1=n1, c_n1=c_n1, c_att=c_att, o2=o2, n2=n2, c_n2=c_n2,
                 g=g, u=u, a=a, ang=ang, B=B, S=S)
    return x3, cache


def llama_layer_bwd(dx3, P, pre, cfg, cache, need_dx=True):
    """Backward of llama_layer_fwd; returns (dx or None, grads dict)."""
    B, S = cache["B"], cache["S"]
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    G = {}
    da, G[pre + "wd"] = ops.linear_bwd(dx3, cache["a"], P[pre + "wd"])
    dg, du = ops.swiglu_bwd(da, cache["g"], cache["u"])
    dn2_g, G[pre + "wg"] = ops.linear_bwd(dg, cache["n2"], P[pre + "wg"])
    dn2_u, G[pre + "wu"] = ops.linear_bwd(du, cache["n2"], P[pre + "wu"])
    dx2_n, G[pre + "ln2_w"] = ops.rmsnorm_bwd(dn2_g + dn2_u, cache["c_n2"])
    dx2 = dx3 + dx2_n
    do2, G[pre + "wo"] = ops.linear_bwd(dx2, cache["o2"], P[pre + "wo"])
    dqr, dkr, dv = ops.attention_bwd(do2.reshape(B, S, Hq, hd), cache["c_att"])
    dq = ops.rope_bwd(dqr, cache["ang"]).reshape(B * S, Hq * hd)
    dk = ops.rope_bwd(dkr, cache["ang"]).reshape(B * S, Hkv * hd)
    dv = dv.reshape(B * S, Hkv * hd)
    n1 = cache["n1"]
    dn1_q, G[pre + "wq"] = ops.linear_bwd(dq, n1, P[pre + "wq"])
    dn1_k, G[pre + "wk"] = ops.linear_bwd(dk, n1, P[pre + "wk"])
    dn1_v, G[pre + "wv"] = ops.linear_bwd(dv, n1, P[pre + "wv"])
    dx_n, G[pre + "ln1_w"] = ops.rmsnorm_bwd(dn1_q + dn1_k + dn1_v, cache["c_n1"])
    dx = dx2 + dx_n if need_dx else None
    return dx, G


def gpt2_layer_fwd(x, P, pre, cfg, ang, seq_lens, B, S):
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    dq, dkv = Hq * hd, Hkv * hd
    n1, c_n1 = ops.layernorm_fwd(x, P[pre + "ln1_w"], P[pre + "ln1_b"], cfg.norm_eps)
    qkv = ops.linear_fwd(n1, P[pre + "wqkv"], P[pre + "bqkv"])
    q = _split_heads(qkv[:, :dq], B, S, Hq, hd)
    k = _split_heads(qkv[:, dq:dq + dkv], B, S, Hkv, hd)
    v = _split_heads(qkv[:, dq + dkv:], B, S, Hkv, hd)
    o, c_att = ops.attention_fwd(q, k, v, seq_lens)
    o2 = o.reshape(B * S, dq)
    x2 = x + ops.linear_fwd(o2, P[pre + "wo"], P[pre + "bo"])
    n2, c_n2 = ops.layernorm_fwd(x2, P[pre + "ln2_w"], P[pre + "ln2_b"], cfg.norm_eps)
    hfc = ops.linear_fwd(n2, P[pre + "wfc"], P[pre + "bfc"])
    a = ops.gelu_fwd(hfc)
    x3 = x2 + ops.linear_fwd(a, P[pre + "wproj"], P[pre + "bproj"])
    cache = dict(x=x, n1=n1, c_n1=c_n1, c_att=c_att, o2=o2, n2=n2, c_n2=c_n2,
                 hfc=hfc, a=a, B=B, S=S)
    return x3, cache


def gpt2_layer_bwd(dx3, P, pre, cfg, cache, need_dx=True):
    B, S = cache["B"], cache["S"]
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    G = {}
    da, G[pre + "wproj"], G[pre + "bproj"] = ops.linear_bwd(dx3, cache["a"], P[pre + "wproj"], True)
    dh = ops.gelu_bwd(da, cache["hfc"])
    dn2, G[pre + "wfc"], G[pre + "bfc"] = ops.linear_bwd(dh, cache["n2"], P[pre + "wfc"], True)
    dx2_n, G[pre + "ln2_w"], G[pre + "ln2_b"] = ops.layernorm_bwd(dn2, cache["c_n2"])
    dx2 = dx3 + dx2_n
    do2, G[pre + "wo"], G[pre + "bo"] = ops.linear_bwd(dx2, cache["o2"], P[pre + "wo"], True)
    dq, dk, dv = ops.attention_bwd(do2.reshape(B, S, Hq, hd), cache["c_att"])
    dqkv = np.concatenate([dq.reshape(B * S, -1), dk.reshape(B * S, -1), dv.reshape(B * S, -1)], axis=1)
    dn1, G[pre + "wqkv"], G[pre + "bqkv"] = ops.linear_bwd(dqkv, cache["n1"], P[pre + "wqkv"], True)
    dx_n, G[pre + "ln1_w"], G[pre + "ln1_b"] = ops.layernorm_bwd(dn1, cache["c_n1"])
    dx = dx2 + dx_n if need_dx else None
    return dx, G
