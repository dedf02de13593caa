"""Per-op forward and hand-derived backward, fp64 NumPy.

Every function follows a textbook definition; the chunk map of Eq. (1) is
built from them in blocks.py.  Shapes: x [T, d] token rows, attention
tensors [B, S, heads, hd].
"""
import numpy as np


# ---------------------------------------------------------------- RMSNorm
def rmsnorm_fwd(x, w, eps):
    """y = x * w / sqrt(mean(x^2) + eps), row-wise."""
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    xhat = x * rstd
    return xhat * w, (xhat, rstd, w)


def rmsnorm_bwd(dy, cache):
    xhat, rstd, w = cache
    g = dy * w
    dw = np.sum(dy * xhat, axis=0)
    dx = rstd * (g - xhat * np.mean(g * xhat, axis=-1, keepdims=True))
    return dx, dw


# -------------------------------------------------------------- LayerNorm
def layernorm_fwd(x, w, b, eps):
    """y = (x - mean) / sqrt(var + eps) * w + b, row-wise (biased var)."""
    mu = np.mean(x, axis=-1, keepdims=True)
    xc = x - mu
    var = np.mean(xc * xc, axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = xc * rstd
    return xhat * w + b, (xhat, rstd, w)


def layernorm_bwd(dy, cache):
    xhat, rstd, w = cache
    g = dy * w
    dw = np.sum(dy * xhat, axis=0)
    db = np.sum(dy, axis=0)
    dx = rstd * (g - np.mean(g, axis=-1, keepdims=True)
                 - xhat * np.mean(g * xhat, axis=-1, keepdims=True))
    return dx, dw, db


# ------------------------------------------------------------------ RoPE
def rope_angles(pos, head_dim, theta):
    """angle[..., j] = pos * theta^(-2j/hd) for j < hd/2 (rotate-half form)."""
    half = head_dim // 2
    inv = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    return pos[..., None].astype(np.float64) * inv


def rope_fwd(u, ang):
    """u [B, S, H, hd]; ang [B, S, hd/2].

    u'_j = u_j cos - u_{j+h} sin,  u'_{j+h} = u_{j+h} cos + u_j sin.
    """
    half = u.shape[-1] // 2
    c = np.cos(ang)[:, :, None, :]
    s = np.sin(ang)[:, :, None, :]
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def rope_bwd(du, ang):
    """Transpose of the rotation: rotate by -angle."""
    return rope_fwd(du, -ang)


# ------------------------------------------------------------- attention
def attention_mask(B, S, seq_lens):
    """allowed[b, i, j] iff j <= i and j < seq_len[b] (causal, right padding)."""
    i = np.arange(S)[:, None]
    j = np.arange(S)[None, :]
    causal = j <= i
    m = np.zeros((B, S, S), bool)
    for b in range(B):
        m[b] = causal & (j < int(seq_lens[b]))
    return m


def _exact(x):
    return x


def attention_fwd(q, k, v, seq_lens, st=None):
    """Causal GQA attention; q [B,S,Hq,hd], k,v [B,S,Hkv,hd].

    q-head h reads kv-head h // (Hq/Hkv).  Scores q.k / sqrt(hd).  A query
    with no allowed key gets output 0.  st (measuring the bf16 storage
    floor only): how the probabilities are kept as the operand of P V.
    """
    st = _exact if st is None else st
    B, S, Hq, hd = q.shape
    Hkv = k.shape[2]
    grp = Hq // Hkv
    allowed = attention_mask(B, S, seq_lens)
    scale = 1.0 / np.sqrt(hd)
    o = np.zeros_like(q)
    P = np.zeros((B, Hq, S, S))
    for b in range(B):
        for h in range(Hq):
            g = h // grp
            s = (q[b, :, h, :] @ k[b, :, g, :].T) * scale
            s = np.where(allowed[b], s, -np.inf)
            mx = np.max(s, axis=-1, keepdims=True)
            mx = np.where(np.isfinite(mx), mx, 0.0)
            e = np.where(allowed[b], np.exp(s - mx), 0.0)
            den = np.sum(e, axis=-1, keepdims=True)
            p = np.where(den > 0, e / np.where(den > 0, den, 1.0), 0.0)
            P[b, h] = p
            o[b, :, h, :] = st(p) @ v[b, :, g, :]
    return o, (q, k, v, P, st)


def attention_bwd(do, cache):
    """st of the forward (if any) also keeps P as the operand of P^T dO and
    dS as the operand of dS K and dS^T Q."""
    q, k, v, P, st = cache
    B, S, Hq, hd = q.shape
    Hkv = k.shape[2]
    grp = Hq // Hkv
    scale = 1.0 / np.sqrt(hd)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        for h in range(Hq):
            g = h // grp
            p = P[b, h]
            dv[b, :, g, :] += st(p).T @ do[b, :, h, :]
            dp = do[b, :, h, :] @ v[b, :, g, :].T
            ds = st(p * (dp - np.sum(dp * p, axis=-1, keepdims=True)))
            dq[b, :, h, :] = (ds @ k[b, :, g, :]) * scale
            dk[b, :, g, :] += (ds.T @ q[b, :, h, :]) * scale
    return dq, dk, dv


# ----------------------------------------------------------- activations
def sigmoid(x):
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def swiglu_fwd(g, u):
    """a = silu(g) * u with silu(g) = g * sigmoid(g)."""
    return g * sigmoid(g) * u


def swiglu_bwd(da, g, u):
    sg = sigmoid(g)
    silu = g * sg
    dsilu = sg * (1.0 + g * (1.0 - sg))
    return da * u * dsilu, da * silu


_GELU_C = np.sqrt(2.0 / np.pi)


def gelu_fwd(x):
    """GELU, tanh form: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(_GELU_C * (x + 0.044715 * x ** 3)))


def gelu_bwd(dy, x):
    t = np.tanh(_GELU_C * (x + 0.044715 * x ** 3))
    dt = (1.0 - t * t) * _GELU_C * (1.0 + 3.0 * 0.044715 * x * x)
    return dy * (0.5 * (1.0 + t) + 0.5 * x * dt)


# ---------------------------------------------------------------- linear
def linear_fwd(x, w, b=None):
    """y = x W^T (+ b); W is [out, in]."""
    y = x @ w.T
    return y if b is None else y + b


def linear_bwd(dy, x, w, with_bias=False):
    """Returns dx = dy W, dW = dy^T x, db = sum_rows dy."""
    dx = dy @ w
    dw = dy.T @ x
    if with_bias:
        return dx, dw, np.sum(dy, axis=0)
    return dx, dw
