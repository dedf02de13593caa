"""Frozen readout head and the local objective (Sec. II.A, Eq. (2)-(5)).

Readout (Eq. (2)): z = Norm(h) W_lm^T, p = softmax(z) row-wise, with Norm the
model's frozen final norm (static model head, Sec. III-B (a)).

Local loss (Eq. (3)): L = alpha * L_task + (1 - alpha) * L_consis, each a mean
over the labelled set Omega.
  * L_task: cross-entropy -log p(y) -- the practical replacement of the
    Bregman/KL term that Eq. (4) names; taken with a plus sign, the sign
    used in the proof of Lemma 1 (the minus printed in Eq. (4) would push p
    away from the target).
  * L_consis: KL divergence to the stop-gradient readout of the chunk's own
    input (Eq. (5)); "reverse" is KL(p_k || p_{k-1}) as in Eq. (5) with the
    negative-entropy potential and the KL form of Sec. II.C; "forward" is
    KL(p_{k-1} || p_k).  p_{k-1} is recomputed from h_{k-1} because stages
    exchange hidden states only (Sec. III-A (III)).
The mean runs over all labelled tokens of the micro-batch; with no labelled
token the loss and its gradient are zero.
"""
import numpy as np

from . import ops

IGNORE = -100


def head_norm_fwd(h, arch, w, b, eps):
    if arch == "llama":
        return ops.rmsnorm_fwd(h, w, eps)
    return ops.layernorm_fwd(h, w, b, eps)


def head_norm_bwd(dn, arch, cache):
    """Gradient to h only: the head norm is frozen."""
    if arch == "llama":
        dx, _ = ops.rmsnorm_bwd(dn, cache)
    else:
        dx, _, _ = ops.layernorm_bwd(dn, cache)
    return dx


def head_logits_ref(h, head_w, arch, hn_w, hn_b, eps):
    n, _ = head_norm_fwd(np.asarray(h, np.float64), arch, hn_w, hn_b, eps)
    return n @ np.asarray(head_w, np.float64).T


def log_softmax(z):
    m = np.max(z, axis=-1, keepdims=True)
    return z - (m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True)))


def reverse_kl_rows(logp, logr):
    """KL(p || r) per row and its gradient with respect to the logits of p.

    With d = log p - log r: KL = sum_v p_v d_v and, through the softmax,
    d KL / d z_j = p_j (d_j - KL).
    """
    p = np.exp(logp)
    d = logp - logr
    kl = np.sum(p * d, axis=-1)
    return kl, p * (d - kl[:, None])


def soft_target_objective(z, logt, zp, alpha):
    """alpha KL(p || t) + (1 - alpha) KL(p || q) per row, and d/dz.

    The KL form of the local loss used in the analysis of Sec. II.C, with a
    soft target t in place of the one-hot p_y (which makes KL(p || p_y)
    infinite).  Shares reverse_kl_rows with the consistency term.
    """
    logp = log_softmax(z)
    kt, gt = reverse_kl_rows(logp, logt)
    kq, gq = reverse_kl_rows(logp, log_softmax(zp))
    return alpha * kt + (1.0 - alpha) * kq, alpha * gt + (1.0 - alpha) * gq


def loss_and_dlogits(z, zp, labels, alpha, consis):
    """Per-row terms and dL/dz for logits z (of h_out) and zp (of h_in).

    Returns (loss, dz, rows) with rows a dict of per-row ce, kl (0 outside
    Omega).  zp may be None when alpha == 1.
    """
    T, V = z.shape
    mask = labels != IGNORE
    n_omega = int(np.sum(mask))
    logp = log_softmax(z)
    p = np.exp(logp)
    ce = np.zeros(T)
    kl = np.zeros(T)
    dz = np.zeros_like(z)
    if n_omega == 0:
        return 0.0, dz, dict(ce=ce, kl=kl, n_omega=0)
    idx = np.nonzero(mask)[0]
    y = labels[idx]
    ce[idx] = -logp[idx, y]
    onehot = np.zeros((len(idx), V))
    onehot[np.arange(len(idx)), y] = 1.0
    g = alpha * (p[idx] - onehot)
    if alpha < 1.0:
        logq = log_softmax(zp)
        q = np.exp(logq)
        if consis == "reverse":
            kl[idx], gk = reverse_kl_rows(logp[idx], logq[idx])
            g = g + (1.0 - alpha) * gk
        elif consis == "forward":
            # KL(q || p) = sum_v q (log q - log p); d/dz = p - q
            kl[idx] = np.sum(q[idx] * (logq[idx] - logp[idx]), axis=-1)
            g = g + (1.0 - alpha) * (p[idx] - q[idx])
        else:
            raise ValueError(consis)
    dz[idx] = g / n_omega
    loss = float(np.sum(alpha * ce[idx] + (1.0 - alpha) * kl[idx]) / n_omega)
    return loss, dz, dict(ce=ce, kl=kl, n_omega=n_omega)


def _keep(x):
    return x


def _block_fp16(z, width=64):
    """z kept as fp16 offsets from the maximum of each row's 64-column block
    (measuring the storage floor only)."""
    out = np.empty_like(z)
    for c0 in range(0, z.shape[1], width):
        blk = z[:, c0:c0 + width]
        m = np.max(blk, axis=1, keepdims=True)
        out[:, c0:c0 + width] = m + (blk - m).astype(np.float16).astype(np.float64)
    return out


def adapter_fwd(h, w1, w2, st=_keep):
    """Readout adapter (Sec. III-B, Local Update interface (b)): a residual
    MLP h' = h + gelu(h W1^T) W2^T, W1 [r, d], W2 [d, r], that is the
    identity when W2 = 0.  st: how stored intermediates are kept (exact by
    default; bf16 rounding when the storage floor is measured)."""
    hs = st(h)
    u = st(hs @ w1.T)
    a = st(ops.gelu_fwd(u))
    return h + a @ w2.T, (hs, u, a, w1, w2)


def adapter_bwd(dhp, cache, st=_keep):
    """dL/dh and the weight gradients from dL/dh'."""
    h, u, a, w1, w2 = cache
    dhs = st(dhp)
    du = st(ops.gelu_bwd(dhs @ w2, u))
    return dhp + du @ w1, dict(w1=du.T @ h, w2=dhs.T @ a)


def local_objective_ref(h_out, h_in, labels, head_w, arch, hn_w, hn_b, eps,
                        alpha, consis="reverse", adapter=None, store=None):
    """Loss and dL/dh_out for one micro-batch.  h_* [T, d], labels [T].

    h_in enters only through the stop-gradient readout; no gradient to it is
    formed.  adapter: optional (W1, W2); h_out is read out through it, the
    consistency target from h_in is the static head's readout.  The adapter
    weight gradients are returned in info["adapter_grads"].  store: optional
    rounding of the stored intermediates (the normalised rows the head reads
    and dL/dz), used only to measure the bf16 storage floor.
    """
    st = _keep if store is None else store
    h_out = np.asarray(h_out, np.float64)
    W = np.asarray(head_w, np.float64)
    ad_cache = None
    if adapter is not None:
        h_out, ad_cache = adapter_fwd(h_out, np.asarray(adapter[0], np.float64),
                                      np.asarray(adapter[1], np.float64), st)
    n, c = head_norm_fwd(h_out, arch, hn_w, hn_b, eps)
    z = st(n) @ W.T
    zp = None
    if alpha < 1.0:
        n_in, _ = head_norm_fwd(np.asarray(h_in, np.float64), arch, hn_w, hn_b, eps)
        zp = st(n_in) @ W.T
    loss, dz, rows = loss_and_dlogits(z, zp, np.asarray(labels).reshape(-1), alpha, consis)
    if store is not None:
        # the logits as cached for dL/dz: fp16 values of z minus the maximum
        # of their 64-column block; the loss keeps its exact statistics
        _, dz, _ = loss_and_dlogits(_block_fp16(z), None if zp is None else _block_fp16(zp),
                                    np.asarray(labels).reshape(-1), alpha, consis)
    dn = st(dz) @ W
    dh = head_norm_bwd(dn, arch, c)
    info = dict(z=z, zp=zp, dz=dz, **rows)
    if ad_cache is not None:
        info["dh_adapted"] = dh
        dh, info["adapter_grads"] = adapter_bwd(dh, ad_cache, st)
    return loss, dh, info
