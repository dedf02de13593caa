"""Pin the oracle's ops and its hand-written backward against torch's CPU
library routines in fp64 (an independent implementation): sdpa, rms_norm,
layer_norm, gelu(tanh), silu, cross_entropy, kl_div, autograd, and
torch.optim.AdamW / SGD."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import ops
from oracle.objective import loss_and_dlogits
from tests.oracle_cases import rel_err, tiny_case

def T(a):
    return torch.tensor(np.asarray(a, np.float64), dtype=torch.float64)


def test_norms_and_activations():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((7, 12)) * 3
    w, b = rng.standard_normal(12), rng.standard_normal(12)
    y, _ = ops.rmsnorm_fwd(x, w, 1e-5)
    np.testing.assert_allclose(y, F.rms_norm(T(x), (12,), T(w), eps=1e-5).numpy(), rtol=1e-13)
    y, _ = ops.layernorm_fwd(x, w, b, 1e-5)
    np.testing.assert_allclose(y, F.layer_norm(T(x), (12,), T(w), T(b), eps=1e-5).numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(ops.gelu_fwd(x), F.gelu(T(x), approximate="tanh").numpy(), rtol=1e-13, atol=1e-15)
    g, u = x, rng.standard_normal(x.shape)
    np.testing.assert_allclose(ops.swiglu_fwd(g, u), (F.silu(T(g)) * T(u)).numpy(), rtol=1e-13, atol=1e-15)


def test_attention_vs_sdpa():
    rng = np.random.default_rng(1)
    B, S, Hq, Hkv, hd = 2, 9, 6, 2, 8
    q, k, v = (rng.standard_normal((B, S, h, hd)) for h in (Hq, Hkv, Hkv))
    lens = np.array([9, 6])
    o, cache = ops.attention_fwd(q, k, v, lens)
    allowed = torch.tensor(ops.attention_mask(B, S, lens))[:, None]
    qt, kt, vt = (T(a).transpose(1, 2).requires_grad_() for a in (q, k, v))
    ot = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=allowed, enable_gqa=True)
    np.testing.assert_allclose(o, ot.transpose(1, 2).detach().numpy(), rtol=1e-12, atol=1e-14)
    do = rng.standard_normal(o.shape)
    ot.backward(T(do).transpose(1, 2))
    dq, dk, dv = ops.attention_bwd(do, cache)
    for mine, ref in ((dq, qt), (dk, kt), (dv, vt)):
        np.testing.assert_allclose(mine, ref.grad.transpose(1, 2).numpy(), rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("consis", ["reverse", "forward"])
def test_objective_vs_torch_losses(consis):
    rng = np.random.default_rng(2)
    Tn, V, alpha = 12, 17, 0.3
    z, zp = rng.standard_normal((Tn, V)) * 2, rng.standard_normal((Tn, V)) * 2
    lab = rng.integers(0, V, Tn)
    lab[[1, 5]] = -100
    loss, dz, _ = loss_and_dlogits(z, zp, lab, alpha, consis)
    zt = T(z).requires_grad_()
    idx = torch.tensor(lab != -100)
    ce = F.cross_entropy(zt, torch.tensor(lab, dtype=torch.long), ignore_index=-100)
    lp, lq = F.log_softmax(zt, -1)[idx], F.log_softmax(T(zp), -1)[idx]
    if consis == "reverse":   # KL(p || q): kl_div(input=log q, target=log p)
        kl = F.kl_div(lq, lp, log_target=True, reduction="batchmean")
    else:                     # KL(q || p)
        kl = F.kl_div(lp, lq, log_target=True, reduction="batchmean")
    lt = alpha * ce + (1 - alpha) * kl
    lt.backward()
    assert loss == pytest.approx(lt.item(), rel=1e-13)
    np.testing.assert_allclose(dz, zt.grad.numpy(), rtol=1e-12, atol=1e-16)


def _torch_chunk_loss(c, params):
    """The chunk update's loss built from torch library primitives."""
    cfg, shp = c["cfg"], c["shape"]
    B, S, d = c["h_in"].shape
    Hq, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    allowed = torch.tensor(ops.attention_mask(B, S, c["seq_lens"]))[:, None]
    pos = T(c["pos_ids"])
    inv = cfg.rope_theta ** (-(2.0 * torch.arange(hd // 2, dtype=torch.float64)) / hd)
    ang = pos[..., None] * inv
    cos, sin = torch.cos(ang)[:, :, None], torch.sin(ang)[:, :, None]

    def rope(u):
        a, b = u[..., : hd // 2], u[..., hd // 2:]
        return torch.cat([a * cos - b * sin, b * cos + a * sin], -1)

    x = T(c["h_in"])
    for l in range(cfg.n_layers):
        p = lambda n: params[f"L{l}.{n}"]
        if cfg.arch == "llama":
            n1 = F.rms_norm(x, (d,), p("ln1_w"), eps=cfg.norm_eps)
            q = rope(F.linear(n1, p("wq")).view(B, S, Hq, hd))
            k = rope(F.linear(n1, p("wk")).view(B, S, Hkv, hd))
            v = F.linear(n1, p("wv")).view(B, S, Hkv, hd)
        else:
            n1 = F.layer_norm(x, (d,), p("ln1_w"), p("ln1_b"), eps=cfg.norm_eps)
            qkv = F.linear(n1, p("wqkv"), p("bqkv"))
            q = qkv[..., : Hq * hd].view(B, S, Hq, hd)
            k = qkv[..., Hq * hd: (Hq + Hkv) * hd].view(B, S, Hkv, hd)
            v = qkv[..., (Hq + Hkv) * hd:].view(B, S, Hkv, hd)
        o = F.scaled_dot_product_attention(q.transpose(1, 2), k.transpose(1, 2), v.transpose(1, 2),
                                           attn_mask=allowed, enable_gqa=True)
        o = o.transpose(1, 2).reshape(B, S, Hq * hd)
        if cfg.arch == "llama":
            x = x + F.linear(o, p("wo"))
            n2 = F.rms_norm(x, (d,), p("ln2_w"), eps=cfg.norm_eps)
            x = x + F.linear(F.silu(F.linear(n2, p("wg"))) * F.linear(n2, p("wu")), p("wd"))
        else:
            x = x + F.linear(o, p("wo"), p("bo"))
            n2 = F.layer_norm(x, (d,), p("ln2_w"), p("ln2_b"), eps=cfg.norm_eps)
            x = x + F.linear(F.gelu(F.linear(n2, p("wfc"), p("bfc")), approximate="tanh"), p("wproj"), p("bproj"))

    def head(h):
        if cfg.arch == "llama":
            n = F.rms_norm(h, (d,), T(c["hn_w"]), eps=cfg.norm_eps)
        else:
            n = F.layer_norm(h, (d,), T(c["hn_w"]), T(c["hn_b"]), eps=cfg.norm_eps)
        return F.linear(n, T(c["head_w"])).reshape(B * S, -1)

    z = head(x)
    zp = head(T(c["h_in"])).detach()
    lab = torch.tensor(c["labels"].reshape(-1), dtype=torch.long)
    idx = lab != -100
    ce = F.cross_entropy(z, lab, ignore_index=-100)
    lp, lq = F.log_softmax(z, -1)[idx], F.log_softmax(zp, -1)[idx]
    if cfg.consis == "reverse":
        kl = F.kl_div(lq, lp, log_target=True, reduction="batchmean")
    else:
        kl = F.kl_div(lp, lq, log_target=True, reduction="batchmean")
    return cfg.alpha * ce + (1 - cfg.alpha) * kl, x


@pytest.mark.parametrize("arch,gqa,consis", [("llama", False, "reverse"), ("llama", True, "forward"),
                                             ("gpt2", False, "reverse")])
def test_chunk_update_vs_torch_autograd(arch, gqa, consis):
    c = tiny_case(arch, gqa=gqa, alpha=0.45, consis=consis, d=16, hd=4, ff=24, V=29, S=7, B=3)
    params = {k: T(v).requires_grad_() for k, v in c["P"].items()}
    lt, xt = _torch_chunk_loss(c, params)
    lt.backward()
    r = oracle.chunk_grads_ref(c["cfg"], c["P"], c["h_in"], c["labels"], c["head_w"], c["hn_w"],
                               c["hn_b"], c["seq_lens"], c["pos_ids"])
    assert r["loss"] == pytest.approx(lt.item(), rel=1e-12)
    np.testing.assert_allclose(r["h_out"], xt.detach().numpy(), rtol=1e-12, atol=1e-13)
    for k in c["P"]:
        assert rel_err(r["grads"][k], params[k].grad.numpy()) < 1e-11, k


@pytest.mark.parametrize("opt", ["adamw", "sgd"])
def test_optimizer_vs_torch_optim(opt):
    rng = np.random.default_rng(6)
    theta = rng.standard_normal(50)
    grads = [rng.standard_normal(50) * 10 ** rng.uniform(-4, 1) for _ in range(3)]
    tp = torch.nn.Parameter(T(theta))
    if opt == "adamw":
        topt = torch.optim.AdamW([tp], lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.01)
    else:
        topt = torch.optim.SGD([tp], lr=1e-3)
    th, m, v = theta.copy(), 0.0, 0.0
    for t, g in enumerate(grads, start=1):
        tp.grad = T(g)
        topt.step()
        if opt == "adamw":
            th, m, v = oracle.adamw_step_ref(th, g, m, v, t, 1e-3, 0.9, 0.999, 1e-8, 0.01)
        else:
            th = oracle.sgd_step_ref(th, g, 1e-3)
        np.testing.assert_allclose(th, tp.detach().numpy(), rtol=1e-13, atol=1e-16)
