"""Closed forms and invariants that pin the oracle (no implementation of the
paper exists to compare against, and the paper prints no worked value for a
chunk update)."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import ops
from oracle.chunk import chunk_backward_ref, chunk_forward_ref, init_opt_state, optimizer_step_ref
from oracle.objective import (log_softmax, loss_and_dlogits, local_objective_ref,
                              soft_target_objective)
from tests.oracle_cases import rel_err, tiny_case

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")))


def _grads(c, **over):
    P = over.pop("P", c["P"])
    h_in = over.pop("h_in", c["h_in"])
    head_w = over.pop("head_w", c["head_w"])
    return oracle.chunk_grads_ref(c["cfg"], P, h_in, c["labels"], head_w, c["hn_w"], c["hn_b"],
                                  c["seq_lens"], c["pos_ids"])


# P1 ------------------------------------------------------------------------
@pytest.mark.parametrize("case", GOLD["uniform_head_loss"]["cases"])
@pytest.mark.parametrize("arch", ["llama", "gpt2"])
def test_p1_uniform_head(case, arch):
    """W_lm = 0 => p = q = uniform => L = alpha ln V exactly, dh_out = 0 (Eq. (2)-(5))."""
    c = tiny_case(arch, alpha=case["alpha"], V=case["vocab"])
    assert case["loss"] == pytest.approx(case["alpha"] * math.log(case["vocab"]), abs=1e-15)
    r = _grads(c, head_w=np.zeros_like(c["head_w"]))
    assert r["loss"] == pytest.approx(case["loss"], rel=1e-13, abs=1e-13)
    assert np.max(np.abs(r["dh_out"])) == 0.0
    for g in r["grads"].values():
        assert np.max(np.abs(g)) == 0.0


# P2 ------------------------------------------------------------------------
@pytest.mark.parametrize("arch", ["llama", "gpt2"])
@pytest.mark.parametrize("consis", ["reverse", "forward"])
def test_p2_identity_chunk(arch, consis):
    """Zero output projections make f_k the identity (Eq. (1)): KL = 0 and the
    loss is alpha * mean CE of the input's readout; branch weights get no
    gradient."""
    c = tiny_case(arch, alpha=0.6, consis=consis)
    P = dict(c["P"])
    zero = ["wo", "wd"] if arch == "llama" else ["wo", "wproj", "bo", "bproj"]
    for k in P:
        if k.split(".")[1] in zero:
            P[k] = np.zeros_like(P[k])
    r = _grads(c, P=P)
    np.testing.assert_array_equal(r["h_out"], c["h_in"])
    assert np.max(np.abs(r["info"]["kl"])) < 1e-14
    # textbook cross-entropy of the input's readout, via scipy's logsumexp
    from scipy.special import logsumexp
    T = c["h_in"].shape[0] * c["h_in"].shape[1]
    h = c["h_in"].reshape(T, -1)
    if arch == "llama":
        n = h / np.sqrt(np.mean(h ** 2, 1, keepdims=True) + 1e-5) * c["hn_w"]
    else:
        mu = h.mean(1, keepdims=True)
        n = (h - mu) / np.sqrt(h.var(1, keepdims=True) + 1e-5) * c["hn_w"] + c["hn_b"]
    z = n @ c["head_w"].T
    lab = c["labels"].reshape(-1)
    idx = lab != -100
    ce = logsumexp(z[idx], axis=1) - z[idx, lab[idx]]
    assert r["loss"] == pytest.approx(0.6 * ce.mean(), rel=1e-12)
    cut = ["wq", "wk", "wv", "wg", "wu", "ln1_w", "ln2_w"] if arch == "llama" else \
          ["wqkv", "bqkv", "wfc", "bfc", "ln1_w", "ln1_b", "ln2_w", "ln2_b"]
    for k, g in r["grads"].items():
        if k.split(".")[1] in cut:
            assert np.max(np.abs(g)) == 0.0, k
        if k.split(".")[1] in ("wo", "wd", "wproj"):
            assert np.max(np.abs(g)) > 0.0, k


# P3 / P4 -------------------------------------------------------------------
@pytest.mark.parametrize("arch", ["llama", "gpt2"])
def test_p3_single_chunk_is_backprop(arch):
    """K = 1, alpha = 1: the chunk-local update is ordinary BP on the final
    head (Remark 1: layers inside a chunk are updated by BP; L = L_task)."""
    c = tiny_case(arch, alpha=1.0)
    loc = _grads(c)
    glob = oracle.global_bp_ref(c["cfg"], [c["P"]], c["h_in"], c["labels"], c["head_w"], c["hn_w"],
                                c["hn_b"], c["seq_lens"], c["pos_ids"])
    assert loc["loss"] == pytest.approx(glob["loss"], rel=1e-14)
    for k in c["P"]:
        assert rel_err(loc["grads"][k], glob["grads"][0][k]) < 1e-12, k


def test_p4_last_chunk_block_diagonal():
    """K = 2, alpha = 1: the last chunk's local gradient equals the global-BP
    gradient restricted to it (block-diagonal Jacobian, Sec. II.C); the first
    chunk's differs, since no gradient crosses the chunk boundary."""
    c1 = tiny_case("llama", alpha=1.0, seed=0)
    c2 = tiny_case("llama", alpha=1.0, seed=1)
    cfg = c1["cfg"]
    args = (c1["labels"], c1["head_w"], c1["hn_w"], c1["hn_b"], c1["seq_lens"], c1["pos_ids"])
    glob = oracle.global_bp_ref(cfg, [c1["P"], c2["P"]], c1["h_in"], *args)
    h1, _ = chunk_forward_ref(cfg, c1["P"], c1["h_in"], c1["seq_lens"], c1["pos_ids"])
    loc2 = oracle.chunk_grads_ref(cfg, c2["P"], h1, *args)
    loc1 = oracle.chunk_grads_ref(cfg, c1["P"], c1["h_in"], *args)
    assert loc2["loss"] == pytest.approx(glob["loss"], rel=1e-13)
    for k in c2["P"]:
        assert rel_err(loc2["grads"][k], glob["grads"][1][k]) < 1e-12, k
    diffs = [rel_err(loc1["grads"][k], glob["grads"][0][k]) for k in c1["P"]]
    assert max(diffs) > 1e-3


# P5 ------------------------------------------------------------------------
def test_p5_detached_input():
    """No gradient to h_{k-1} is formed (Remark 1) and h_in is not modified."""
    c = tiny_case("llama")
    h = c["h_in"].copy()
    r = _grads(c)
    np.testing.assert_array_equal(c["h_in"], h)
    _, fw = chunk_forward_ref(c["cfg"], c["P"], c["h_in"], c["seq_lens"], c["pos_ids"])
    dx, _ = chunk_backward_ref(c["cfg"], r["dh_out"], fw, need_dx=False)
    assert dx is None
    # the same values reached through a different "upstream" give the same update
    r2 = _grads(c, h_in=np.array(c["h_in"] * 1.0))
    for k in c["P"]:
        np.testing.assert_array_equal(r["grads"][k], r2["grads"][k])


# P6 ------------------------------------------------------------------------
def test_p6_forward_kl_mixture_optimum():
    """Forward KL: alpha CE + (1-alpha) KL(q || p) is minimised over p by the
    arithmetic mixture alpha e_y + (1-alpha) q, where the logit gradient is 0."""
    rng = np.random.default_rng(3)
    T, V, alpha = 6, 9, 0.35
    zp = rng.standard_normal((T, V))
    q = np.exp(log_softmax(zp))
    y = rng.integers(0, V, T)
    mix = (1 - alpha) * q
    mix[np.arange(T), y] += alpha
    z = np.log(mix) + rng.standard_normal((T, 1))  # any row shift
    _, dz, _ = loss_and_dlogits(z, zp, y, alpha, "forward")
    assert np.max(np.abs(dz)) < 1e-15
    _, dz2, _ = loss_and_dlogits(z + 0.01 * rng.standard_normal((T, V)), zp, y, alpha, "forward")
    assert np.max(np.abs(dz2)) > 1e-4


# P7 ------------------------------------------------------------------------
def test_p7_lemma2_lemma3():
    """Lemma 2: alpha KL(p||t) + (1-alpha) KL(p||q) = KL(p||p*) - log Z with
    p* the normalised geometric mixture t^alpha q^(1-alpha).
    Lemma 3: grad_p L = log p - log p* + 1, so the logit gradient is the
    softmax Jacobian applied to it, and sums to zero over the vocabulary."""
    rng = np.random.default_rng(4)
    T, V = 7, 13
    for alpha in (0.2, 0.5, 0.9):
        z = rng.standard_normal((T, V)) * 2
        zp = rng.standard_normal((T, V))
        logt = log_softmax(rng.standard_normal((T, V)) * 3)
        L, dz = soft_target_objective(z, logt, zp, alpha)
        logq = log_softmax(zp)
        logw = alpha * logt + (1 - alpha) * logq
        logZ = np.log(np.sum(np.exp(logw), axis=1))
        logpstar = logw - logZ[:, None]
        logp = log_softmax(z)
        p = np.exp(logp)
        kl_star = np.sum(p * (logp - logpstar), axis=1)
        np.testing.assert_allclose(L, kl_star - logZ, rtol=1e-12, atol=1e-13)
        gp = logp - logpstar + 1.0
        jac = p * (gp - np.sum(p * gp, axis=1, keepdims=True))
        np.testing.assert_allclose(dz, jac, rtol=1e-11, atol=1e-14)
        np.testing.assert_allclose(dz.sum(1), 0.0, atol=1e-14)


@pytest.mark.parametrize("consis", ["reverse", "forward"])
def test_p7_logit_gradient_rows_sum_to_zero(consis):
    """Softmax shift invariance: each row of dL/dz sums to 0; unlabelled rows are 0."""
    c = tiny_case("llama", alpha=0.5, consis=consis)
    rng = np.random.default_rng(8)
    z = rng.standard_normal((10, 11))
    zp = rng.standard_normal((10, 11))
    lab = c["labels"].reshape(-1)
    _, dz, _ = loss_and_dlogits(z, zp, lab, 0.5, consis)
    np.testing.assert_allclose(dz.sum(1), 0.0, atol=1e-15)
    assert np.all(dz[lab == -100] == 0.0)


# P8 ------------------------------------------------------------------------
def test_p8_attention_and_rope():
    rng = np.random.default_rng(5)
    B, Hq, Hkv, hd = 2, 4, 2, 8
    q = rng.standard_normal((B, 1, Hq, hd))
    k = rng.standard_normal((B, 1, Hkv, hd))
    v = rng.standard_normal((B, 1, Hkv, hd))
    o, _ = ops.attention_fwd(q, k, v, np.array([1, 1]))
    np.testing.assert_allclose(o, np.repeat(v, 2, axis=2))          # S = 1 returns v
    S = 6
    k = rng.standard_normal((B, S, Hkv, hd))
    v = rng.standard_normal((B, S, Hkv, hd))
    o, _ = ops.attention_fwd(np.zeros((B, S, Hq, hd)), k, v, np.array([S, 4]))
    for i in range(S):                                              # uniform scores -> prefix mean
        np.testing.assert_allclose(o[0, i, 0], v[0, : i + 1, 0].mean(0), atol=1e-14)
        np.testing.assert_allclose(o[1, i, 3], v[1, : min(i + 1, 4), 1].mean(0), atol=1e-14)
    q = rng.standard_normal((B, S, Hq, hd))
    o1, _ = ops.attention_fwd(q, k, v, np.array([S, S]))
    k2, v2 = k.copy(), v.copy()
    k2[:, 4] += 1.0
    v2[:, 4] -= 2.0
    o2, _ = ops.attention_fwd(q, k2, v2, np.array([S, S]))          # causality
    np.testing.assert_array_equal(o1[:, :4], o2[:, :4])
    assert np.max(np.abs(o1[:, 4:] - o2[:, 4:])) > 1e-3
    # RoPE: position 0 is the identity, norms are kept, and scores depend on m - n only
    u = rng.standard_normal((1, 8, 1, hd))
    pos = np.arange(8)[None]
    ang = ops.rope_angles(pos, hd, 1e4)
    ru = ops.rope_fwd(u, ang)
    np.testing.assert_allclose(ru[0, 0], u[0, 0], atol=0)
    np.testing.assert_allclose(np.linalg.norm(ru, axis=-1), np.linalg.norm(u, axis=-1), rtol=1e-14)
    qv, kv = rng.standard_normal(hd), rng.standard_normal(hd)
    def score(m, n):
        a = ops.rope_fwd(qv[None, None, None], ops.rope_angles(np.array([[m]]), hd, 1e4))
        b = ops.rope_fwd(kv[None, None, None], ops.rope_angles(np.array([[n]]), hd, 1e4))
        return float(np.sum(a * b))
    assert score(5, 2) == pytest.approx(score(13, 10), rel=1e-12)
    # rotate-half RoPE as multiplication by e^{i pos theta_j} of the complex pairs (u_j, u_{j+h})
    half = hd // 2
    cpx = (u[..., :half] + 1j * u[..., half:]) * np.exp(1j * ang[:, :, None, :])
    np.testing.assert_allclose(ru[..., :half], cpx.real, atol=1e-14)
    np.testing.assert_allclose(ru[..., half:], cpx.imag, atol=1e-14)


# P9 ------------------------------------------------------------------------
@pytest.mark.parametrize("case", GOLD["adamw_first_step"]["cases"])
def test_p9_adamw_first_step(case):
    g = GOLD["adamw_first_step"]
    new, m, v = oracle.adamw_step_ref(np.array(case["theta"]), np.array(case["g"]), 0.0, 0.0, 1,
                                      g["lr"], 0.9, 0.999, g["eps"], g["wd"])
    assert float(new - case["theta"]) == pytest.approx(case["delta"], rel=1e-12, abs=1e-18)


def test_p9_sgd_step():
    th, gr = np.array([1.0, -2.0]), np.array([0.5, 0.25])
    np.testing.assert_allclose(oracle.sgd_step_ref(th, gr, 0.1) - th, -0.1 * gr, rtol=0, atol=1e-16)


# P10 -----------------------------------------------------------------------
def test_p10_window_accumulation():
    """Two micro-batches with grad_scale 1/2 and equal |Omega| give the same
    gradient as one batch holding both (Sec. III-B S3)."""
    c = tiny_case("llama", pad=False, drop_labels=False, B=4)
    cfg = c["cfg"]
    mbs = [dict(h_in=c["h_in"][i:i + 2], labels=c["labels"][i:i + 2], seq_lens=c["seq_lens"][i:i + 2],
                pos_ids=c["pos_ids"][i:i + 2]) for i in (0, 2)]
    hw = (c["head_w"], c["hn_w"], c["hn_b"])
    win = oracle.chunk_update_ref(cfg, c["P"], init_opt_state(), mbs, *hw, grad_scale=0.5)
    one = oracle.chunk_update_ref(cfg, c["P"], init_opt_state(),
                                  [dict(h_in=c["h_in"], labels=c["labels"], seq_lens=c["seq_lens"],
                                        pos_ids=c["pos_ids"])], *hw, grad_scale=1.0)
    for k in c["P"]:
        assert rel_err(win["grads"][k], one["grads"][k]) < 1e-13, k
        assert rel_err(win["params"][k], one["params"][k]) < 1e-13, k


def test_empty_omega():
    """|Omega| = 0: loss 0 and zero gradient (mean over an empty set read as 0)."""
    c = tiny_case("gpt2")
    c["labels"][:] = -100
    r = _grads(c)
    assert r["loss"] == 0.0
    for g in r["grads"].values():
        assert np.max(np.abs(g)) == 0.0


def test_bf16_mode_rounds_matrices_only():
    c = tiny_case("gpt2", alpha=0.5)
    cfg = c["cfg"]
    cfg.dtype = "bf16"
    P = oracle.chunk.effective_params(cfg, c["P"])
    for k, v in P.items():
        if v.ndim == 2:
            np.testing.assert_array_equal(v, oracle.bf16_round(v))
            assert rel_err(v, c["P"][k]) < 4e-3
        else:
            np.testing.assert_array_equal(v, c["P"][k])
    # bf16 rounding: nearest, ties to even, on exactly representable boundaries
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -3.5, 65504.0])
    np.testing.assert_array_equal(oracle.bf16_round(x),
                                  [1.0, 1.0, 1.0 + 2 ** -6, 1.0, -3.5, 65536.0])


def _adapter_case(arch, w1_zero=False, w2_zero=False):
    c = tiny_case(arch, alpha=0.5, adapter_rank=3)
    L = c["shape"].n_layers
    if w1_zero:
        c["P"][f"L{L}.ad_w1"] = np.zeros_like(c["P"][f"L{L}.ad_w1"])
    if w2_zero:
        c["P"][f"L{L}.ad_w2"] = np.zeros_like(c["P"][f"L{L}.ad_w2"])
    base = tiny_case(arch, alpha=0.5)  # same seeds, no adapter
    return c, base, L


def _adapter_grads(c):
    return oracle.chunk_grads_ref(c["cfg"], c["P"], c["h_in"], c["labels"], c["head_w"], c["hn_w"],
                                  c["hn_b"], c["seq_lens"], c["pos_ids"])


@pytest.mark.parametrize("arch", ["llama", "gpt2"])
def test_p11_adapter_is_identity_at_zero_output(arch):
    """Readout adapter (Sec. III-B (b)) with W2 = 0: exactly the static head,
    and no gradient reaches W1 (it only acts through W2)."""
    c, base, L = _adapter_case(arch, w2_zero=True)
    r, r0 = _adapter_grads(c), _adapter_grads(base)
    assert r["loss"] == r0["loss"]
    np.testing.assert_array_equal(r["dh_out"], r0["dh_out"])
    assert not np.any(r["grads"][f"L{L}.ad_w1"])
    for k in r0["grads"]:
        np.testing.assert_array_equal(r["grads"][k], r0["grads"][k])


@pytest.mark.parametrize("arch", ["llama", "gpt2"])
def test_p11_adapter_gradient_at_zero_input(arch):
    """W1 = 0: h' = h (gelu(0) = 0), so dW2 = 0 and, with gelu'(0) = 1/2,
    dW1 = 1/2 W2^T (dL/dh)^T h with dL/dh the static-head gradient."""
    c, base, L = _adapter_case(arch, w1_zero=True)
    r, r0 = _adapter_grads(c), _adapter_grads(base)
    assert abs(r["loss"] - r0["loss"]) < 1e-13
    assert not np.any(r["grads"][f"L{L}.ad_w2"])
    B, S, d = c["h_in"].shape
    h = r0["h_out"].reshape(B * S, d)
    dh = r0["dh_out"].reshape(B * S, d)
    want = 0.5 * c["P"][f"L{L}.ad_w2"].T @ (dh.T @ h)
    assert rel_err(r["grads"][f"L{L}.ad_w1"], want) < 1e-12


def _lora_run(c, P):
    return oracle.chunk_grads_ref(c["cfg"], P, c["h_in"], c["labels"], c["head_w"], c["hn_w"],
                                  c["hn_b"], c["seq_lens"], c["pos_ids"])


@pytest.mark.parametrize("arch", ["llama", "gpt2"])
def test_p12_lora_with_zero_B_is_the_base_model(arch):
    """Eq. (6) LoRA with B = 0: the base model exactly, and dA = 0 (the A
    factors act only through B)."""
    c = tiny_case(arch, alpha=0.5, lora_rank=2)
    P = {k: (np.zeros_like(v) if k.endswith("_lb") else v) for k, v in c["P"].items()}
    base_cfg = oracle.OracleConfig.from_shape(c["shape"].with_(lora_rank=0), alpha=0.5)
    base = {k: v for k, v in P.items() if not (k.endswith("_la") or k.endswith("_lb"))}
    r = _lora_run(c, P)
    r0 = oracle.chunk_grads_ref(base_cfg, base, c["h_in"], c["labels"], c["head_w"], c["hn_w"],
                                c["hn_b"], c["seq_lens"], c["pos_ids"])
    assert r["loss"] == r0["loss"]
    np.testing.assert_array_equal(r["dh_out"], r0["dh_out"])
    assert set(r["grads"]) == set(c["trainable"])
    for k in c["trainable"]:
        if k.endswith("_la"):
            assert not np.any(r["grads"][k]), k


@pytest.mark.parametrize("arch", ["llama", "gpt2"])
def test_p12_lora_equals_merged_weight_update(arch):
    """x W^T + s (x A^T) B^T = x (W + s B A)^T, so the LoRA loss equals the
    full chunk's with W' = W + s B A, and the chain rule through W' gives
    dB = s dW' A^T, dA = s B^T dW' from the full chunk's gradient dW'."""
    c = tiny_case(arch, alpha=0.5, lora_rank=2, lora_alpha=3.0)
    s = c["cfg"].lora_scale
    r = _lora_run(c, c["P"])
    merged, pairs = {}, []
    for k, v in c["P"].items():
        if k.endswith("_la") or k.endswith("_lb"):
            continue
        a, b = c["P"].get(k + "_la"), c["P"].get(k + "_lb")
        merged[k] = v + s * b @ a if a is not None else v
        if a is not None:
            pairs.append((k, a, b))
    full_cfg = oracle.OracleConfig.from_shape(c["shape"].with_(lora_rank=0), alpha=0.5)
    rf = oracle.chunk_grads_ref(full_cfg, merged, c["h_in"], c["labels"], c["head_w"], c["hn_w"],
                                c["hn_b"], c["seq_lens"], c["pos_ids"])
    assert abs(r["loss"] - rf["loss"]) < 1e-12 * max(1.0, abs(rf["loss"]))
    assert len(pairs) == (7 if arch == "llama" else 4) * c["shape"].n_layers
    for k, a, b in pairs:
        dW = rf["grads"][k]
        assert rel_err(r["grads"][k + "_lb"], s * dW @ a.T) < 1e-10, k
        assert rel_err(r["grads"][k + "_la"], s * b.T @ dW) < 1e-10, k


def test_p12_lora_update_moves_only_the_factors():
    c = tiny_case("llama", alpha=0.5, lora_rank=2)
    mb = dict(h_in=c["h_in"], labels=c["labels"], seq_lens=c["seq_lens"], pos_ids=c["pos_ids"])
    out = oracle.chunk_update_ref(c["cfg"], c["P"], init_opt_state(), [mb], c["head_w"], c["hn_w"],
                                  c["hn_b"])
    for k, v in c["P"].items():
        if k in c["trainable"]:
            assert np.any(out["params"][k] != v), k
        else:
            np.testing.assert_array_equal(out["params"][k], v, err_msg=k)
