"""End-to-end parity of the chunk-local update: libzl through the C ABI vs
the fp64 oracle on the same seeded inputs.

Gates (tests/parity.py): per tensor the relative error and the worst row and
column against a typical row (column) of the oracle's tensor.  fp32: 1e-4 on
everything (rows and columns 1e-3).  bf16: the loss and the updated master
parameters at 2e-2; h_out, dL/dh_out and every gradient at the larger of
2e-2 and 1.5x the bf16 storage floor of the same tensor on the same inputs
(the oracle run with bf16-rounded stored intermediates, reading r4; stored
in tests/golden/bf16_floor.json), rows and columns at the larger of 0.1 and
1.5x their floor; update deltas: SGD like the gradient, AdamW on the
elements whose first-step gradient is resolvable in the precision."""
import numpy as np
import pytest

import oracle
import workload
from oracle.chunk import chunk_forward_ref, init_opt_state
from tests.gpu_cases import (case_inputs, device_chunk, make_inputs, oracle_cfg, oracle_run,
                             rel_err, to_dev)
from tests.parity import TOL, gate, load_floor

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _run_device(shp, params, batch, steps=1, **kw):
    ch = device_chunk(shp, params, batch, **kw)
    d = to_dev(batch, shp.dtype)
    out = dict(grads=[], masters=[ch.tensors(ch.master)], losses=[], moments=[])
    adam = ch.adam_m is not None
    for _ in range(steps):
        if adam:  # the optimizer state entering this step
            out["moments"].append((ch.tensors(ch.adam_m), ch.tensors(ch.adam_v)))
        h_out = ch.forward(d["h_in"], d["seq_lens"], d["pos_ids"])
        ch.objective(d["labels"])
        if not out["grads"]:
            out["h_out"] = h_out.double().cpu().numpy()
            out["dh_out"] = ch.inspect("dh_out")
        ch.backward(1.0, 0)
        torch.cuda.synchronize()
        out["losses"].append(float(ch.loss.item()))
        out["grads"].append(ch.tensors(ch.grad))
        ch.step()
        out["masters"].append(ch.tensors(ch.master))
    out["h_in_after"] = d["h_in"].double().cpu().numpy()
    _check_lora_padding(ch)
    if ch.base_master is not None:  # LoRA: the frozen base is never written
        torch.cuda.synchronize()
        for k, t in ch.base_by_key.items():
            got = ch.base_master[t["offset"]: t["offset"] + t["numel"]].cpu().numpy()
            np.testing.assert_array_equal(got, np.asarray(params[k], np.float32).reshape(-1), err_msg=k)
    ch.close()
    return out


def _check_lora_padding(ch):
    """A LoRA rank below its stored width: the padding of every factor is
    exactly zero in master, shadow, gradient and the AdamW moments."""
    torch.cuda.synchronize()
    for key in ch.by_key:
        for buf in (ch.master, ch.shadow, ch.grad, ch.adam_m, ch.adam_v):
            if buf is not None:
                pad = ch.padding(buf, key)
                assert pad.numel() == 0 or not bool(pad.float().abs().max() > 0), key


def _window_device(shp, params, batches, **kw):
    """m micro-batches, grad_scale 1/m, accumulate, then one step (S3)."""
    ch = device_chunk(shp, params, batches[0], **kw)
    out = dict(losses=[], masters=[ch.tensors(ch.master)])
    for b in batches:
        d = to_dev(b, shp.dtype)
        h_out = ch.forward(d["h_in"], d["seq_lens"], d["pos_ids"])
        ch.objective(d["labels"])
        out["h_out"] = h_out.double().cpu().numpy()  # of the last micro-batch
        out["dh_out"] = ch.inspect("dh_out")
        ch.backward(1.0 / len(batches), 1)
        torch.cuda.synchronize()
        out["losses"].append(float(ch.loss.item()))
    out["grads"] = [ch.tensors(ch.grad)]
    ch.step()
    out["masters"].append(ch.tensors(ch.master))
    ch.close()
    return out


def _case(shp, steps=1, seed=0, stress=True, seq_lens=None, drop=0, alpha=0.5, consis="reverse",
          optimizer="adamw", lr=1e-4, wd=0.01, h_in=None):
    """An fp32 case, gated at 1e-4."""
    assert shp.dtype == "f32"
    params, batch = make_inputs(shp, seed=seed, stress=stress, seq_lens=seq_lens, drop=drop)
    if h_in is not None:
        batch["h_in"] = h_in
    kw = dict(alpha=alpha, consis=consis, optimizer=optimizer, lr=lr, wd=wd)
    dev = _run_device(shp, params, batch, steps=steps, **kw)
    ref = oracle_run(shp, params, batch, steps=steps, **kw)
    np.testing.assert_array_equal(dev["h_in_after"].astype(np.float32), batch["h_in"])
    return gate(dev, ref, "f32", optimizer)


def _named(name):
    """A bf16 case of tests.gpu_cases.BF16_CASES, gated against its floor."""
    shp, kw, steps, params, batch = case_inputs(name)
    if isinstance(batch, list):
        floor = load_floor(name, params, batch[0])
        dev = _window_device(shp, params, batch, **kw)
        from tests.gpu_cases import oracle_window
        ref = oracle_window(shp, params, batch, **kw)
    else:
        floor = load_floor(name, params, batch)
        dev = _run_device(shp, params, batch, steps=steps, **kw)
        ref = oracle_run(shp, params, batch, steps=steps, **kw)
        np.testing.assert_array_equal(dev["h_in_after"].astype(np.float32), batch["h_in"])
        if steps > 1:
            return _gate_steps(shp, kw, params, batch, dev, ref,
                               load_floor(name, params, batch, per_step=True))
    return gate(dev, ref, "bf16", kw["optimizer"], floor)


def _gate_steps(shp, kw, params, batch, dev, ref, floors):
    """Several bf16 steps.  The trajectories of device and oracle drift apart
    by bf16 noise that Adam's sign-like first steps amplify, so each step is
    gated from the state the device reached: the oracle runs that step from
    the device's parameters and AdamW moments (step s's gradients, delta and
    loss), against the floors of step s (measured from the same step of the
    exact trajectory).  The whole trajectory is gated at the stated
    tolerance on every step's loss and the final parameters."""
    from oracle.chunk import chunk_update_ref
    cfg = oracle_cfg(shp, **kw)
    mb = dict(h_in=batch["h_in"], labels=batch["labels"], seq_lens=batch["seq_lens"],
              pos_ids=batch["pos_ids"])
    frozen = {k: np.asarray(v, np.float64) for k, v in params.items() if k not in dev["masters"][0]}
    out = {}
    for s in range(len(dev["grads"])):
        P = dict(frozen, **dev["masters"][s])
        if dev["moments"]:
            m, v = dev["moments"][s]
            state = dict(m=m, v=v, t=s)
        else:
            state = init_opt_state()
        r = chunk_update_ref(cfg, P, state, [mb], batch["head_w"], batch["head_norm_w"],
                             batch["head_norm_b"], grad_scale=1.0)
        one_dev = dict(losses=[dev["losses"][s]], grads=[dev["grads"][s]],
                       masters=[dev["masters"][s], dev["masters"][s + 1]])
        one_ref = dict(losses=r["losses"], grads=[r["grads"]],
                       masters=[{k: P[k] for k in dev["masters"][s]},
                                {k: r["params"][k] for k in dev["masters"][s]}])
        if s == 0:
            one_dev.update(h_out=dev["h_out"], dh_out=dev["dh_out"])
            one_ref.update(h_out=ref["h_out"], dh_out=ref["dh_out"])
        for k, v in gate(one_dev, one_ref, "bf16", kw["optimizer"], floors[s]).items():
            out[f"step{s}/{k}"] = v
    for s, (a, b) in enumerate(zip(dev["losses"], ref["losses"])):
        assert abs(a - b) <= TOL["bf16"] * abs(b), ("trajectory loss", s, a, b)
    last = len(dev["masters"]) - 1
    for k in dev["masters"][last]:
        e = rel_err(dev["masters"][last][k], ref["masters"][last][k])
        assert e < TOL["bf16"], ("trajectory parameters", k, e)
    return out


# ----------------------------------------------------------------- fp32 tiny
TINY = workload.get_config("tiny")


@pytest.mark.parametrize("alpha,consis", [(0.5, "reverse"), (1.0, "reverse"), (0.3, "forward"),
                                         (0.05, "reverse"), (0.05, "forward")])
def test_tiny_fp32_chunk1(alpha, consis):
    """alpha = 1: cross-entropy only; alpha = 0.05: almost all consistency
    term (Eq. (3); alpha is read as a weight in (0, 1]), both KL directions."""
    _case(TINY, alpha=alpha, consis=consis)


def test_tiny_fp32_chunk2_input_from_chunk1():
    """Chunk k = 2 of 2: its input is chunk 1's output (oracle forward)."""
    p1, b1 = make_inputs(TINY, seed=0)
    cfg = oracle_cfg(TINY)
    h1, _ = chunk_forward_ref(cfg, p1, b1["h_in"], b1["seq_lens"], b1["pos_ids"])
    _case(TINY, seed=1, h_in=h1.astype(np.float32))


def test_tiny_fp32_padding_and_ignored_labels():
    _case(TINY, seq_lens=[32, 17, 1, 9], drop=20, alpha=0.6)


def test_tiny_fp32_three_adamw_steps():
    _case(TINY, steps=3, lr=1e-3)


def test_tiny_fp32_sgd():
    _case(TINY, optimizer="sgd", lr=0.05, alpha=0.7, consis="forward")


def test_tiny_gqa_fp32():
    shp = TINY.with_(n_kv_heads=2, name="tiny-gqa")
    _case(shp, alpha=0.4)


def test_tiny_gpt2_fp32():
    shp = workload.configs.ChunkShape("tiny-gpt2", "gpt2", 2, 64, 4, 4, 16, 256, 97, 4, 24, "f32",
                                      0.0, 2)
    _case(shp, alpha=0.5, seq_lens=[24, 20, 3, 24])


# ---------------------------------------------------------- window (m = 2)
def test_window_accumulation_fp32():
    """Two micro-batches with their own tokens, grad_scale 1/2, accumulate
    -> one step (S3)."""
    shp = TINY
    params, b1 = make_inputs(shp, seed=0, tokens_seed=1)
    _, b2 = make_inputs(shp, seed=0, tokens_seed=6)
    for k in ("head_w", "head_norm_w", "head_norm_b"):
        b2[k] = b1[k]
    assert not np.array_equal(b1["labels"], b2["labels"])
    from tests.gpu_cases import oracle_window
    dev = _window_device(shp, params, [b1, b2])
    ref = oracle_window(shp, params, [b1, b2])
    gate(dev, ref, "f32", "adamw")


# --------------------------------------------------------------- bf16 shapes
def test_llama1b_bf16_lora_window_two_microbatches():
    """The window in bf16 with LoRA at T = 512: the factor weight gradients
    split K, so the second micro-batch adds its split partials into the
    first one's gradient."""
    _named("1b_lora_window")


def test_gpt2_bf16_reduced_tokens():
    _named("gpt2_reduced")


def test_gpt2_bf16_sgd_delta():
    _named("gpt2_sgd_forward_kl")


def test_gpt2_bf16_full_shape():
    _named("gpt2_full")


def test_llama1b_bf16_one_layer_slice():
    _named("1b_slice")


def test_llama8b_bf16_one_layer_slice():
    _named("8b_slice")


def test_llama8b_bf16_two_layers_alpha1_sgd():
    _named("8b_two_layers_sgd")


def test_llama1b_bf16_ragged_tokens():
    """200 tokens: the last row tile and 32-row epilogue block of every GEMM
    are partial (residual, RoPE, SwiGLU backward, delta and logit
    epilogues)."""
    _named("1b_ragged")


def test_llama1b_bf16_confident_logits():
    """Logits up to about 30 with the label its row's most likely token:
    dL/dz = p - 1 at the label is a small difference of large terms, and the
    fp16 logit cache must resolve p there."""
    _named("1b_confident_logits")


# ------------------------------------------------------ readout adapter
@pytest.mark.parametrize("alpha", [0.5, 1.0])
def test_tiny_fp32_readout_adapter(alpha):
    _case(TINY.with_(adapter_rank=16), alpha=alpha, seq_lens=[32, 17, 1, 9], drop=5)


def test_tiny_fp32_readout_adapter_three_steps():
    _case(TINY.with_(adapter_rank=16), steps=3, lr=1e-3)


def test_tiny_gpt2_fp32_readout_adapter():
    shp = workload.configs.ChunkShape("tiny-gpt2", "gpt2", 2, 64, 4, 4, 16, 256, 97, 4, 24, "f32",
                                      0.0, 2, adapter_rank=32)
    _case(shp, alpha=0.5)


def test_gpt2_bf16_readout_adapter():
    _named("gpt2_adapter")


def test_llama1b_bf16_one_layer_readout_adapter():
    _named("1b_adapter")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_readout_adapter_with_zero_output_is_the_static_head(dtype):
    """W2 = 0: loss, dL/dh_out and every layer gradient equal those of the
    chunk without an adapter bit for bit, and dW1 is exactly 0."""
    shp = TINY.with_(dtype=dtype)
    params, batch = make_inputs(shp, seed=0)
    shp_a = shp.with_(adapter_rank=16)
    pa = workload.init_params(workload.param_specs(shp_a), seed=0, perturb=False)
    L = shp.n_layers
    params_a = dict(params, **{f"L{L}.ad_w1": pa[f"L{L}.ad_w1"],
                               f"L{L}.ad_w2": np.zeros_like(pa[f"L{L}.ad_w2"])})
    out = []
    for s, p in ((shp, params), (shp_a, params_a)):
        ch = device_chunk(s, p, batch)
        d = to_dev(batch, dtype)
        ch.forward(d["h_in"], d["seq_lens"], d["pos_ids"])
        ch.objective(d["labels"])
        dh = ch.inspect("dh_out")
        ch.backward(1.0, 0)
        torch.cuda.synchronize()
        out.append((float(ch.loss.item()), dh, ch.tensors(ch.grad)))
        ch.close()
    (l0, dh0, g0), (l1, dh1, g1) = out
    assert l0 == l1
    np.testing.assert_array_equal(dh0, dh1)
    for k in g0:
        np.testing.assert_array_equal(g0[k], g1[k], err_msg=k)
    assert not np.any(g1[f"L{L}.ad_w1"])


# ------------------------------------------------------------------- LoRA
# Eq. (6) on the LoRA factors of Sec. II.A: every linear is
# x W^T + s (x A^T) B^T with W, norms and biases frozen.
@pytest.mark.parametrize("alpha", [0.5, 1.0])
def test_tiny_fp32_lora(alpha):
    _case(TINY.with_(lora_rank=8, lora_alpha=24.0), alpha=alpha, seq_lens=[32, 17, 1, 9], drop=5)


def test_tiny_fp32_lora_with_adapter_three_steps():
    _case(TINY.with_(lora_rank=8, adapter_rank=16), steps=3, lr=1e-3)


def test_tiny_gqa_fp32_lora_sgd():
    _case(TINY.with_(n_kv_heads=2, name="tiny-gqa", lora_rank=16), optimizer="sgd", lr=0.05,
          alpha=0.7, consis="forward")


def test_tiny_gpt2_fp32_lora():
    shp = workload.configs.ChunkShape("tiny-gpt2", "gpt2", 2, 64, 4, 4, 16, 256, 97, 4, 24, "f32",
                                      0.0, 2, lora_rank=16)
    _case(shp, alpha=0.5, seq_lens=[24, 20, 3, 24])


def test_gpt2_bf16_lora():
    _named("gpt2_lora")


def test_llama1b_bf16_one_layer_lora():
    _named("1b_lora")


def test_llama8b_bf16_two_layers_lora():
    _named("8b_two_layers_lora")


def test_tiny_fp32_lora_rank4_three_adamw_steps():
    """The paper's LoRA setting, rank 4 with scaling factor 16 (s = 4),
    against the unpadded rank-4 oracle over three AdamW steps; the padding
    of the stored rank-8 factors stays exactly zero."""
    _case(TINY.with_(lora_rank=4, lora_alpha=16.0), steps=3, lr=1e-3, seq_lens=[32, 17, 1, 9],
          drop=5)


def test_lora_rank4_padding_is_zeroed_at_load():
    """Non-zero values left in the padding before the parameters are loaded
    are cleared by zl_refresh_shadow, so the chunk computes rank 4."""
    shp = TINY.with_(lora_rank=4, lora_alpha=16.0)
    params, batch = make_inputs(shp)
    ch = device_chunk(shp, params, batch)
    for key in ch.by_key:
        ch.padding(ch.master, key).fill_(1.0)
    ch.load_params({k: v for k, v in params.items() if k in ch.by_key})
    _check_lora_padding(ch)
    ch.close()


def test_llama1b_bf16_lora_rank4_three_adamw_steps():
    _named("1b_lora_r4")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_lora_with_zero_B_is_the_base_chunk(dtype):
    """B = 0: the chunk computes its base model, so the loss and dL/dh_out
    equal those of the full chunk with the same weights bit for bit, and
    dA = s (dy B)^T x is exactly 0."""
    shp = TINY.with_(dtype=dtype)
    shp_l = shp.with_(lora_rank=8)
    params, batch = make_inputs(shp_l, seed=0)
    params = {k: (np.zeros_like(v) if k.endswith("_lb") else v) for k, v in params.items()}
    full = {k: params[k] for k, _, _ in workload.base_specs(shp)}
    out = []
    for s, p in ((shp, full), (shp_l, params)):
        ch = device_chunk(s, p, batch)
        d = to_dev(batch, dtype)
        h = ch.forward(d["h_in"], d["seq_lens"], d["pos_ids"])
        ch.objective(d["labels"])
        dh = ch.inspect("dh_out")
        ch.backward(1.0, 0)
        torch.cuda.synchronize()
        out.append((float(ch.loss.item()), h.double().cpu().numpy(), dh, ch.tensors(ch.grad)))
        ch.close()
    (l0, h0, dh0, _), (l1, h1, dh1, g1) = out
    assert l0 == l1
    np.testing.assert_array_equal(h0, h1)
    np.testing.assert_array_equal(dh0, dh1)
    for k, g in g1.items():
        if k.endswith("_la"):
            assert not np.any(g), k
        else:
            assert np.all(np.isfinite(g)) and np.any(g), k
