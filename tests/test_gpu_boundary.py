"""Behaviour of the C ABI on the GPU: call order, argument checks, input
immutability, defaults, the empty labelled set, and determinism."""
import numpy as np
import pytest

import workload
from tests.gpu_cases import device_chunk, make_inputs, to_dev

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TINY = workload.get_config("tiny")


def _zl():
    from paper_2608_07974_amd import zl
    return zl


def _setup(shp=TINY, **kw):
    params, batch = make_inputs(shp, seed=0)
    return device_chunk(shp, params, batch, **kw), to_dev(batch, shp.dtype), params, batch


def test_call_order_errors():
    zl = _zl()
    ch, d, _, _ = _setup()
    with pytest.raises(zl.ZlError) as e:
        ch.objective(d["labels"])
    assert e.value.status == zl.ZL_ERR_STATE
    with pytest.raises(zl.ZlError) as e:
        ch.backward()
    assert e.value.status == zl.ZL_ERR_STATE
    with pytest.raises(zl.ZlError) as e:
        ch.step()
    assert e.value.status == zl.ZL_ERR_STATE
    ch.forward(d["h_in"])
    with pytest.raises(zl.ZlError) as e:
        ch.backward()
    assert e.value.status == zl.ZL_ERR_STATE
    ch.objective(d["labels"])
    ch.backward()
    ch.step()
    assert zl.zl_get_step(ch.handle) == 1
    with pytest.raises(zl.ZlError) as e:
        ch.step()
    assert e.value.status == zl.ZL_ERR_STATE
    ch.close()


def test_argument_errors_launch_nothing():
    zl = _zl()
    ch, d, _, _ = _setup()
    before = ch.master.clone()
    with pytest.raises(zl.ZlError) as e:
        zl.zl_chunk_forward(ch.handle, d["h_in"].data_ptr(), 0, 0, TINY.batch, TINY.seq,
                            d["h_in"].data_ptr(), 0)
    assert e.value.status == zl.ZL_ERR_INVALID_ARG
    big = torch.zeros(TINY.batch + 1, TINY.seq, TINY.d_model, dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):  # the binding refuses before any call
        ch.forward(big)
    out = torch.empty_like(big)
    with pytest.raises(zl.ZlError) as e:  # and so does the library
        zl.zl_chunk_forward(ch.handle, big.data_ptr(), 0, 0, TINY.batch + 1, TINY.seq,
                            out.data_ptr(), 0)
    assert e.value.status == zl.ZL_ERR_INVALID_ARG
    with pytest.raises(zl.ZlError) as e:
        zl.zl_chunk_backward(ch.handle, float("nan"), 0, 0)
    torch.cuda.synchronize()
    assert torch.equal(before, ch.master)
    ch.close()


def test_defaults_match_explicit_and_input_untouched():
    ch, d, _, _ = _setup()
    h0 = d["h_in"].clone()
    a = ch.forward(d["h_in"], None, None).clone()
    ch.objective(d["labels"])
    la = float(ch.loss.item())
    b = ch.forward(d["h_in"], d["seq_lens"], d["pos_ids"]).clone()
    ch.objective(d["labels"])
    lb = float(ch.loss.item())
    assert torch.equal(a, b) and la == lb
    assert torch.equal(h0, d["h_in"])
    ch.close()


def test_empty_omega_gives_zero_loss_and_gradient():
    ch, d, _, _ = _setup()
    lab = torch.full_like(d["labels"], -100)
    ch.forward(d["h_in"])
    ch.objective(lab)
    ch.backward()
    torch.cuda.synchronize()
    assert float(ch.loss.item()) == 0.0
    assert float(ch.grad.abs().max().item()) == 0.0
    ch.close()


def test_out_of_range_labels_count_as_ignored():
    ch, d, _, _ = _setup()
    lab = d["labels"].clone()
    ch.forward(d["h_in"])
    ch.objective(lab)
    l1 = float(ch.loss.item())
    lab2 = lab.clone()
    lab2[lab2 == -100] = TINY.vocab + 5
    ch.forward(d["h_in"])
    ch.objective(lab2)
    assert float(ch.loss.item()) == l1
    ch.close()


@pytest.mark.parametrize("name", ["tiny", "gpt2"])
def test_deterministic_updates(name):
    shp = workload.get_config(name)
    if name == "gpt2":
        shp = shp.with_(batch=2, seq=64)
    runs = []
    for _ in range(2):
        ch, d, _, _ = _setup(shp)
        ch.forward(d["h_in"], d["seq_lens"], d["pos_ids"])
        ch.objective(d["labels"])
        ch.backward()
        ch.step()
        torch.cuda.synchronize()
        runs.append((float(ch.loss.item()), ch.grad.clone(), ch.master.clone()))
        ch.close()
    assert runs[0][0] == runs[1][0]
    assert torch.equal(runs[0][1], runs[1][1])
    assert torch.equal(runs[0][2], runs[1][2])


def test_first_backward_after_step_overwrites():
    """accumulate=1 right after a step starts the new window from zero."""
    import oracle
    from oracle.chunk import init_opt_state
    from tests.gpu_cases import oracle_cfg, rel_err
    ch, d, params, batch = _setup()
    ch.forward(d["h_in"]); ch.objective(d["labels"]); ch.backward(1.0, 0)
    torch.cuda.synchronize()
    g1 = ch.grad.clone()
    ch.step()
    ch.forward(d["h_in"]); ch.objective(d["labels"]); ch.backward(1.0, 1)
    torch.cuda.synchronize()
    g2 = ch.tensors(ch.grad)
    cfg = oracle_cfg(TINY)
    mb = dict(h_in=batch["h_in"], labels=batch["labels"])
    r1 = oracle.chunk_update_ref(cfg, params, init_opt_state(), [mb], batch["head_w"],
                                 batch["head_norm_w"])
    r2 = oracle.chunk_update_ref(cfg, r1["params"], r1["state"], [mb], batch["head_w"],
                                 batch["head_norm_w"])
    for k in params:   # the fresh second-step gradient, not g1 + g2
        assert rel_err(g2[k], r2["grads"][k]) < 1e-4, k
    ch.close()
