"""The single-GPU runtime through the C ABI: the stage pipeline with early
forwarding (zl_pipeline_*) and per-chunk checkpoint / resume.

Pipeline parity: K chunks, update windows of m micro-batches, against the
oracle run window by window (within a window a chunk's weights are fixed,
so stage k+1's inputs are stage k's pre-update outputs of the window's
micro-batches).  Gates as in test_gpu_parity: fp32 1e-4; bf16 2e-2 on
losses and parameters.  The pipeline must also match the same chunks run
one after another on one stream bit for bit (same kernels, same order per
chunk), which checks the event ordering independently of tolerances."""
import numpy as np
import pytest

import oracle
import workload
from oracle.chunk import init_opt_state
from tests.gpu_cases import make_inputs, oracle_cfg, rel_err

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

from paper_2608_07974_amd import zl  # noqa: E402
from paper_2608_07974_amd.chunk import TorchChunk, config_from_shape, current_stream  # noqa: E402
from paper_2608_07974_amd.pipeline import Pipeline  # noqa: E402

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _stage_inputs(shp, K, n_mb):
    params = [make_inputs(shp, seed=10 + k)[0] for k in range(K)]
    batches = [workload.make_batch(shp, seed_tokens=1 + i, stress=True, perturb_head=True)
               for i in range(n_mb)]
    return params, batches


def _oracle_pipeline(shp, params, batches, window, **kw):
    cfg = oracle_cfg(shp, **kw)
    K = len(params)
    P = [{k: np.asarray(v, np.float64) for k, v in p.items()} for p in params]
    st = [init_opt_state() for _ in range(K)]
    head = batches[0]
    losses = np.zeros((len(batches), K))
    outs = []
    for w0 in range(0, len(batches), window):
        win = batches[w0:w0 + window]
        h = [b["h_in"] for b in win]
        for k in range(K):
            mbs = [dict(h_in=h[i], labels=b["labels"], seq_lens=b["seq_lens"], pos_ids=b["pos_ids"])
                   for i, b in enumerate(win)]
            r = oracle.chunk_update_ref(cfg, P[k], st[k], mbs, head["head_w"], head["head_norm_w"],
                                        head["head_norm_b"])
            losses[w0:w0 + len(win), k] = r["losses"]
            h = [run["h_out"] for run in r["runs"]]
            P[k], st[k] = r["params"], r["state"]
        outs.extend(h)
    return P, losses, outs


def _device_pipeline(shp, params, batches, window, depth, **kw):
    cfg = config_from_shape(shp, **kw)
    pipe = Pipeline([cfg] * len(params), window=window, depth=depth)
    head = batches[0]
    pipe.chunks[0].load_head(head["head_w"], head["head_norm_w"], head["head_norm_b"])
    for ch, p in zip(pipe.chunks, params):
        ch.load_params(p)
    tdt = pipe.dtype
    dev = torch.device("cuda")
    ins = [dict(h0=torch.tensor(b["h_in"], device=dev).to(tdt),
                labels=torch.tensor(b["labels"], device=dev),
                pos_ids=torch.tensor(b["pos_ids"], device=dev),
                seq_lens=torch.tensor(b["seq_lens"], device=dev)) for b in batches]
    losses, outs = [], []
    for x in ins:
        mb, l = pipe.submit(x["h0"], x["labels"], x["pos_ids"], x["seq_lens"])
        losses.append(l)
        outs.append(pipe.output(mb, tuple(x["h0"].shape)))
    pipe.sync()
    torch.cuda.synchronize()
    res = dict(params=[c.tensors(c.master) for c in pipe.chunks],
               losses=np.stack([l.cpu().double().numpy() for l in losses]),
               outs=[o.double().cpu().numpy() for o in outs], progress=pipe.progress())
    pipe.close()
    return res


def _sequential(shp, params, batches, window, **kw):
    """The same chunks, one after another on the current stream."""
    head = batches[0]
    chunks = []
    for p in params:
        ch = TorchChunk(config_from_shape(shp, **kw))
        ch.load_head(head["head_w"], head["head_norm_w"], head["head_norm_b"])
        ch.load_params(p)
        chunks.append(ch)
    dev = torch.device("cuda")
    tdt = chunks[0].dtype
    losses = []
    for i, b in enumerate(batches):
        h = torch.tensor(b["h_in"], device=dev).to(tdt)
        lab = torch.tensor(b["labels"], device=dev)
        pos = torch.tensor(b["pos_ids"], device=dev)
        sl = torch.tensor(b["seq_lens"], device=dev)
        row = []
        for ch in chunks:
            h = ch.forward(h, sl, pos)
            row.append(ch.objective(lab).clone())
            ch.backward(1.0 / window, 0 if i % window == 0 else 1)
            if i % window == window - 1:
                ch.step()
        losses.append(torch.cat(row))
    torch.cuda.synchronize()
    res = dict(params=[c.tensors(c.master) for c in chunks],
               losses=np.stack([l.cpu().double().numpy() for l in losses]))
    for c in chunks:
        c.close()
    return res


@pytest.mark.parametrize("name,K,window,depth", [("tiny", 2, 2, 2), ("tiny", 3, 1, 1)])
def test_pipeline_matches_oracle_fp32(name, K, window, depth):
    shp = workload.get_config(name)
    params, batches = _stage_inputs(shp, K, 4)
    dev = _device_pipeline(shp, params, batches, window, depth)
    P, losses, outs = _oracle_pipeline(shp, params, batches, window)
    tol = TOL[shp.dtype]
    assert dev["progress"] == (4, 4 // window)
    assert rel_err(dev["losses"], losses) < tol
    for i in range(4):
        assert rel_err(dev["outs"][i], outs[i]) < tol, i
    for k in range(K):
        worst = max(rel_err(dev["params"][k][n], P[k][n]) for n in P[k])
        assert worst < tol, (k, worst)


def test_pipeline_matches_oracle_bf16():
    shp = workload.get_config("tiny").with_(dtype="bf16")
    params, batches = _stage_inputs(shp, 2, 4)
    dev = _device_pipeline(shp, params, batches, window=2, depth=2)
    P, losses, _ = _oracle_pipeline(shp, params, batches, window=2)
    assert rel_err(dev["losses"], losses) < TOL["bf16"]
    for k in range(2):
        worst = max(rel_err(dev["params"][k][n], P[k][n]) for n in P[k])
        assert worst < TOL["bf16"], (k, worst)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pipeline_bit_identical_to_sequential(dtype):
    shp = workload.get_config("tiny").with_(dtype=dtype)
    params, batches = _stage_inputs(shp, 3, 6)
    a = _device_pipeline(shp, params, batches, window=2, depth=2)
    b = _sequential(shp, params, batches, window=2)
    np.testing.assert_array_equal(a["losses"], b["losses"])
    for k in range(3):
        for n in b["params"][k]:
            np.testing.assert_array_equal(a["params"][k][n], b["params"][k][n], err_msg=f"{k} {n}")


def test_read_output_of_reused_entry_is_rejected():
    shp = workload.get_config("tiny")
    params, batches = _stage_inputs(shp, 2, 3)
    pipe = Pipeline([config_from_shape(shp)] * 2, window=1, depth=1)
    for ch, p in zip(pipe.chunks, params):
        ch.load_params(p)
    dev = torch.device("cuda")
    for b in batches:
        pipe.submit(torch.tensor(b["h_in"], device=dev), torch.tensor(b["labels"], device=dev))
    with pytest.raises(zl.ZlError) as e:
        pipe.output(0, batches[0]["h_in"].shape)
    assert e.value.status == zl.ZL_ERR_INVALID_ARG
    pipe.output(2, batches[2]["h_in"].shape)
    pipe.sync()
    pipe.close()


def _run_updates(ch, batches, dev):
    for b in batches:
        ch.update(torch.tensor(b["h_in"], device=dev).to(ch.dtype),
                  torch.tensor(b["labels"], device=dev))


@pytest.mark.parametrize("dtype,optimizer", [("f32", "adamw"), ("bf16", "adamw"), ("f32", "sgd")])
def test_checkpoint_resume_is_bit_identical(tmp_path, dtype, optimizer):
    shp = workload.get_config("tiny").with_(dtype=dtype)
    params, batches = _stage_inputs(shp, 1, 4)
    head = batches[0]
    dev = torch.device("cuda")
    cfg = config_from_shape(shp, optimizer=optimizer, lr=1e-3)
    a = TorchChunk(cfg)
    a.load_head(head["head_w"], head["head_norm_w"], head["head_norm_b"])
    a.load_params(params[0])
    _run_updates(a, batches[:2], dev)
    path = str(tmp_path / "stage.ckpt")
    a.save(path, microbatches=2, windows=2)
    info = zl.zl_checkpoint_read_info(path)
    assert (info["step"], info["microbatches"], info["windows"]) == (2, 2, 2)
    assert info["n_params"] == a.n_params
    _run_updates(a, batches[2:], dev)
    torch.cuda.synchronize()
    want = a.tensors(a.master)

    b = TorchChunk(cfg)
    b.load_head(head["head_w"], head["head_norm_w"], head["head_norm_b"])
    assert b.restore(path) == (2, 2)
    assert zl.zl_get_step(b.handle) == 2
    _run_updates(b, batches[2:], dev)
    torch.cuda.synchronize()
    got = b.tensors(b.master)
    for n in want:
        np.testing.assert_array_equal(got[n], want[n], err_msg=n)
    a.close()
    b.close()


def test_checkpoint_mismatch_leaves_chunk_unchanged(tmp_path):
    shp = workload.get_config("tiny")
    params, batches = _stage_inputs(shp, 1, 1)
    a = TorchChunk(config_from_shape(shp))
    a.load_params(params[0])
    path = str(tmp_path / "a.ckpt")
    a.save(path)
    other = TorchChunk(config_from_shape(shp.with_(n_layers=1)))
    before = other.master.clone()
    with pytest.raises(zl.ZlError) as e:
        other.restore(path)
    assert e.value.status == zl.ZL_ERR_INVALID_ARG and "n_layers" in str(e.value)
    torch.cuda.synchronize()
    assert torch.equal(other.master, before)
    # a corrupted payload is caught by the checksum before anything is written
    raw = bytearray(open(path, "rb").read())
    raw[-4] ^= 0xFF
    open(path, "wb").write(bytes(raw))
    b = TorchChunk(config_from_shape(shp))
    before = b.master.clone()
    with pytest.raises(zl.ZlError) as e:
        b.restore(path)
    assert "checksum" in str(e.value)
    assert torch.equal(b.master, before)
    for c in (a, other, b):
        c.close()


def test_pipeline_checkpoint_only_at_window_boundary(tmp_path):
    shp = workload.get_config("tiny")
    params, batches = _stage_inputs(shp, 2, 3)
    pipe = Pipeline([config_from_shape(shp)] * 2, window=2, depth=2)
    for ch, p in zip(pipe.chunks, params):
        ch.load_params(p)
    dev = torch.device("cuda")
    for b in batches[:2]:
        pipe.submit(torch.tensor(b["h_in"], device=dev), torch.tensor(b["labels"], device=dev))
    pipe.checkpoint(1, str(tmp_path / "s1.ckpt"))
    info = zl.zl_checkpoint_read_info(str(tmp_path / "s1.ckpt"))
    assert (info["microbatches"], info["windows"], info["step"]) == (2, 1, 1)
    pipe.submit(torch.tensor(batches[2]["h_in"], device=dev),
                torch.tensor(batches[2]["labels"], device=dev))
    with pytest.raises(zl.ZlError) as e:
        pipe.checkpoint(0, str(tmp_path / "s0.ckpt"))
    assert e.value.status == zl.ZL_ERR_STATE
    pipe.sync()
    pipe.close()
