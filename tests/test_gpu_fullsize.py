"""Full-size checks of the benchmarked workloads (1b, 1b-long, 8b) in the
launch configuration bench.py times (B x S of the workload, random-init
weights of the architecture, Zipf token ids), against outputs the oracle can
compute one by one plus properties that hold at any size:

- causal prefixes: h_out of the first P positions of every sequence depends
  only on those positions, so the oracle runs them through all L layers at
  full width; the per-row loss and dL/dh_out of those rows follow from them
  and the full-vocabulary head (Eq. (2)-(5));
- the optimizer step (Eq. (6), AdamW) is elementwise: sampled parameters are
  checked against the oracle's step from the device's own gradient;
- |Omega| is an exact integer count; gradients, loss and outputs are finite;
  the bf16 shadow is the round-to-nearest-even of the new master, bit for bit.
"""
import numpy as np
import pytest

import oracle
import workload
from oracle import blocks, ops
from oracle.chunk import bf16_round
from oracle.objective import local_objective_ref
from oracle.optim import adamw_step_ref
from tests.gpu_cases import rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

P = 16  # prefix positions per sequence


def _bench_chunk(shp):
    """The chunk, inputs and labels as bench.py builds them."""
    from paper_2608_07974_amd import zl
    from paper_2608_07974_amd.chunk import TorchChunk, config_from_shape, current_stream
    dev = torch.device("cuda:0")
    torch.manual_seed(0)
    ch = TorchChunk(config_from_shape(shp, alpha=0.5), device=dev)
    ch.master.normal_(0.0, 0.02)
    for t in ch.layout:
        v = ch.master[t["offset"]: t["offset"] + t["numel"]]
        if t["name"].startswith("ln") and t["name"].endswith("_w"):
            v.fill_(1.0)
        elif len(t["shape"]) == 1:
            v.zero_()
    ch.head_w.normal_(0.0, 0.02)
    zl.zl_refresh_shadow(ch.handle, current_stream())
    B, S = shp.batch, shp.seq
    tokens = workload.zipf_tokens(B, S, shp.vocab, seed=1)
    labels = torch.tensor(workload.labels_from_tokens(tokens), device=dev)
    table = torch.empty(shp.vocab, shp.d_model, dtype=ch.dtype, device=dev).normal_(0.0, 0.02)
    h_in = table[torch.tensor(tokens, device=dev, dtype=torch.long)].contiguous()
    del table
    return ch, h_in, labels


def _layer_params(ch, master, layer):
    """Layer tensors of `master` as the device consumes them (bf16
    matrices), fp64."""
    out = {}
    for key in ch.by_key:
        if key.startswith(f"L{layer}."):
            a = ch.view(master, key).detach().cpu().double().numpy()
            out[key] = bf16_round(a) if a.ndim == 2 else a
    return out


@pytest.mark.parametrize("name", ["1b", "1b-long", "8b"])
def test_full_size_prefixes_and_step(name):
    shp = workload.get_config(name)
    B, S, d = shp.batch, shp.seq, shp.d_model
    ch, h_in, labels = _bench_chunk(shp)
    theta0 = ch.master.clone()
    h_out = ch.forward(h_in)
    ch.objective(labels)
    torch.cuda.synchronize()
    loss = float(ch.loss.item())
    row_loss = ch.inspect("row_loss").reshape(B, S)
    dh_dev = ch.inspect("dh_out").reshape(B, S, d)[:, :P]
    n_dev = float(ch.inspect("n_omega").reshape(-1)[0])
    ch.backward(1.0, 0)
    ch.step()
    torch.cuda.synchronize()

    lab = labels.cpu().numpy()
    n_total = int(np.sum((lab >= 0) & (lab < shp.vocab)))
    assert n_dev == n_total
    assert np.isfinite(loss)
    assert bool(torch.isfinite(ch.grad).all())
    assert bool(torch.isfinite(h_out).all())

    # causal prefixes through all layers at full width
    cfg = oracle.OracleConfig.from_shape(shp, alpha=0.5)
    x = h_in[:, :P].float().cpu().double().numpy().reshape(B * P, d)
    pos = np.tile(np.arange(P), (B, 1))
    ang = ops.rope_angles(pos, shp.head_dim, shp.rope_theta)
    lens = np.full(B, P)
    for layer in range(shp.n_layers):
        x, _ = blocks.llama_layer_fwd(x, _layer_params(ch, theta0, layer), f"L{layer}.", cfg, ang,
                                      lens, B, P)
    got = h_out[:, :P].float().cpu().double().numpy().reshape(B * P, d)
    assert rel_err(got, x) < 2e-2

    # per-row objective and dL/dh_out of the prefix rows (full vocabulary)
    W = ch.head_w.float().cpu().double().numpy()
    hn = ch.head_norm_w.double().cpu().numpy()
    lab_p = lab[:, :P].reshape(-1)
    _, dh_ref, info = local_objective_ref(x, h_in[:, :P].float().cpu().double().numpy().reshape(B * P, d),
                                          lab_p, W, shp.arch, hn, None, shp.norm_eps, 0.5)
    rows_ref = 0.5 * info["ce"] + 0.5 * info["kl"]
    assert rel_err(row_loss[:, :P].reshape(-1), rows_ref) < 2e-2
    n_p = info["n_omega"]
    assert rel_err(dh_dev.reshape(B * P, d) * n_total, dh_ref * n_p) < 4e-2
    del W

    # AdamW, first step, on a sample of parameters, from the device gradient
    rng = np.random.default_rng(7)
    idx = torch.tensor(rng.choice(ch.n_params, size=200_000, replace=False), device=h_in.device)
    th0 = theta0[idx].double().cpu().numpy()
    g = ch.grad[idx].double().cpu().numpy()
    th1 = ch.master[idx].double().cpu().numpy()
    m1 = ch.adam_m[idx].double().cpu().numpy()
    v1 = ch.adam_v[idx].double().cpu().numpy()
    sh = ch.shadow[idx].float().double().cpu().numpy()
    th_ref, m_ref, v_ref = adamw_step_ref(th0, g, 0.0, 0.0, 1, cfg.lr, cfg.beta1, cfg.beta2,
                                          cfg.eps, cfg.weight_decay)
    # (1 - beta) is formed in fp32 on the device: 0.1 to 2.4e-7, 0.001 to 1.3e-5
    assert np.all(np.abs(m1 - m_ref) <= 1e-6 * np.abs(m_ref) + 1e-30)
    assert np.all(np.abs(v1 - v_ref) <= 1e-4 * np.abs(v_ref) + 1e-30)
    ulp = np.spacing(np.abs(th_ref).astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(th1 - th_ref) <= 4 * ulp + 1e-4 * cfg.lr)
    assert np.array_equal(sh, bf16_round(th1))
    ch.close()
    del ch, theta0, h_in, h_out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["8b", "1b-long"])
def test_attention_full_size_one_head_group(name):
    """The attention kernels at the workload's full B x S and head counts
    (the launch the update times), bf16: forward output, log-sum-exp, dQ, dK
    and dV of one (sequence, kv-head group) against the oracle's attention
    over that whole sequence; every output finite."""
    from paper_2608_07974_amd import zl
    shp = workload.get_config(name)
    B, S, Hq, Hkv, hd = shp.batch, shp.seq, shp.n_heads, shp.n_kv_heads, shp.head_dim
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev).manual_seed(11)
    ld = (Hq + 2 * Hkv) * hd
    QKV = torch.randn(B * S, ld, device=dev, generator=gen).to(torch.bfloat16)
    DO = torch.randn(B * S, Hq * hd, device=dev, generator=gen).to(torch.bfloat16)
    O = torch.zeros(B * S, Hq * hd, device=dev, dtype=torch.bfloat16)
    LSE = torch.zeros(B, Hq, S, dtype=torch.float32, device=dev)
    DQKV = torch.zeros_like(QKV)
    DEL = torch.zeros(B, Hq, S, dtype=torch.float32, device=dev)
    SL = torch.full((B,), S, dtype=torch.int32, device=dev)
    base, esz = QKV.data_ptr(), QKV.element_size()
    stream = torch.cuda.current_stream().cuda_stream
    args = (B, S, Hq, Hkv, hd, base, base + Hq * hd * esz, base + (Hq + Hkv) * hd * esz, ld,
            SL.data_ptr(), O.data_ptr(), LSE.data_ptr())
    zl.zl_kernel_attention(*args, 0, 0, 0, 0, 0, zl.ZL_BF16, 0, stream)
    dbase = DQKV.data_ptr()
    zl.zl_kernel_attention(*args, DO.data_ptr(), dbase, dbase + Hq * hd * esz,
                           dbase + (Hq + Hkv) * hd * esz, DEL.data_ptr(), zl.ZL_BF16, 1, stream)
    torch.cuda.synchronize()
    for t in (O, LSE, DQKV):
        assert bool(torch.isfinite(t).all())

    b, g = B - 1, Hkv - 1
    grp = Hq // Hkv
    heads = slice(g * grp, (g + 1) * grp)
    rows = slice(b * S, (b + 1) * S)
    r = QKV[rows].double().cpu().numpy()
    q = r[:, : Hq * hd].reshape(1, S, Hq, hd)[:, :, heads]
    k = r[:, Hq * hd: (Hq + Hkv) * hd].reshape(1, S, Hkv, hd)[:, :, g:g + 1]
    v = r[:, (Hq + Hkv) * hd:].reshape(1, S, Hkv, hd)[:, :, g:g + 1]
    do = DO[rows].double().cpu().numpy().reshape(1, S, Hq, hd)[:, :, heads]
    o_ref, cache = ops.attention_fwd(q, k, v, np.array([S], np.int32))
    dq_ref, dk_ref, dv_ref = ops.attention_bwd(do, cache)
    del cache
    o = O[rows].double().cpu().numpy().reshape(1, S, Hq, hd)[:, :, heads]
    d = DQKV[rows].double().cpu().numpy()
    dq = d[:, : Hq * hd].reshape(1, S, Hq, hd)[:, :, heads]
    dk = d[:, Hq * hd: (Hq + Hkv) * hd].reshape(1, S, Hkv, hd)[:, :, g:g + 1]
    dv = d[:, (Hq + Hkv) * hd:].reshape(1, S, Hkv, hd)[:, :, g:g + 1]
    tol = 1.2e-2
    assert rel_err(o, o_ref) < tol
    assert rel_err(dq, dq_ref) < tol
    assert rel_err(dk, dk_ref) < tol
    assert rel_err(dv, dv_ref) < tol
    # log-sum-exp of the group's rows, from the oracle's own scores
    scale = 1.0 / np.sqrt(hd)
    lse = LSE[b, heads].double().cpu().numpy()
    causal = np.tril(np.ones((S, S), bool))
    for j in range(grp):
        s = (q[0, :, j] @ k[0, :, 0].T) * scale
        s = np.where(causal, s, -np.inf)
        mx = s.max(axis=1, keepdims=True)
        ref = (np.log(np.exp(s - mx).sum(axis=1, keepdims=True)) + mx)[:, 0]
        assert np.max(np.abs(lse[j] - ref) / np.maximum(1.0, np.abs(ref))) < 1e-4


def _rows_per_tile(T, rng, tile=256):
    """One row from every tile of `tile` rows (the GEMMs' row tiles)."""
    return np.array([t + int(rng.integers(min(tile, T - t))) for t in range(0, T, tile)])


def _dev_rows(ch, name, rows, layer=0):
    t = ch.inspect_device(name, layer)
    return t[torch.tensor(rows, device=t.device, dtype=torch.long)].double().cpu().numpy()


def _dev_cols(ch, name, cols, layer=0):
    t = ch.inspect_device(name, layer)
    return t[:, torch.tensor(cols, device=t.device, dtype=torch.long)].double().cpu().numpy()


def _near_bf16(got, ref, what):
    """got is ref stored in bf16 (up to fp32 accumulation order): every
    element within 2^-8 of itself plus 1e-3 of its row's RMS."""
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    bad = np.abs(got - ref) > 2.0 ** -8 * np.abs(ref) + 1e-3 * rms
    assert not bad.any(), (what, np.argwhere(bad)[:5])


def _near_f32(got, ref, scale, what, rel=1e-4):
    """got is ref accumulated in fp32: within rel of the size of its terms."""
    bad = np.abs(got - ref) > rel * scale + 1e-30
    assert not bad.any(), (what, np.argwhere(bad)[:5], np.max(np.abs(got - ref) / (scale + 1e-30)))


def _rms_norm(x, w, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


@pytest.mark.parametrize("name", ["8b", "1b-long"])
def test_full_size_every_row_tile_and_weight_gradients(name):
    """At the benchmarked B x S, element-wise, on layer 0 of the update:
    one row from every 256-row tile of each forward GEMM's output (norm 1,
    QKV with RoPE, output projection + residual, norm 2, gate/up, SwiGLU,
    down + residual) and of the data gradients (down with the SwiGLU
    backward, output projection, QKV), each from the device's own bf16
    operands in fp64; sampled entries of the four weight gradients
    dW = dy^T x over all B*S tokens (the two paired launches); sampled
    entries of the head's data gradient dZ W_lm over the full vocabulary
    (split over K at the 1B width); and the head's per-row loss and
    dL/dh_out of one row from every tile against the oracle."""
    shp = workload.get_config(name)
    B, S, d, V = shp.batch, shp.seq, shp.d_model, shp.vocab
    T = B * S
    ff, hd = shp.d_ff, shp.head_dim
    dq, dkv = shp.n_heads * hd, shp.n_kv_heads * hd
    nqkv = dq + 2 * dkv
    rng = np.random.default_rng(3)
    ch, h_in, labels = _bench_chunk(shp)
    ch.forward(h_in)
    ch.objective(labels)
    torch.cuda.synchronize()
    dz_last = ch.inspect_device("dz")
    R = dz_last.shape[0]
    row_loss = ch.inspect("row_loss").reshape(-1)
    dh_out = ch.inspect_device("dh_out")
    rows = _rows_per_tile(T, rng)
    dh_rows = dh_out[torch.tensor(rows, device=dh_out.device)].double().cpu().numpy()
    # head data gradient of the last row block: entries over the full vocabulary
    W_dev = ch.head_w
    ii = np.concatenate([[0, R - 1], rng.integers(R, size=14)])
    jj = np.concatenate([[0, d - 1], rng.integers(d, size=14)])
    dnf = ch.inspect("dnf")
    dzr = dz_last[torch.tensor(ii, device=dz_last.device)][:, :V].double().cpu().numpy()
    Wc = W_dev[:, torch.tensor(jj, device=W_dev.device)].double().cpu().numpy()
    terms = dzr[:, :, None] * Wc[None, :, :]  # [i, v, j]
    ref = terms.sum(axis=1)
    _near_f32(dnf[ii][:, jj], ref, np.abs(terms).sum(axis=1), "head dgrad", rel=2e-4)
    del terms, dzr, Wc
    ch.backward(1.0, 0)
    torch.cuda.synchronize()

    P0 = _layer_params(ch, ch.master, 0)
    pos = rows % S
    eps = shp.norm_eps
    # ---- forward, one row per 256-row tile
    x0 = _dev_rows(ch, "x", rows, 0)
    n1 = _dev_rows(ch, "n1", rows)
    _near_bf16(n1, _rms_norm(x0, P0["L0.ln1_w"], eps), "n1")
    wqkv = np.concatenate([P0["L0.wq"], P0["L0.wk"], P0["L0.wv"]])
    y = n1 @ wqkv.T
    ang = ops.rope_angles(pos[None, :], hd, shp.rope_theta)  # [1, rows, hd/2]
    nh = shp.n_heads + shp.n_kv_heads
    qk = ops.rope_fwd(y[:, : nh * hd].reshape(1, len(rows), nh, hd), ang).reshape(len(rows), -1)
    _near_bf16(_dev_rows(ch, "qkv", rows), np.concatenate([qk, y[:, nh * hd:]], axis=1), "qkv")
    o = _dev_rows(ch, "o", rows)
    x2 = _dev_rows(ch, "x2", rows)
    _near_f32(x2, x0 + o @ P0["L0.wo"].T, np.abs(x0) + np.abs(o) @ np.abs(P0["L0.wo"]).T,
              "output projection + residual")
    n2 = _dev_rows(ch, "n2", rows)
    _near_bf16(n2, _rms_norm(x2, P0["L0.ln2_w"], eps), "n2")
    wgu = np.concatenate([P0["L0.wg"], P0["L0.wu"]])
    up = _dev_rows(ch, "up", rows)
    _near_bf16(up, n2 @ wgu.T, "gate/up")
    act = _dev_rows(ch, "act", rows)
    g, u = up[:, :ff], up[:, ff:]
    _near_bf16(act, ops.swiglu_fwd(g, u), "swiglu")
    x1 = _dev_rows(ch, "x", rows, 1)
    t = act @ P0["L0.wd"].T
    scale = np.abs(x2) + np.abs(act) @ np.abs(P0["L0.wd"]).T
    _near_f32(x1, x2 + t, scale, "down + residual")
    # ---- backward data gradients of layer 0, one row per tile
    dxa = _dev_rows(ch, "dxa", rows)
    dup = _dev_rows(ch, "dup", rows)
    dg, du = ops.swiglu_bwd(dxa @ P0["L0.wd"], g, u)
    _near_bf16(dup, np.concatenate([dg, du], axis=1), "down dgrad + SwiGLU backward")
    dxb = _dev_rows(ch, "dxb", rows)
    _near_bf16(_dev_rows(ch, "do", rows), dxb @ P0["L0.wo"], "output projection dgrad")
    dqkv = _dev_rows(ch, "dqkv", rows)
    t = dqkv @ wqkv
    _near_f32(_dev_rows(ch, "dn", rows), t, np.abs(dqkv) @ np.abs(wqkv), "QKV dgrad")
    # ---- weight gradients dW[o, i] = sum_t dy[t, o] x[t, i] over all T tokens
    for wname, dyn, xn, nout, nin in (("wd", "dxa", "act", d, ff), ("wg", "dup", "n2", 2 * ff, d),
                                      ("wo", "dxb", "o", d, dq), ("wq", "dqkv", "n1", nqkv, d)):
        oo = np.concatenate([[0, nout - 1], rng.integers(nout, size=10)])
        kk = np.concatenate([[0, nin - 1], rng.integers(nin, size=10)])
        dy = _dev_cols(ch, dyn, oo)
        xx = _dev_cols(ch, xn, kk)
        terms = dy[:, :, None] * xx[:, None, :]  # [T, o, i]
        tv = ch.by_key[f"L0.{wname}"]
        G = ch.grad[tv["offset"]: tv["offset"] + nout * nin].view(nout, nin)
        got = G[torch.tensor(oo, device=G.device)][:, torch.tensor(kk, device=G.device)]
        _near_f32(got.double().cpu().numpy(), terms.sum(0), np.abs(terms).sum(0),
                  f"dW {wname}", rel=2e-4)
        del terms
    # ---- the head: loss row and dL/dh_out of one row per tile (oracle)
    lab = labels.cpu().numpy().reshape(-1)
    hL = _dev_rows(ch, "x", rows, shp.n_layers)
    hin = h_in.reshape(T, d)[torch.tensor(rows, device=h_in.device)].double().cpu().numpy()
    Wh = W_dev.double().cpu().numpy()
    hn = ch.head_norm_w.double().cpu().numpy()
    _, dh_ref, info = local_objective_ref(hL, hin, lab[rows], Wh, shp.arch, hn, None, eps, 0.5)
    del Wh
    rows_ref = 0.5 * info["ce"] + 0.5 * info["kl"]
    assert np.max(np.abs(row_loss[rows] - rows_ref) / np.maximum(np.abs(rows_ref), 1.0)) < 1e-3
    n_total = int(np.sum((lab >= 0) & (lab < V)))
    a, b = dh_rows * n_total, dh_ref * info["n_omega"]
    rn = np.linalg.norm(a - b, axis=1) / np.maximum(np.linalg.norm(b, axis=1), 1e-30)
    assert np.max(rn) < 2e-2, (rows[np.argmax(rn)], np.max(rn))
    ch.close()
    del ch, h_in
    torch.cuda.empty_cache()
