"""Single-kernel parity on the GPU through the C ABI (zl_inspect.h):
the GEMM in its operand layouts (with the LoRA segment and split K) and causal GQA attention, against
fp64 references computed on the CPU from the same (bf16-rounded) inputs."""
import numpy as np
import pytest

import oracle
from oracle import ops
from tests.gpu_cases import rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _zl():
    from paper_2608_07974_amd import zl
    return zl


def _dev():
    return torch.device("cuda")


def _stream():
    return torch.cuda.current_stream().cuda_stream


# bf16 operands with contiguous M need M % 8 == 0 (16-byte rows; the library
# rejects the rest, tested on the CPU); the fp32 SIMT path is sized for small
# problems, so it is not run at 4096 x 3848.
_LAYOUT_CASES = [(dt, lay, M, N, K)
                 for dt in ("bf16", "f32") for lay in ("nt", "nn", "tn")
                 for M, N, K in ((8, 8, 8), (1, 8, 8), (304, 520, 200), (129, 136, 1000),
                                 (4096, 3848, 264))
                 if not (dt == "bf16" and lay == "tn" and M % 8)
                 and not (dt == "f32" and M * N * K > 1e9)]


@pytest.mark.parametrize("dtype,layout,M,N,K", _LAYOUT_CASES)
def test_gemm_layouts(dtype, layout, M, N, K):
    """C = A B^T with A(m,k), B(n,k) stored K-major or MN-major (fwd: nt,
    dgrad: nn, wgrad: tn), ragged in every dimension."""
    zl = _zl()
    rng = np.random.default_rng(M + N + K)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    a_k = layout in ("nt", "nn")
    b_k = layout == "nt"
    A = rng.standard_normal((M, K) if a_k else (K, M)).astype(np.float32)
    B = rng.standard_normal((N, K) if b_k else (K, N)).astype(np.float32)
    At = torch.tensor(A, device=_dev()).to(tdt)
    Bt = torch.tensor(B, device=_dev()).to(tdt)
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device=_dev())
    torch.cuda.synchronize()
    zl.zl_kernel_gemm(M, N, K, At.data_ptr(), At.shape[1], a_k, Bt.data_ptr(), Bt.shape[1], b_k,
                      C.data_ptr(), N, zl.ZL_BF16 if dtype == "bf16" else zl.ZL_F32, _stream())
    torch.cuda.synchronize()
    a64 = At.double().cpu().numpy()
    b64 = Bt.double().cpu().numpy()
    ref = (a64 if a_k else a64.T) @ (b64 if b_k else b64.T).T
    got = C.cpu().double().numpy()
    assert np.all(np.isfinite(got))
    bound = 1e-5 * np.sqrt(K) * (np.abs(a64).max() * np.abs(b64).max()) + 1e-6
    assert np.max(np.abs(got - ref)) < bound * 8
    assert rel_err(got, ref) < 2e-6


def _gemm_operands(rng, layout, M, N, K, tdt):
    a_k = layout in ("nt", "nn")
    b_k = layout == "nt"
    A = rng.standard_normal((M, K) if a_k else (K, M)).astype(np.float32)
    B = rng.standard_normal((N, K) if b_k else (K, N)).astype(np.float32)
    return (torch.tensor(A, device=_dev()).to(tdt), torch.tensor(B, device=_dev()).to(tdt), a_k, b_k)


def _gemm_ref(At, Bt, a_k, b_k):
    a64 = At.double().cpu().numpy()
    b64 = Bt.double().cpu().numpy()
    return (a64 if a_k else a64.T) @ (b64 if b_k else b64.T).T


@pytest.mark.parametrize("dtype,layout,M,N,K,K2", [
    (dt, lay, M, N, K, K2) for dt in ("bf16", "f32") for lay in ("nt", "nn", "tn")
    for M, N, K, K2 in ((304, 520, 200, 8), (4096, 3848, 264, 48), (512, 768, 4096, 16),
                        (136, 64, 8, 200))
    if not (dt == "f32" and M * N * (K + K2) > 1e9)])
def test_gemm_second_segment(dtype, layout, M, N, K, K2):
    """C = A B^T + A2 B2^T with the second pair in the layouts of the first
    (the low-rank term of a LoRA projection), ragged in every dimension."""
    zl = _zl()
    rng = np.random.default_rng(M + N + K + K2)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    At, Bt, a_k, b_k = _gemm_operands(rng, layout, M, N, K, tdt)
    A2, B2, _, _ = _gemm_operands(rng, layout, M, N, K2, tdt)
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device=_dev())
    torch.cuda.synchronize()
    zl.zl_kernel_gemm(M, N, K, At.data_ptr(), At.shape[1], a_k, Bt.data_ptr(), Bt.shape[1], b_k,
                      C.data_ptr(), N, zl.ZL_BF16 if dtype == "bf16" else zl.ZL_F32, _stream(),
                      K2=K2, A2=A2.data_ptr(), lda2=A2.shape[1], B2=B2.data_ptr(), ldb2=B2.shape[1])
    torch.cuda.synchronize()
    ref = _gemm_ref(At, Bt, a_k, b_k) + _gemm_ref(A2, B2, a_k, b_k)
    got = C.cpu().double().numpy()
    assert np.all(np.isfinite(got))
    assert rel_err(got, ref) < 2e-6


@pytest.mark.parametrize("a_k,b_k", [(True, True), (True, False), (False, False), (False, True)])
@pytest.mark.parametrize("M,N,K,K2", [(16, 4104, 16384, 0), (4096, 16, 16384, 16), (200, 136, 3000, 24),
                                      (48, 1000, 1024, 0)])
def test_gemm_split_k(a_k, b_k, M, N, K, K2):
    """Outputs of too few tiles to fill the GPU (the LoRA factor GEMMs) split
    K into fp32 partials in the caller's workspace: same result as one pass
    within fp32 summation error, identical on a repeat (fixed summation
    order), and still correct when the workspace only holds two partials."""
    zl = _zl()
    rng = np.random.default_rng(M + N + K + K2 + 2 * a_k + b_k)

    def op(rows, k, kmaj):
        x = rng.standard_normal((rows, k) if kmaj else (k, rows)).astype(np.float32)
        return torch.tensor(x, device=_dev()).to(torch.bfloat16)
    At, Bt = op(M, K, a_k), op(N, K, b_k)
    A2, B2 = (op(M, K2, a_k), op(N, K2, b_k)) if K2 else (None, None)
    seg = dict(K2=K2, A2=A2.data_ptr(), lda2=A2.shape[1], B2=B2.data_ptr(), ldb2=B2.shape[1]) if K2 else {}

    def run(ws_elems):
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device=_dev())
        ws = torch.full((max(ws_elems, 1),), float("nan"), dtype=torch.float32, device=_dev())
        torch.cuda.synchronize()
        zl.zl_kernel_gemm(M, N, K, At.data_ptr(), At.shape[1], a_k, Bt.data_ptr(), Bt.shape[1], b_k,
                          C.data_ptr(), N, zl.ZL_BF16, _stream(), workspace=ws.data_ptr() if ws_elems else None,
                          workspace_elems=ws_elems, **seg)
        torch.cuda.synchronize()
        return C.cpu().double().numpy()
    ref = _gemm_ref(At, Bt, a_k, b_k) + (_gemm_ref(A2, B2, a_k, b_k) if K2 else 0.0)
    one = run(0)
    split = run(64 * M * N)
    again = run(64 * M * N)
    two = run(2 * M * N)
    for got in (one, split, two):
        assert np.all(np.isfinite(got))
        assert rel_err(got, ref) < 2e-6
    assert np.array_equal(split, again)


@pytest.mark.parametrize("a_k,b_k", [(True, False), (True, True)])
def test_gemm_long_k_large_tiles_split(a_k, b_k):
    """A long reduction over few large tiles (the head's data gradient, K = V
    with rows x d small: here 2048 x 1024 x 65536, 32 tiles of 256 x 256)
    runs as large tiles split eight ways over K: sampled rows against fp64,
    the whole output against the unsplit launch, identical on a repeat."""
    zl = _zl()
    M, N, K = 2048, 1024, 65536
    gen = torch.Generator(device=_dev()).manual_seed(5)
    At = torch.randn((M, K) if a_k else (K, M), device=_dev(), generator=gen).to(torch.bfloat16)
    Bt = torch.randn((N, K) if b_k else (K, N), device=_dev(), generator=gen).to(torch.bfloat16)

    def run(ws_elems):
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device=_dev())
        ws = torch.full((max(ws_elems, 1),), float("nan"), dtype=torch.float32, device=_dev())
        torch.cuda.synchronize()
        zl.zl_kernel_gemm(M, N, K, At.data_ptr(), At.shape[1], a_k, Bt.data_ptr(), Bt.shape[1], b_k,
                          C.data_ptr(), N, zl.ZL_BF16, _stream(),
                          workspace=ws.data_ptr() if ws_elems else None, workspace_elems=ws_elems)
        torch.cuda.synchronize()
        return C
    one = run(0)
    split = run(8 * M * N)
    again = run(8 * M * N)
    assert bool(torch.isfinite(split).all())
    assert torch.equal(split, again)
    assert rel_err(split.cpu().double().numpy(), one.cpu().double().numpy()) < 2e-6
    rows = np.random.default_rng(3).choice(M, size=48, replace=False)
    ridx = torch.tensor(rows, device=_dev())
    a = (At[ridx] if a_k else At[:, ridx].t()).double().cpu().numpy()
    b = (Bt if b_k else Bt.t()).double().cpu().numpy()
    ref = a @ b.T
    assert rel_err(split[ridx].cpu().double().numpy(), ref) < 2e-6


def test_gemm_register_staged_path_with_second_segment():
    """Both operands MN-major with A's row stride 16384 and K = 66000: A's
    tile offsets pass 2^31 bytes, so the direct-to-LDS kernel is not used and
    the register-staged MFMA kernel computes C = A B^T + A2 B2^T."""
    zl = _zl()
    M, N, K, K2, lda = 256, 256, 66000, 16, 16384
    rng = np.random.default_rng(5)
    A = torch.zeros((K, lda), dtype=torch.bfloat16, device=_dev())
    A[:, :M] = torch.tensor(rng.standard_normal((K, M)).astype(np.float32), device=_dev()).to(torch.bfloat16)
    Bt = torch.tensor(rng.standard_normal((K, N)).astype(np.float32), device=_dev()).to(torch.bfloat16)
    A2 = torch.tensor(rng.standard_normal((K2, M)).astype(np.float32), device=_dev()).to(torch.bfloat16)
    B2 = torch.tensor(rng.standard_normal((K2, N)).astype(np.float32), device=_dev()).to(torch.bfloat16)
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device=_dev())
    torch.cuda.synchronize()
    zl.zl_kernel_gemm(M, N, K, A.data_ptr(), lda, False, Bt.data_ptr(), N, False, C.data_ptr(), N,
                      zl.ZL_BF16, _stream(), K2=K2, A2=A2.data_ptr(), lda2=M, B2=B2.data_ptr(),
                      ldb2=N)
    torch.cuda.synchronize()
    ref = _gemm_ref(A[:, :M], Bt, False, False) + _gemm_ref(A2, B2, False, False)
    del A
    got = C.cpu().double().numpy()
    assert np.all(np.isfinite(got))
    assert rel_err(got, ref) < 2e-6


def _attn_inputs(B, S, Hq, Hkv, hd, lens, seed):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, S, Hq, hd)).astype(np.float32)
    k = rng.standard_normal((B, S, Hkv, hd)).astype(np.float32)
    v = rng.standard_normal((B, S, Hkv, hd)).astype(np.float32)
    do = rng.standard_normal((B, S, Hq, hd)).astype(np.float32)
    return q, k, v, do, np.array(lens, np.int32)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,S,Hq,Hkv,hd,lens", [
    (2, 37, 4, 2, 16, [37, 20]),
    (1, 130, 8, 2, 64, [130]),
    (2, 200, 4, 4, 128, [200, 77]),
    (1, 300, 4, 1, 128, [300]),
    (1, 5, 2, 1, 64, [0]),
    (3, 64, 2, 2, 32, [1, 64, 63]),
])
def test_attention_fwd_bwd(dtype, B, S, Hq, Hkv, hd, lens):
    zl = _zl()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    q, k, v, do, lens = _attn_inputs(B, S, Hq, Hkv, hd, lens, S + hd)
    ld = (Hq + 2 * Hkv) * hd
    qkv = np.concatenate([q.reshape(B * S, -1), k.reshape(B * S, -1), v.reshape(B * S, -1)], 1)
    QKV = torch.tensor(qkv, device=_dev()).to(tdt).contiguous()
    DO = torch.tensor(do.reshape(B * S, -1), device=_dev()).to(tdt)
    O = torch.zeros(B * S, Hq * hd, device=_dev(), dtype=tdt)
    LSE = torch.zeros(B, Hq, S, dtype=torch.float32, device=_dev())
    DQKV = torch.zeros_like(QKV)
    DEL = torch.zeros(B, Hq, S, dtype=torch.float32, device=_dev())
    SL = torch.tensor(lens, device=_dev())
    base = QKV.data_ptr()
    esz = QKV.element_size()
    torch.cuda.synchronize()
    args = (B, S, Hq, Hkv, hd, base, base + Hq * hd * esz, base + (Hq + Hkv) * hd * esz, ld,
            SL.data_ptr(), O.data_ptr(), LSE.data_ptr())
    dt = zl.ZL_BF16 if dtype == "bf16" else zl.ZL_F32
    zl.zl_kernel_attention(*args, 0, 0, 0, 0, 0, dt, 0, _stream())
    dbase = DQKV.data_ptr()
    zl.zl_kernel_attention(*args, DO.data_ptr(), dbase, dbase + Hq * hd * esz,
                           dbase + (Hq + Hkv) * hd * esz, DEL.data_ptr(), dt, 1, _stream())
    torch.cuda.synchronize()
    r = QKV.double().cpu().numpy()
    q64 = r[:, : Hq * hd].reshape(B, S, Hq, hd)
    k64 = r[:, Hq * hd: (Hq + Hkv) * hd].reshape(B, S, Hkv, hd)
    v64 = r[:, (Hq + Hkv) * hd:].reshape(B, S, Hkv, hd)
    do64 = DO.double().cpu().numpy().reshape(B, S, Hq, hd)
    o_ref, cache = ops.attention_fwd(q64, k64, v64, lens)
    dq_ref, dk_ref, dv_ref = ops.attention_bwd(do64, cache)
    tol = 1e-5 if dtype == "f32" else 1.2e-2
    o = O.double().cpu().numpy().reshape(B, S, Hq, hd)
    assert rel_err(o, o_ref) < tol
    d = DQKV.double().cpu().numpy()
    assert rel_err(d[:, : Hq * hd].reshape(dq_ref.shape), dq_ref) < tol
    assert rel_err(d[:, Hq * hd: (Hq + Hkv) * hd].reshape(dk_ref.shape), dk_ref) < tol
    assert rel_err(d[:, (Hq + Hkv) * hd:].reshape(dv_ref.shape), dv_ref) < tol
    # lse of rows with at least one visible key
    lse = LSE.cpu().double().numpy()
    scale = 1.0 / np.sqrt(hd)
    for b in range(B):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            s = (q64[b, :, h] @ k64[b, :, g].T) * scale
            allowed = ops.attention_mask(B, S, lens)[b]
            for i in range(S):
                if allowed[i].any():
                    ref = np.log(np.sum(np.exp(s[i][allowed[i]] - s[i][allowed[i]].max()))) + s[i][allowed[i]].max()
                    assert abs(lse[b, h, i] - ref) < 1e-4 * max(1, abs(ref))
                else:
                    assert lse[b, h, i] == -np.inf


def _backward_profile(shp):
    import workload
    from tests.gpu_cases import make_inputs, device_chunk, to_dev
    zl = _zl()
    params, batch = make_inputs(shp, seed=3)
    ch = device_chunk(shp, params, batch)
    d = to_dev(batch, shp.dtype)
    ch.forward(d["h_in"], d["seq_lens"], d["pos_ids"])
    ch.objective(d["labels"])
    torch.cuda.synchronize()
    zl.zl_profile_begin(ch.handle, 4096)
    ch.backward(1.0, 0)
    torch.cuda.synchronize()
    prof = zl.zl_profile_end(ch.handle, 256)
    ch.close()
    return [e for e in prof if e["name"].endswith("_mn")]


def test_backward_pairs_weight_gradients():
    """The weight-gradient GEMMs of an 8B-shaped layer run as two launches,
    down with QKV and up with the output projection (their tiles fill whole
    waves together), each carrying the FLOPs of both; a 1B-shaped layer's
    QKV and output projections have too few tiles to pair and run alone."""
    import workload
    shp = workload.get_config("8b").with_(n_layers=1, batch=1, seq=256)
    T, d, ff = 256, shp.d_model, shp.d_ff
    nqkv = (shp.n_heads + 2 * shp.n_kv_heads) * shp.head_dim
    mn = _backward_profile(shp)
    assert [e["name"] for e in mn] == ["gemm_dma_256x256_mn"]
    assert mn[0]["launches"] == 2
    want = 2.0 * T * (d * ff + 2 * ff * d + d * shp.n_heads * shp.head_dim + nqkv * d)
    assert mn[0]["flops"] == pytest.approx(want, rel=1e-9)
    shp1 = workload.get_config("1b").with_(n_layers=1, batch=1, seq=512)
    launches = sum(e["launches"] for e in _backward_profile(shp1))
    assert launches == 4
