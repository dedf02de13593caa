"""The no-allocation attention backward (zl_kernel_attention_bwd_noalloc)
against zl_kernel_attention's backward with a caller-provided delta buffer,
through the C ABI: identical dq, dk and dv on two calls in a row, the second
with a smaller input (the scratch array keeps the first call's contents)."""
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _attn_case(B, S, Hq, Hkv, hd, dtype, seed):
    from paper_2608_07974_amd import zl
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev).manual_seed(seed)
    tdt = torch.bfloat16 if dtype == zl.ZL_BF16 else torch.float32
    ld = (Hq + 2 * Hkv) * hd
    qkv = torch.randn(B * S, ld, device=dev, generator=gen).to(tdt)
    dout = torch.randn(B * S, Hq * hd, device=dev, generator=gen).to(tdt)
    o = torch.zeros(B * S, Hq * hd, device=dev, dtype=tdt)
    lse = torch.zeros(B, Hq, S, device=dev, dtype=torch.float32)
    seq = torch.tensor([S - (b * 7) % max(S // 3, 1) for b in range(B)], device=dev,
                       dtype=torch.int32)
    esz = qkv.element_size()
    base = qkv.data_ptr()
    q, k, v = base, base + Hq * hd * esz, base + (Hq + Hkv) * hd * esz
    stream = torch.cuda.current_stream().cuda_stream
    zl.zl_kernel_attention(B, S, Hq, Hkv, hd, q, k, v, ld, seq.data_ptr(), o.data_ptr(),
                           lse.data_ptr(), 0, 0, 0, 0, 0, dtype, 0, stream)
    return dict(B=B, S=S, Hq=Hq, Hkv=Hkv, hd=hd, q=q, k=k, v=v, ld=ld, seq=seq, o=o, lse=lse,
                dout=dout, qkv=qkv, dtype=dtype, stream=stream)


def _grads(c, noalloc):
    from paper_2608_07974_amd import zl
    d = torch.zeros_like(c["qkv"])
    esz = d.element_size()
    Hq, Hkv, hd = c["Hq"], c["Hkv"], c["hd"]
    dq, dk, dv = d.data_ptr(), d.data_ptr() + Hq * hd * esz, d.data_ptr() + (Hq + Hkv) * hd * esz
    args = (c["B"], c["S"], Hq, Hkv, hd, c["q"], c["k"], c["v"], c["ld"], c["seq"].data_ptr(),
            c["o"].data_ptr(), c["lse"].data_ptr(), c["dout"].data_ptr(), dq, dk, dv)
    if noalloc:
        zl.zl_kernel_attention_bwd_noalloc(*args, c["dtype"], c["stream"])
    else:
        delta = torch.zeros(c["B"], Hq, c["S"], device=d.device, dtype=torch.float32)
        zl.zl_kernel_attention(*args[:11], args[11], args[12], dq, dk, dv, delta.data_ptr(),
                               c["dtype"], 1, c["stream"])
    torch.cuda.synchronize()
    return d


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_noalloc_backward_matches_the_allocating_entry_point(dt):
    from paper_2608_07974_amd import zl
    dtype = zl.ZL_BF16 if dt == "bf16" else zl.ZL_F32
    # the second call is smaller than the first
    for shape, seed in (((2, 640, 8, 2, 128), 1), ((1, 200, 4, 4, 64), 2)):
        c = _attn_case(*shape, dtype, seed)
        want = _grads(c, noalloc=False)
        got = _grads(c, noalloc=True)
        assert torch.isfinite(want).all()
        assert torch.equal(got, want), shape


def test_noalloc_rejects_sizes_beyond_its_scratch():
    """B * Hq * S above 2^20 floats is refused before any launch."""
    from paper_2608_07974_amd import zl
    dev = torch.device("cuda:0")
    t = torch.zeros(64, dtype=torch.bfloat16, device=dev)
    s = torch.zeros(4, dtype=torch.int32, device=dev)
    lse = torch.zeros(4, dtype=torch.float32, device=dev)
    p = t.data_ptr()
    with pytest.raises(zl.ZlError) as e:
        zl.zl_kernel_attention_bwd_noalloc(4, 8192, 64, 8, 128, p, p, p, 64, s.data_ptr(), p,
                                           lse.data_ptr(), p, p, p, p, zl.ZL_BF16, 0)
    assert e.value.status == zl.ZL_ERR_UNSUPPORTED and "scratch" in str(e.value)
