"""The C-ABI library loads, exports every symbol its headers declare, and its
host-only calls (layout, workspace, config validation) behave as documented.
No compute call is made here (no GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2608_07974_amd import zl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not h.endswith(".h"):
            continue
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(zl_[a-z_]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    lib = zl.load()
    declared = _declared()
    assert {"zl_chunk_forward", "zl_local_objective", "zl_chunk_backward", "zl_optimizer_step",
            "zl_chunk_update"} <= declared
    for name in declared:
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", zl.LIB_PATH], capture_output=True,
                         text=True).stdout
    exported = set(re.findall(r" T (zl_[a-z_]+)", out))
    assert declared <= exported, declared - exported
    assert set(zl.EXPORTED) == declared


def _cfg(**kw):
    base = dict(rope_theta=1e4, max_batch=4, max_seq=32)
    base.update(kw)
    return zl.make_config(zl.ZL_ARCH_LLAMA, 2, 64, 4, 4, 16, 256, 256, **base)


@pytest.mark.parametrize("adapter_rank", [0, 32])
def test_layout_matches_workload_specs(adapter_rank):
    import workload
    for name in ("tiny", "gpt2", "8b"):
        shp = workload.get_config(name, adapter_rank=adapter_rank)
        arch = zl.ZL_ARCH_LLAMA if shp.arch == "llama" else zl.ZL_ARCH_GPT2
        cfg = zl.make_config(arch, shp.n_layers, shp.d_model, shp.n_heads, shp.n_kv_heads,
                             shp.head_dim, shp.d_ff, shp.vocab, rope_theta=max(shp.rope_theta, 2.0),
                             max_batch=1, max_seq=8, adapter_rank=adapter_rank)
        n, lay = zl.zl_param_layout(cfg)
        specs = workload.param_specs(shp)
        assert [f"L{t['layer']}.{t['name']}" for t in lay] == [k for k, _, _ in specs]
        for t, (_, shape, _) in zip(lay, specs):
            assert tuple(t["shape"]) == tuple(shape)
            assert t["offset"] % 64 == 0
        ends = [t["offset"] + t["numel"] for t in lay]
        assert n >= max(ends) and n % 64 == 0
        # fused projections are adjacent
        by = {(t["layer"], t["name"]): t for t in lay}
        if shp.arch == "llama":
            assert by[(0, "wk")]["offset"] == by[(0, "wq")]["offset"] + by[(0, "wq")]["numel"]
            assert by[(0, "wv")]["offset"] == by[(0, "wk")]["offset"] + by[(0, "wk")]["numel"]
            assert by[(0, "wu")]["offset"] == by[(0, "wg")]["offset"] + by[(0, "wg")]["numel"]
    assert zl.zl_param_layout(zl.make_config(zl.ZL_ARCH_LLAMA, 8, 4096, 32, 8, 128, 14336, 128256,
                                             rope_theta=5e5))[0] >= 1_744_896_000


@pytest.mark.parametrize("adapter_rank", [0, 16])
def test_lora_layout_matches_workload_specs(adapter_rank):
    """With LoRA the trainable layout is the factors (and adapter) in
    param_specs order; the base buffers follow the full layout of the config
    without LoRA and adapter; stacked factors are adjacent."""
    import workload
    for name, r in (("tiny", 8), ("gpt2", 16), ("8b", 8)):
        shp = workload.get_config(name, adapter_rank=adapter_rank, lora_rank=r)
        arch = zl.ZL_ARCH_LLAMA if shp.arch == "llama" else zl.ZL_ARCH_GPT2
        cfg = zl.make_config(arch, shp.n_layers, shp.d_model, shp.n_heads, shp.n_kv_heads,
                             shp.head_dim, shp.d_ff, shp.vocab, rope_theta=max(shp.rope_theta, 2.0),
                             max_batch=1, max_seq=8, adapter_rank=adapter_rank, lora_rank=r)
        n, lay = zl.zl_param_layout(cfg)
        specs = workload.param_specs(shp)
        assert [f"L{t['layer']}.{t['name']}" for t in lay] == [k for k, _, _ in specs]
        for t, (_, shape, _) in zip(lay, specs):
            assert tuple(t["shape"]) == tuple(shape) and t["offset"] % 64 == 0
        assert n >= max(t["offset"] + t["numel"] for t in lay)
        nb, base = zl.zl_param_layout(zl.base_config(cfg))
        assert [f"L{t['layer']}.{t['name']}" for t in base] == \
            [k for k, _, _ in workload.base_specs(shp)]
        if name == "8b":
            assert n * 100 < nb
        by = {(t["layer"], t["name"]): t for t in lay}
        groups = ([("wq_la", "wk_la", "wv_la"), ("wq_lb", "wk_lb", "wv_lb"), ("wg_la", "wu_la"),
                   ("wg_lb", "wu_lb")] if shp.arch == "llama" else [])
        for l in range(shp.n_layers):
            for g in groups:
                for a, b in zip(g, g[1:]):
                    assert by[(l, b)]["offset"] == by[(l, a)]["offset"] + by[(l, a)]["numel"]


@pytest.mark.parametrize("rank,lalpha", [(-8, 16.0), (-1, 16.0), (257, 16.0), (264, 16.0),
                                         (8, 0.0), (4, 0.0), (8, float("nan"))])
def test_lora_rank_validated(rank, lalpha):
    b = ctypes.c_size_t()
    cfg = _cfg(lora_rank=rank, lora_alpha=lalpha)
    assert zl.load().zl_workspace_size(ctypes.byref(cfg), ctypes.byref(b)) == zl.ZL_ERR_INVALID_ARG


@pytest.mark.parametrize("rank", [1, 4, 12])
def test_lora_rank_below_a_multiple_of_8_is_stored_padded(rank):
    """The paper's rank 4 (Sec. IV setting): the factors are stored 8 (16)
    wide, A [r8, in] and B [out, r8], in the order and offsets of the
    rank-r8 layout; the configured rank sets the scale (lora_alpha / r)."""
    import workload
    r8 = (rank + 7) // 8 * 8
    shp = workload.get_config("tiny", lora_rank=rank)
    cfg = zl.make_config(zl.ZL_ARCH_LLAMA, shp.n_layers, shp.d_model, shp.n_heads, shp.n_kv_heads,
                         shp.head_dim, shp.d_ff, shp.vocab, rope_theta=1e4, max_batch=1,
                         max_seq=8, lora_rank=rank, lora_alpha=16.0)
    n, lay = zl.zl_param_layout(cfg)
    cfg8 = zl.make_config(zl.ZL_ARCH_LLAMA, shp.n_layers, shp.d_model, shp.n_heads,
                          shp.n_kv_heads, shp.head_dim, shp.d_ff, shp.vocab, rope_theta=1e4,
                          max_batch=1, max_seq=8, lora_rank=r8, lora_alpha=16.0)
    n8, lay8 = zl.zl_param_layout(cfg8)
    assert n == n8 and lay == lay8
    specs = workload.param_specs(shp)
    for t, (_, shape, _) in zip(lay, specs):
        want = (r8, shape[1]) if t["name"].endswith("_la") else (shape[0], r8)
        assert tuple(t["shape"]) == want


def test_lora_create_needs_base_buffers():
    for dtype, bufs in ((zl.ZL_F32, zl.zl_buffers(4096, 0, 8192, 12288, 16384, 20480, 24576, 0)),
                        (zl.ZL_BF16, zl.zl_buffers(4096, 32768, 8192, 12288, 16384, 20480, 24576, 0,
                                                   28672, 0))):
        with pytest.raises(zl.ZlError) as ei:
            zl.zl_chunk_create(_cfg(lora_rank=8, dtype=dtype), bufs, 256, 1 << 40)
        assert ei.value.status == zl.ZL_ERR_INVALID_ARG and "base" in str(ei.value)


@pytest.mark.parametrize("rank", [-16, 8, 24])
def test_adapter_rank_validated(rank):
    import ctypes
    b = ctypes.c_size_t()
    assert zl.load().zl_workspace_size(ctypes.byref(_cfg(adapter_rank=rank)), ctypes.byref(b)) == \
        zl.ZL_ERR_INVALID_ARG


def test_workspace_grows_with_tokens():
    a = zl.zl_workspace_size(_cfg(max_batch=1, max_seq=16))
    b = zl.zl_workspace_size(_cfg(max_batch=2, max_seq=16))
    assert b > a > 0


@pytest.mark.parametrize("bad,status", [
    (dict(d_model=60), zl.ZL_ERR_INVALID_ARG),
    (dict(n_kv_heads=3), zl.ZL_ERR_INVALID_ARG),
    (dict(alpha=0.0), zl.ZL_ERR_INVALID_ARG),
    (dict(alpha=1.5), zl.ZL_ERR_INVALID_ARG),
    (dict(dtype=7), zl.ZL_ERR_INVALID_ARG),
    (dict(max_seq=0), zl.ZL_ERR_INVALID_ARG),
    (dict(head_dim=24), zl.ZL_ERR_UNSUPPORTED),
    (dict(consis=5), zl.ZL_ERR_INVALID_ARG),
])
def test_config_validation(bad, status):
    base = dict(arch=zl.ZL_ARCH_LLAMA, n_layers=2, d_model=64, n_heads=4, n_kv_heads=4,
                head_dim=16, d_ff=256, vocab=256, rope_theta=1e4, max_batch=4, max_seq=32)
    base.update(bad)
    args = [base.pop(k) for k in ("arch", "n_layers", "d_model", "n_heads", "n_kv_heads",
                                  "head_dim", "d_ff", "vocab")]
    cfg = zl.make_config(*args, **base)
    with pytest.raises(zl.ZlError) as ei:
        zl.zl_workspace_size(cfg)
    assert ei.value.status == status
    assert zl.load().zl_last_error()


def test_create_rejects_bad_buffers_without_gpu():
    cfg = _cfg()
    bufs = zl.zl_buffers(0, 0, 0, 0, 0, 0, 0, 0)
    with pytest.raises(zl.ZlError) as ei:
        zl.zl_chunk_create(cfg, bufs, 0, 0)
    assert ei.value.status == zl.ZL_ERR_INVALID_ARG
    bufs = zl.zl_buffers(4096, 0, 8192, 12288, 16384, 20480, 24576, 0)
    with pytest.raises(zl.ZlError) as ei:
        zl.zl_chunk_create(cfg, bufs, 0, 0)
    assert ei.value.status == zl.ZL_ERR_WORKSPACE
    with pytest.raises(zl.ZlError) as ei:
        zl.zl_chunk_create(cfg, bufs, 256, 16)
    assert ei.value.status == zl.ZL_ERR_WORKSPACE


@pytest.mark.parametrize("M,N,K,a_k,b_k,lda,ldb,A", [
    (129, 136, 1000, False, True, 129, 1000, 4096),   # M-contiguous A, M % 8 != 0
    (128, 130, 64, True, False, 64, 130, 4096),       # N-contiguous B, N % 8 != 0
    (128, 128, 60, True, True, 60, 60, 4096),          # K-contiguous operands, K % 8 != 0
    (128, 128, 64, True, True, 64, 64, 4100),          # A not 16-byte aligned
])
def test_kernel_gemm_rejects_unaligned_bf16(M, N, K, a_k, b_k, lda, ldb, A):
    """bf16 operands are read in 16-byte chunks: a contiguous dimension or
    leading dimension not a multiple of 8 elements, or a pointer not 16-byte
    aligned, is an argument error raised before anything is launched."""
    with pytest.raises(zl.ZlError) as ei:
        zl.zl_kernel_gemm(M, N, K, A, lda, a_k, 8192, ldb, b_k, 12288, N, zl.ZL_BF16)
    assert ei.value.status == zl.ZL_ERR_INVALID_ARG and "8-element" in str(ei.value)


def test_null_handle_calls_fail_cleanly():
    lib = zl.load()
    assert lib.zl_chunk_forward(None, None, None, None, 1, 1, None, None) == zl.ZL_ERR_INVALID_ARG
    assert lib.zl_local_objective(None, None, None, None) == zl.ZL_ERR_INVALID_ARG
    assert lib.zl_chunk_backward(None, 1.0, 0, None) == zl.ZL_ERR_INVALID_ARG
    assert lib.zl_optimizer_step(None, None) == zl.ZL_ERR_INVALID_ARG
    assert zl.status_string(zl.ZL_ERR_STATE) == "ZL_ERR_STATE"
