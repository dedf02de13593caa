"""ctypes binding of libzl (include/zl.h, include/zl_inspect.h).

Argument marshalling only: every function here forwards to the C call of the
same name, raising ZlError on a negative status.  Pointers are plain ints
(device addresses); streams are hipStream_t handles as ints (0 = default).
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libzl.so")

ZL_OK, ZL_ERR_INVALID_ARG, ZL_ERR_UNSUPPORTED, ZL_ERR_HIP, ZL_ERR_STATE, ZL_ERR_WORKSPACE = \
    0, -1, -2, -3, -4, -5
ZL_ARCH_LLAMA, ZL_ARCH_GPT2 = 0, 1
ZL_F32, ZL_BF16 = 0, 1
ZL_KL_REVERSE, ZL_KL_FORWARD = 0, 1
ZL_ADAMW, ZL_SGD = 0, 1

EXPORTED = [
    "zl_param_layout", "zl_workspace_size", "zl_chunk_create", "zl_chunk_destroy",
    "zl_refresh_shadow", "zl_chunk_forward", "zl_local_objective", "zl_chunk_backward",
    "zl_optimizer_step", "zl_chunk_update", "zl_get_step", "zl_set_step",
    "zl_status_string", "zl_last_error", "zl_inspect", "zl_kernel_gemm", "zl_kernel_attention",
    "zl_profile_begin", "zl_profile_end", "zl_device_info",
    "zl_chunk_get_config", "zl_chunk_get_buffers", "zl_chunk_num_params",
    "zl_pipeline_entry_bytes", "zl_pipeline_create", "zl_pipeline_submit", "zl_pipeline_read_output",
    "zl_pipeline_sync", "zl_pipeline_progress", "zl_pipeline_checkpoint", "zl_pipeline_destroy",
    "zl_chunk_save", "zl_chunk_load", "zl_checkpoint_read_info",
    "zl_kernel_attention_bwd_noalloc",
]


class ZlError(RuntimeError):
    def __init__(self, status, func, detail):
        self.status = status
        super().__init__(f"{func}: {status_string(status)} ({status}): {detail}")


class zl_config(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_int), ("n_layers", ctypes.c_int), ("d_model", ctypes.c_int),
                ("n_heads", ctypes.c_int), ("n_kv_heads", ctypes.c_int),
                ("head_dim", ctypes.c_int), ("d_ff", ctypes.c_int), ("vocab", ctypes.c_int),
                ("norm_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("dtype", ctypes.c_int), ("alpha", ctypes.c_float), ("consis", ctypes.c_int),
                ("optimizer", ctypes.c_int), ("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("max_batch", ctypes.c_int),
                ("max_seq", ctypes.c_int), ("adapter_rank", ctypes.c_int),
                ("lora_rank", ctypes.c_int), ("lora_alpha", ctypes.c_float)]


class zl_tensor_desc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 16), ("layer", ctypes.c_int), ("ndim", ctypes.c_int),
                ("shape", ctypes.c_int64 * 2), ("offset", ctypes.c_size_t),
                ("numel", ctypes.c_size_t)]


class zl_buffers(ctypes.Structure):
    _fields_ = [("master", ctypes.c_void_p), ("shadow", ctypes.c_void_p),
                ("grad", ctypes.c_void_p), ("adam_m", ctypes.c_void_p),
                ("adam_v", ctypes.c_void_p), ("head_w", ctypes.c_void_p),
                ("head_norm_w", ctypes.c_void_p), ("head_norm_b", ctypes.c_void_p),
                ("base_master", ctypes.c_void_p), ("base_shadow", ctypes.c_void_p)]


class zl_view(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_void_p), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("ld", ctypes.c_int64), ("dtype", ctypes.c_int)]


class zl_checkpoint_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("arch", "n_layers", "d_model", "n_heads",
                                              "n_kv_heads", "head_dim", "d_ff", "vocab",
                                              "dtype", "optimizer")] + \
               [("n_params", ctypes.c_uint64), ("step", ctypes.c_int64),
                ("microbatches", ctypes.c_int64), ("windows", ctypes.c_int64),
                ("checksum", ctypes.c_uint64)]


class zl_profile_entry(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double)]


_lib = None


def load(path=None):
    """Load libzl.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"libzl.so not found at {p}; build it with "
                           "`python -m paper_2608_07974_amd.build` (or __graft_entry__.build())")
    lib = ctypes.CDLL(p)
    c, vp, i64, sz = ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "zl_param_layout": [P(zl_config), P(sz), P(zl_tensor_desc), P(c)],
        "zl_workspace_size": [P(zl_config), P(sz)],
        "zl_chunk_create": [P(zl_config), P(zl_buffers), vp, sz, P(vp)],
        "zl_chunk_destroy": [vp],
        "zl_refresh_shadow": [vp, vp],
        "zl_chunk_forward": [vp, vp, vp, vp, c, c, vp, vp],
        "zl_local_objective": [vp, vp, vp, vp],
        "zl_chunk_backward": [vp, ctypes.c_float, c, vp],
        "zl_optimizer_step": [vp, vp],
        "zl_chunk_update": [vp, vp, vp, vp, vp, c, c, vp, vp, vp],
        "zl_get_step": [vp, P(i64)],
        "zl_set_step": [vp, i64],
        "zl_status_string": [c],
        "zl_last_error": [],
        "zl_inspect": [vp, ctypes.c_char_p, c, P(zl_view)],
        "zl_kernel_gemm": [c, c, c, vp, i64, c, vp, i64, c, c, vp, i64, vp, i64, vp, i64, vp, sz, c,
                           vp],
        "zl_kernel_attention": [c, c, c, c, c, vp, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp, vp,
                                c, c, vp],
        "zl_kernel_attention_bwd_noalloc": [c, c, c, c, c, vp, vp, vp, i64, vp, vp, vp, vp, vp,
                                            vp, vp, c, vp],
        "zl_profile_begin": [vp, c],
        "zl_profile_end": [vp, P(zl_profile_entry), P(c)],
        "zl_device_info": [c, P(c), P(c), ctypes.c_char_p, c],
        "zl_chunk_get_config": [vp, P(zl_config)],
        "zl_chunk_get_buffers": [vp, P(zl_buffers)],
        "zl_chunk_num_params": [vp, P(sz)],
        "zl_pipeline_entry_bytes": [vp, c, c, P(sz)],
        "zl_pipeline_create": [P(vp), c, P(vp), c, c, vp, sz, P(vp)],
        "zl_pipeline_submit": [vp, vp, vp, vp, vp, c, c, vp, P(i64)],
        "zl_pipeline_read_output": [vp, i64, vp, vp],
        "zl_pipeline_sync": [vp],
        "zl_pipeline_progress": [vp, P(i64), P(i64)],
        "zl_pipeline_checkpoint": [vp, c, ctypes.c_char_p],
        "zl_pipeline_destroy": [vp],
        "zl_chunk_save": [vp, ctypes.c_char_p, i64, i64, vp],
        "zl_chunk_load": [vp, ctypes.c_char_p, P(i64), P(i64), vp],
        "zl_checkpoint_read_info": [ctypes.c_char_p, P(zl_checkpoint_info)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = c
    lib.zl_chunk_destroy.restype = None
    lib.zl_status_string.restype = ctypes.c_char_p
    lib.zl_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(s):
    return load().zl_status_string(s).decode()


def _check(st, name):
    if st != ZL_OK:
        raise ZlError(st, name, load().zl_last_error().decode())


def make_config(arch, n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, *,
                norm_eps=1e-5, rope_theta=1e4, dtype=ZL_F32, alpha=0.5, consis=ZL_KL_REVERSE,
                optimizer=ZL_ADAMW, lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8,
                weight_decay=0.01, max_batch=1, max_seq=1, adapter_rank=0, lora_rank=0,
                lora_alpha=16.0):
    return zl_config(arch, n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab,
                     norm_eps, rope_theta, dtype, alpha, consis, optimizer, lr, beta1, beta2,
                     eps, weight_decay, max_batch, max_seq, adapter_rank, lora_rank, lora_alpha)


def base_config(cfg):
    """The config whose zl_param_layout lays out the frozen base buffers of
    a LoRA chunk (lora_rank = adapter_rank = 0)."""
    b = zl_config()
    ctypes.pointer(b)[0] = cfg
    b.lora_rank = 0
    b.adapter_rank = 0
    return b


def zl_param_layout(cfg):
    """Returns (n_params, [dict(name, layer, shape, offset, numel)])."""
    lib = load()
    n = ctypes.c_size_t()
    cnt = ctypes.c_int()
    _check(lib.zl_param_layout(ctypes.byref(cfg), ctypes.byref(n), None, ctypes.byref(cnt)),
           "zl_param_layout")
    arr = (zl_tensor_desc * cnt.value)()
    _check(lib.zl_param_layout(ctypes.byref(cfg), ctypes.byref(n), arr, ctypes.byref(cnt)),
           "zl_param_layout")
    out = []
    for t in arr:
        shape = (t.shape[0],) if t.ndim == 1 else (t.shape[0], t.shape[1])
        out.append(dict(name=t.name.decode(), layer=t.layer, shape=shape, offset=t.offset,
                        numel=t.numel))
    return n.value, out


def zl_workspace_size(cfg):
    b = ctypes.c_size_t()
    _check(load().zl_workspace_size(ctypes.byref(cfg), ctypes.byref(b)), "zl_workspace_size")
    return b.value


def zl_chunk_create(cfg, bufs, workspace, ws_bytes):
    h = ctypes.c_void_p()
    _check(load().zl_chunk_create(ctypes.byref(cfg), ctypes.byref(bufs), workspace, ws_bytes,
                                  ctypes.byref(h)), "zl_chunk_create")
    return h.value


def zl_chunk_destroy(h):
    load().zl_chunk_destroy(h)


def zl_refresh_shadow(h, stream=0):
    _check(load().zl_refresh_shadow(h, stream), "zl_refresh_shadow")


def zl_chunk_forward(h, h_in, seq_lens, pos_ids, B, S, h_out, stream=0):
    _check(load().zl_chunk_forward(h, h_in, seq_lens, pos_ids, B, S, h_out, stream),
           "zl_chunk_forward")


def zl_local_objective(h, labels, loss_out, stream=0):
    _check(load().zl_local_objective(h, labels, loss_out, stream), "zl_local_objective")


def zl_chunk_backward(h, grad_scale=1.0, accumulate=0, stream=0):
    _check(load().zl_chunk_backward(h, grad_scale, accumulate, stream), "zl_chunk_backward")


def zl_optimizer_step(h, stream=0):
    _check(load().zl_optimizer_step(h, stream), "zl_optimizer_step")


def zl_chunk_update(h, h_in, seq_lens, pos_ids, labels, B, S, h_out, loss_out, stream=0):
    _check(load().zl_chunk_update(h, h_in, seq_lens, pos_ids, labels, B, S, h_out, loss_out,
                                  stream), "zl_chunk_update")


def zl_get_step(h):
    v = ctypes.c_int64()
    _check(load().zl_get_step(h, ctypes.byref(v)), "zl_get_step")
    return v.value


def zl_set_step(h, step):
    _check(load().zl_set_step(h, step), "zl_set_step")


def zl_inspect(h, name, layer=0):
    v = zl_view()
    _check(load().zl_inspect(h, name.encode(), layer, ctypes.byref(v)), "zl_inspect")
    return dict(ptr=v.ptr, rows=v.rows, cols=v.cols, ld=v.ld, dtype=v.dtype)


def zl_kernel_gemm(M, N, K, A, lda, a_kmajor, B, ldb, b_kmajor, C, ldc, dtype, stream=0,
                   K2=0, A2=None, lda2=0, B2=None, ldb2=0, workspace=None, workspace_elems=0):
    _check(load().zl_kernel_gemm(M, N, K, A, lda, int(a_kmajor), B, ldb, int(b_kmajor), K2, A2,
                                 lda2, B2, ldb2, C, ldc, workspace, workspace_elems, dtype, stream),
           "zl_kernel_gemm")


def zl_kernel_attention(B, S, Hq, Hkv, hd, q, k, v, ld_qkv, seq_lens, o, lse, dout, dq, dk, dv,
                        delta, dtype, backward, stream=0):
    _check(load().zl_kernel_attention(B, S, Hq, Hkv, hd, q, k, v, ld_qkv, seq_lens, o, lse, dout,
                                      dq, dk, dv, delta, dtype, int(backward), stream),
           "zl_kernel_attention")


def zl_kernel_attention_bwd_noalloc(B, S, Hq, Hkv, hd, q, k, v, ld_qkv, seq_lens, o, lse, dout,
                                    dq, dk, dv, dtype, stream=0):
    _check(load().zl_kernel_attention_bwd_noalloc(B, S, Hq, Hkv, hd, q, k, v, ld_qkv, seq_lens, o,
                                                  lse, dout, dq, dk, dv, dtype, stream),
           "zl_kernel_attention_bwd_noalloc")


def zl_profile_begin(h, capacity=4096):
    _check(load().zl_profile_begin(h, capacity), "zl_profile_begin")


def zl_device_info(device=0):
    """Returns dict(cu_count, clock_khz, arch) of HIP device `device`."""
    cu, clk = ctypes.c_int(0), ctypes.c_int(0)
    arch = ctypes.create_string_buffer(64)
    _check(load().zl_device_info(device, ctypes.byref(cu), ctypes.byref(clk), arch, 64),
           "zl_device_info")
    return dict(cu_count=cu.value, clock_khz=clk.value, arch=arch.value.decode())


def zl_chunk_get_config(h):
    cfg = zl_config()
    _check(load().zl_chunk_get_config(h, ctypes.byref(cfg)), "zl_chunk_get_config")
    return cfg


def zl_chunk_num_params(h):
    n = ctypes.c_size_t()
    _check(load().zl_chunk_num_params(h, ctypes.byref(n)), "zl_chunk_num_params")
    return n.value


def zl_pipeline_entry_bytes(first_chunk, K, depth):
    n = ctypes.c_size_t()
    _check(load().zl_pipeline_entry_bytes(first_chunk, K, depth, ctypes.byref(n)),
           "zl_pipeline_entry_bytes")
    return n.value


def zl_pipeline_create(chunks, streams, window, depth, entries, entry_bytes):
    K = len(chunks)
    ch = (ctypes.c_void_p * K)(*chunks)
    st = (ctypes.c_void_p * K)(*streams)
    h = ctypes.c_void_p()
    _check(load().zl_pipeline_create(ch, K, st, window, depth, entries, entry_bytes,
                                     ctypes.byref(h)), "zl_pipeline_create")
    return h.value


def zl_pipeline_submit(p, h0, labels, pos_ids, seq_lens, B, S, losses):
    mb = ctypes.c_int64()
    _check(load().zl_pipeline_submit(p, h0, labels, pos_ids, seq_lens, B, S, losses,
                                     ctypes.byref(mb)), "zl_pipeline_submit")
    return mb.value


def zl_pipeline_read_output(p, mb, dst, stream=0):
    _check(load().zl_pipeline_read_output(p, mb, dst, stream), "zl_pipeline_read_output")


def zl_pipeline_sync(p):
    _check(load().zl_pipeline_sync(p), "zl_pipeline_sync")


def zl_pipeline_progress(p):
    mb, w = ctypes.c_int64(), ctypes.c_int64()
    _check(load().zl_pipeline_progress(p, ctypes.byref(mb), ctypes.byref(w)),
           "zl_pipeline_progress")
    return mb.value, w.value


def zl_pipeline_checkpoint(p, stage, path):
    _check(load().zl_pipeline_checkpoint(p, stage, os.fsencode(path)), "zl_pipeline_checkpoint")


def zl_pipeline_destroy(p):
    load().zl_pipeline_destroy(p)


def zl_chunk_save(h, path, microbatches=0, windows=0, stream=0):
    _check(load().zl_chunk_save(h, os.fsencode(path), microbatches, windows, stream),
           "zl_chunk_save")


def zl_chunk_load(h, path, stream=0):
    """Restores the chunk; returns (microbatches, windows) progress."""
    mb, w = ctypes.c_int64(), ctypes.c_int64()
    _check(load().zl_chunk_load(h, os.fsencode(path), ctypes.byref(mb), ctypes.byref(w), stream),
           "zl_chunk_load")
    return mb.value, w.value


def zl_checkpoint_read_info(path):
    info = zl_checkpoint_info()
    _check(load().zl_checkpoint_read_info(os.fsencode(path), ctypes.byref(info)),
           "zl_checkpoint_read_info")
    return {n: getattr(info, n) for n, _ in zl_checkpoint_info._fields_}


def zl_profile_end(h, max_entries=256):
    """Returns [dict(name, launches, total_ms, flops, bytes)] per kernel name."""
    arr = (zl_profile_entry * max_entries)()
    n = ctypes.c_int(max_entries)
    _check(load().zl_profile_end(h, arr, ctypes.byref(n)), "zl_profile_end")
    return [dict(name=e.name.decode(), launches=e.launches, total_ms=e.total_ms, flops=e.flops,
                 bytes=e.bytes) for e in arr[: min(n.value, max_entries)]]
