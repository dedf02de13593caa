"""Host-side runtime checks (no GPU): the checkpoint header parser against
files written here, independently, from the format documented in
include/zl_runtime.h, and argument validation of the pipeline calls."""
import struct

import numpy as np
import pytest

from paper_2608_07974_amd import zl

MAGIC = b"ZLCKPT01"


def _fnv32w(payload):
    """FNV-1a 64 over 32-bit little-endian words, as the format states."""
    h = 0xCBF29CE484222325
    for w in np.frombuffer(payload, dtype="<u4"):
        h ^= int(w)
        h = (h * 0x100000001B3) & 0xFFFFFFFFFFFFFFFF
    return h


def _write(path, *, n=10, optimizer=zl.ZL_ADAMW, tensors=None, shape=(0, 2, 64, 4, 4, 16, 256, 256, 0),
           step=3, mb=12, win=6, magic=MAGIC, header_bytes=256, extra=b"", cut=0, checksum=None):
    tensors = (3 if optimizer == zl.ZL_ADAMW else 1) if tensors is None else tensors
    payload = np.arange(n * max(tensors, 1), dtype=np.float32).tobytes()[: n * tensors * 4]
    ck = _fnv32w(payload) if checksum is None else checksum
    head = magic + struct.pack("<II9iIQqqqQ", header_bytes, optimizer, *shape, tensors, n, step,
                               mb, win, ck)
    head += b"\0" * (256 - len(head))
    data = head + payload + extra
    with open(path, "wb") as f:
        f.write(data[: len(data) - cut] if cut else data)
    return ck


def test_header_fields(tmp_path):
    p = tmp_path / "a.ckpt"
    ck = _write(p)
    info = zl.zl_checkpoint_read_info(str(p))
    assert (info["arch"], info["n_layers"], info["d_model"], info["n_heads"], info["n_kv_heads"],
            info["head_dim"], info["d_ff"], info["vocab"], info["dtype"]) == (0, 2, 64, 4, 4, 16, 256, 256, 0)
    assert info["optimizer"] == zl.ZL_ADAMW and info["n_params"] == 10
    assert (info["step"], info["microbatches"], info["windows"]) == (3, 12, 6)
    assert info["checksum"] == ck


def test_sgd_has_one_tensor(tmp_path):
    p = tmp_path / "s.ckpt"
    _write(p, optimizer=zl.ZL_SGD)
    assert zl.zl_checkpoint_read_info(str(p))["optimizer"] == zl.ZL_SGD


@pytest.mark.parametrize("kw", [dict(magic=b"NOTACKPT"), dict(header_bytes=128), dict(tensors=2),
                                dict(optimizer=7, tensors=1), dict(cut=4), dict(extra=b"\0" * 4)])
def test_malformed_files_rejected(tmp_path, kw):
    p = tmp_path / "bad.ckpt"
    _write(p, **kw)
    with pytest.raises(zl.ZlError) as e:
        zl.zl_checkpoint_read_info(str(p))
    assert e.value.status == zl.ZL_ERR_INVALID_ARG


def test_missing_and_short_files(tmp_path):
    with pytest.raises(zl.ZlError):
        zl.zl_checkpoint_read_info(str(tmp_path / "none.ckpt"))
    p = tmp_path / "short.ckpt"
    p.write_bytes(MAGIC + b"\0" * 20)
    with pytest.raises(zl.ZlError):
        zl.zl_checkpoint_read_info(str(p))


def test_pipeline_calls_reject_null():
    lib = zl.load()
    import ctypes
    n = ctypes.c_size_t()
    assert lib.zl_pipeline_entry_bytes(None, 2, 2, ctypes.byref(n)) == zl.ZL_ERR_INVALID_ARG
    assert lib.zl_pipeline_sync(None) == zl.ZL_ERR_INVALID_ARG
    assert lib.zl_pipeline_progress(None, None, None) == zl.ZL_ERR_INVALID_ARG
    h = ctypes.c_void_p()
    assert lib.zl_pipeline_create(None, 2, None, 1, 1, None, 0, ctypes.byref(h)) == zl.ZL_ERR_INVALID_ARG
    lib.zl_pipeline_destroy(None)  # no-op
