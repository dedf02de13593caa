"""Host-side argument checks of the torch binding (no GPU): every tensor
whose size or placement the kernels take on trust from B and S is checked
before a pointer reaches libzl."""
import pytest

torch = pytest.importorskip("torch")
from paper_2608_07974_amd.chunk import check_batch  # noqa: E402

D = 64
CPU = torch.device("cpu")


def _ok(B=2, S=8, dtype=torch.bfloat16):
    return dict(h_in=torch.zeros(B, S, D, dtype=dtype),
                seq_lens=torch.full((B,), S, dtype=torch.int32),
                pos_ids=torch.zeros(B * S, dtype=torch.int32),
                labels=torch.zeros(B, S, dtype=torch.int32),
                h_out=torch.zeros(B, S, D, dtype=dtype))


def _check(**kw):
    args = _ok()
    args.update(kw)
    check_batch(torch.bfloat16, D, CPU, max_batch=4, max_seq=16, **args)


def test_valid_batch_passes():
    _check()
    check_batch(torch.bfloat16, D, CPU, torch.zeros(1, 1, D, dtype=torch.bfloat16))


@pytest.mark.parametrize("kw,exc", [
    (dict(h_in=torch.zeros(2, 8, D, dtype=torch.float32)), TypeError),      # dtype
    (dict(h_in=torch.zeros(2, 8, 2 * D, dtype=torch.bfloat16)[:, :, :D]), TypeError),  # strided
    (dict(h_in=torch.zeros(16, D, dtype=torch.bfloat16)), TypeError),       # not [B, S, d]
    (dict(h_in=torch.zeros(2, 8, 32, dtype=torch.bfloat16)), ValueError),   # wrong d_model
    (dict(h_in=torch.zeros(8, 8, D, dtype=torch.bfloat16)), ValueError),    # B > max_batch
    (dict(h_in=torch.zeros(2, 32, D, dtype=torch.bfloat16)), ValueError),   # S > max_seq
    (dict(labels=torch.zeros(2, 7, dtype=torch.int32)), ValueError),        # short labels
    (dict(labels=torch.zeros(2, 8, dtype=torch.int64)), TypeError),         # labels dtype
    (dict(pos_ids=torch.zeros(15, dtype=torch.int32)), ValueError),         # short pos_ids
    (dict(seq_lens=torch.zeros(1, dtype=torch.int32)), ValueError),         # short seq_lens
    (dict(h_out=torch.zeros(2, 8, D, dtype=torch.float32)), TypeError),     # h_out dtype
    (dict(h_out=torch.zeros(2, 4, D, dtype=torch.bfloat16)), TypeError),    # h_out shape
])
def test_bad_batch_raises(kw, exc):
    with pytest.raises(exc):
        _check(**kw)


def test_host_tensors_rejected_for_a_device_chunk():
    """A CPU tensor handed to a chunk on a GPU would be dereferenced as a
    device address by the kernels."""
    args = _ok()
    with pytest.raises(ValueError, match="must be on"):
        check_batch(torch.bfloat16, D, torch.device("meta"), **args)
