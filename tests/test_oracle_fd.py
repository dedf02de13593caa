"""Finite-difference pins of every gradient the oracle forms.

Central differences in fp64 of the local loss (Eq. (3)-(5) on the frozen head
of Eq. (2), after the chunk map of Eq. (1)) with respect to every trainable
tensor, for both layer forms, both KL directions, alpha in {1, 0.5}, GQA,
right padding and unlabelled positions.
"""
import numpy as np
import pytest

import oracle
from oracle.objective import local_objective_ref
from tests.oracle_cases import rel_err, tiny_case


def _loss(c, P):
    return oracle.chunk_grads_ref(c["cfg"], P, c["h_in"], c["labels"], c["head_w"], c["hn_w"],
                                  c["hn_b"], c["seq_lens"], c["pos_ids"])["loss"]


def _fd_check(c, tol=1e-6):
    r = oracle.chunk_grads_ref(c["cfg"], c["P"], c["h_in"], c["labels"], c["head_w"], c["hn_w"],
                               c["hn_b"], c["seq_lens"], c["pos_ids"])
    assert set(r["grads"]) == set(c["trainable"])
    worst = 0.0
    for key in c["trainable"]:
        val = c["P"][key]
        fd = np.zeros_like(val)
        flat = val.reshape(-1)
        for i in range(flat.size):
            h = 1e-6 * max(1.0, abs(flat[i]))
            Pp = dict(c["P"])
            a = flat.copy()
            a[i] += h
            Pp[key] = a.reshape(val.shape)
            lp = _loss(c, Pp)
            a[i] -= 2 * h
            Pp[key] = a.reshape(val.shape)
            lm = _loss(c, Pp)
            fd.reshape(-1)[i] = (lp - lm) / (2 * h)
        e = rel_err(r["grads"][key], fd)
        worst = max(worst, e)
        assert e < tol, (key, e)
    return worst


@pytest.mark.parametrize("arch", ["llama", "gpt2"])
@pytest.mark.parametrize("alpha,consis", [(1.0, "reverse"), (0.5, "reverse"), (0.5, "forward")])
def test_fd_every_tensor(arch, alpha, consis):
    _fd_check(tiny_case(arch, alpha=alpha, consis=consis))


def test_fd_gqa():
    _fd_check(tiny_case("llama", gqa=True, alpha=0.3))


@pytest.mark.parametrize("arch", ["llama", "gpt2"])
@pytest.mark.parametrize("alpha", [1.0, 0.5])
def test_fd_readout_adapter(arch, alpha):
    """The readout adapter's two weights and every layer tensor through it."""
    _fd_check(tiny_case(arch, alpha=alpha, adapter_rank=3))


@pytest.mark.parametrize("arch", ["llama", "gpt2"])
def test_fd_lora(arch):
    """LoRA factors of every target linear (the base is frozen), with the
    readout adapter on the llama form."""
    _fd_check(tiny_case(arch, alpha=0.5, lora_rank=2, lora_alpha=3.0,
                        adapter_rank=2 if arch == "llama" else 0))


def test_fd_no_padding_one_layer():
    _fd_check(tiny_case("gpt2", alpha=0.7, pad=False, drop_labels=False, L=1))


@pytest.mark.parametrize("arch", ["llama", "gpt2"])
@pytest.mark.parametrize("consis", ["reverse", "forward"])
def test_fd_objective_wrt_h_out(arch, consis):
    """dL/dh_out of the objective alone (head norm frozen)."""
    c = tiny_case(arch, alpha=0.4, consis=consis)
    rng = np.random.default_rng(5)
    T, d = 10, c["shape"].d_model
    h_out = rng.standard_normal((T, d))
    h_in = rng.standard_normal((T, d))
    labels = c["labels"].reshape(-1)
    args = (c["head_w"], arch, c["hn_w"], c["hn_b"], 1e-5, 0.4, consis)
    loss, dh, _ = local_objective_ref(h_out, h_in, labels, *args)
    fd = np.zeros_like(h_out)
    for i in range(T):
        for j in range(d):
            e = 1e-6
            hp = h_out.copy()
            hp[i, j] += e
            hm = h_out.copy()
            hm[i, j] -= e
            fd[i, j] = (local_objective_ref(hp, h_in, labels, *args)[0]
                        - local_objective_ref(hm, h_in, labels, *args)[0]) / (2 * e)
    assert rel_err(dh, fd) < 1e-6
