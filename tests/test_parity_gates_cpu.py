"""The parity gates themselves, on the CPU (tests/parity.py).

A result that differs from the oracle only by bf16 storage (the oracle with
OracleConfig.store_bf16, reading r4) passes the gates; the same result with
one planted mistake fails them.  The stored bf16 floors are re-derived from
the oracle for one case and must match tests/golden/bf16_floor.json, and a
floor is refused for inputs other than the ones it was measured on."""
import copy
import json

import numpy as np
import pytest

from oracle import bf16_round
from tests import gpu_cases, parity
from tests.gpu_cases import make_inputs, oracle_run
from workload.configs import ChunkShape

# a small bf16 Llama chunk: 2 layers, GQA 4/2 x 64, ff 512, V 1000, 2 x 64 tokens
SHP = ChunkShape("gate", "llama", 2, 256, 4, 2, 64, 512, 1000, 2, 64, "bf16", 1e4, 2)


def _runs(optimizer, steps=1, lr=1e-4):
    params, batch = make_inputs(SHP, seq_lens=[64, 41], drop=6)
    kw = dict(alpha=0.5, optimizer=optimizer, lr=lr)
    exact = oracle_run(SHP, params, batch, steps=steps, **kw)
    faithful = oracle_run(SHP, params, batch, steps=steps, store_bf16=True, **kw)
    faithful["h_out"] = bf16_round(faithful["h_out"])
    # the device keeps its master in fp32
    faithful["masters"] = [{k: v.astype(np.float32).astype(np.float64) for k, v in m.items()}
                           for m in faithful["masters"]]
    floor = {k: v for k, v in parity.results_metrics(faithful, exact).items()
             if k in ("h_out", "dh_out") or k.startswith("g")}
    return exact, faithful, floor


@pytest.fixture(scope="module")
def adamw():
    return _runs("adamw", steps=2)


@pytest.fixture(scope="module")
def sgd():
    return _runs("sgd", lr=1e-2)


def test_faithful_bf16_result_passes(adamw, sgd):
    exact, faithful, floor = adamw
    checks = parity.gate(faithful, exact, "bf16", "adamw", floor)
    # the AdamW deltas are gated, on a good share of every matrix
    assert any(k.startswith("d1:") for k in checks) and any(k.startswith("d2:") for k in checks)
    exact, faithful, floor = sgd
    parity.gate(faithful, exact, "bf16", "sgd", floor)


def _fails(dev, ref, optimizer, floor):
    with pytest.raises(AssertionError, match="parity gate failed"):
        parity.gate(dev, ref, "bf16", optimizer, floor)


def test_one_wrong_column_of_h_out_fails(adamw):
    """One feature column of h_out replaced (here by its neighbour): the
    whole-tensor error stays within 2e-2 (1 of 256 columns), the column
    metric does not."""
    exact, faithful, floor = adamw
    bad = copy.deepcopy(faithful)
    bad["h_out"] = bad["h_out"].copy()
    bad["h_out"][..., 17] = bad["h_out"][..., 18]
    assert parity.rel_err(bad["h_out"], exact["h_out"]) < 0.1
    _fails(bad, exact, "adamw", floor)


def test_one_wrong_token_row_of_dh_out_fails(adamw):
    exact, faithful, floor = adamw
    bad = copy.deepcopy(faithful)
    bad["dh_out"] = bad["dh_out"].copy()
    bad["dh_out"][1, 5, :] *= -1.0
    _fails(bad, exact, "adamw", floor)


@pytest.mark.parametrize("key", ["L0.wq", "L1.wd", "L0.wg"])
def test_one_wrong_row_of_a_weight_gradient_fails(adamw, key):
    exact, faithful, floor = adamw
    bad = copy.deepcopy(faithful)
    g = bad["grads"][0][key]
    i = int(np.argmax(np.linalg.norm(g, axis=1)))
    g[i] = 0.0
    _fails(bad, exact, "adamw", floor)


def test_one_wrong_element_of_a_norm_gradient_fails(adamw):
    exact, faithful, floor = adamw
    bad = copy.deepcopy(faithful)
    g = bad["grads"][0]["L1.ln2_w"]
    i = int(np.argmax(np.abs(g)))
    g[i] = -g[i]
    _fails(bad, exact, "adamw", floor)


def test_adamw_without_bias_correction_fails(adamw):
    """Parameters after the step pass their 2e-2 gate either way (one step
    moves them by about lr); the update deltas do not."""
    exact, faithful, floor = adamw
    bad = copy.deepcopy(faithful)
    for s in (1, 2):
        for k in bad["masters"][s]:
            d = bad["masters"][s][k] - bad["masters"][s - 1][k]
            bad["masters"][s][k] = bad["masters"][s - 1][k] + d * np.sqrt(1 - 0.999) / (1 - 0.9)
    assert all(parity.rel_err(bad["masters"][1][k], exact["masters"][1][k]) < 2e-2
               for k in exact["masters"][1])
    _fails(bad, exact, "adamw", floor)


def test_sgd_with_a_wrong_learning_rate_fails(sgd):
    exact, faithful, floor = sgd
    bad = copy.deepcopy(faithful)
    for k in bad["masters"][1]:
        d = bad["masters"][1][k] - bad["masters"][0][k]
        bad["masters"][1][k] = bad["masters"][0][k] + 1.05 * d
    _fails(bad, exact, "sgd", floor)


def test_stored_floor_is_rederived_from_the_oracle():
    """tests/golden/bf16_floor.json holds what the oracle gives (one case
    recomputed here; the generator computes all of them the same way)."""
    from tests.golden.make_bf16_floor import floor_of
    stored = json.load(open(parity.FLOOR_FILE))
    assert set(stored) == set(gpu_cases.BF16_CASES)
    name = "gpt2_sgd_forward_kl"
    got = floor_of(name)
    assert got["fingerprint"] == stored[name]["fingerprint"]
    assert set(got["tensors"]) == set(stored[name]["tensors"])
    for k, m in got["tensors"].items():
        for metric, v in m.items():
            assert v == pytest.approx(stored[name]["tensors"][k][metric], rel=1e-6, abs=1e-12), \
                (k, metric)
    # every floor is a real rounding effect, well inside the gates' reach
    for case in stored.values():
        for k, m in case["tensors"].items():
            assert 0.0 < m["rel"] < 0.2, k


def test_floor_refused_for_other_inputs():
    shp, kw, steps, params, batch = gpu_cases.case_inputs("gpt2_sgd_forward_kl")
    parity.load_floor("gpt2_sgd_forward_kl", params, batch)
    batch = dict(batch, h_in=batch["h_in"] * 1.5)
    with pytest.raises(ValueError, match="changed"):
        parity.load_floor("gpt2_sgd_forward_kl", params, batch)
