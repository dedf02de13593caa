"""Writes bf16_floor.json: the bf16 storage floor of every bf16 parity case.

For each case of tests/gpu_cases.BF16_CASES the oracle runs twice on the
case's inputs: exactly, and with every intermediate that a bf16
implementation stores in bf16 rounded there (OracleConfig.store_bf16,
reading r4), the arithmetic staying fp64.  The second run differs from the
first by what bf16 storage alone costs; the GPU parity gates of a tensor sit
at a stated multiple of that floor (tests/parity.py).  Only oracle/ and the
seeded inputs of workload/ are used.

    python tests/golden/make_bf16_floor.py [case ...]
"""
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import bf16_round  # noqa: E402
from tests import gpu_cases, parity  # noqa: E402


def _metrics(rounded, exact):
    rounded = dict(rounded, h_out=bf16_round(rounded["h_out"]))  # h_out leaves in bf16
    return {k: {m: float(v) for m, v in d.items()}
            for k, d in parity.results_metrics(rounded, exact).items()
            if k in ("h_out", "dh_out") or k.startswith("g")}


def step_floors(name):
    """Floors of each step of a several-step case, each taken from the same
    state of the exact trajectory: the exact step against the bf16-storage
    step from those parameters and optimizer moments."""
    from oracle.chunk import chunk_update_ref, init_opt_state
    shp, kw, steps, params, batch = gpu_cases.case_inputs(name)
    fp = parity.fingerprint(params, batch)
    mb = dict(h_in=batch["h_in"], labels=batch["labels"], seq_lens=batch["seq_lens"],
              pos_ids=batch["pos_ids"])
    P = {k: np.asarray(v, np.float64) for k, v in params.items()}
    st = init_opt_state()
    out = []
    for _ in range(steps):
        runs = []
        for store in (False, True):
            cfg = gpu_cases.oracle_cfg(shp, store_bf16=store, **kw)
            r = chunk_update_ref(cfg, P, st, [mb], batch["head_w"], batch["head_norm_w"],
                                 batch["head_norm_b"], grad_scale=1.0)
            runs.append(r)
        one = [dict(losses=r["losses"], grads=[r["grads"]], h_out=r["runs"][0]["h_out"],
                    dh_out=r["runs"][0]["dh_out"]) for r in runs]
        out.append(_metrics(one[1], one[0]))
        P, st = runs[0]["params"], runs[0]["state"]
        del runs, one
    return fp, out


def floor_of(name):
    if gpu_cases.BF16_CASES[name].get("steps", 1) > 1:
        fp, steps = step_floors(name)
        return dict(fingerprint=fp, loss_rel=None, tensors=steps[0], steps=steps)
    exact, (params, batch) = gpu_cases.case_oracle(name, masters=False)
    exact.pop("masters")
    fp = parity.fingerprint(params, batch)
    del params, batch
    rounded, _ = gpu_cases.case_oracle(name, store_bf16=True, masters=False)
    rounded.pop("masters")
    # the chunk's output itself is handed over in bf16
    rounded["h_out"] = bf16_round(rounded["h_out"])
    tensors = {k: {m: float(v) for m, v in d.items()}
               for k, d in parity.results_metrics(rounded, exact).items()
               if k in ("h_out", "dh_out") or k.startswith("g")}
    return dict(fingerprint=fp,
                loss_rel=float(abs(rounded["losses"][0] - exact["losses"][0]) /
                               abs(exact["losses"][0])),
                tensors=tensors)


def main(names):
    for name in names:
        t0 = time.time()
        f = floor_of(name)
        worst = max(f["tensors"].items(), key=lambda kv: kv[1]["rel"])
        print(f"{name}: {time.time() - t0:.0f} s, worst rel {worst[0]} {worst[1]['rel']:.4f}",
              flush=True)
        # read, add, write at once: several cases may be generated side by side
        out = json.load(open(parity.FLOOR_FILE)) if os.path.exists(parity.FLOOR_FILE) else {}
        out[name] = f
        tmp = parity.FLOOR_FILE + f".{os.getpid()}"
        json.dump(out, open(tmp, "w"), indent=1, sort_keys=True)
        os.replace(tmp, parity.FLOOR_FILE)


if __name__ == "__main__":
    main(sys.argv[1:] or list(gpu_cases.BF16_CASES))
