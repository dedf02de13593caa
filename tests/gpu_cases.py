"""Builders shared by the GPU tests (not collected by pytest).

Every GPU result comes from libzl through the C ABI; every expected value
comes from oracle/ on the same seeded inputs (workload/)."""
import numpy as np

import oracle
import workload
from oracle.chunk import chunk_forward_ref, init_opt_state

from tests.parity import rel_err  # noqa: F401  (re-exported for the GPU tests)

ARCH = {"llama": 0, "gpt2": 1}


def zl_cfg(shp, **kw):
    from paper_2608_07974_amd.chunk import config_from_shape
    return config_from_shape(shp, **kw)


def oracle_cfg(shp, alpha=0.5, consis="reverse", optimizer="adamw", lr=1e-4, wd=0.01,
               store_bf16=False):
    return oracle.OracleConfig.from_shape(shp, alpha=alpha, consis=consis, optimizer=optimizer,
                                          lr=lr, weight_decay=wd, store_bf16=store_bf16)


def make_inputs(shp, seed=0, stress=True, seq_lens=None, drop=0, tokens_seed=1):
    """Seeded parameters and batch; parity cases perturb norms/biases and use
    the stress scale so the consistency term is exercised.  The batch's
    tokens (and so h_in and the labels) come from tokens_seed."""
    params = workload.init_params(workload.param_specs(shp), seed=seed, perturb=True, stress=stress)
    if getattr(shp, "lora_rank", 0):  # the frozen base of a LoRA chunk
        params.update(workload.init_params(workload.base_specs(shp), seed=seed + 50, perturb=True,
                                           stress=stress))
    batch = workload.make_batch(shp, seed_tokens=tokens_seed, stress=stress, seq_lens=seq_lens,
                                perturb_head=True)
    if drop:
        rng = np.random.default_rng(seed + 7)
        lab = batch["labels"].reshape(-1)
        lab[rng.choice(lab.size, size=drop, replace=False)] = -100
    return params, batch


def device_chunk(shp, params, batch, **cfg_kw):
    import torch
    from paper_2608_07974_amd.chunk import TorchChunk
    ch = TorchChunk(zl_cfg(shp, **cfg_kw))
    ch.load_params(params)
    ch.load_head(batch["head_w"], batch["head_norm_w"], batch["head_norm_b"])
    return ch


def to_dev(batch, dtype):
    import torch
    dev = torch.device("cuda")
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    return dict(h_in=torch.tensor(batch["h_in"], device=dev).to(tdt),
                labels=torch.tensor(batch["labels"], device=dev),
                seq_lens=torch.tensor(batch["seq_lens"], device=dev),
                pos_ids=torch.tensor(batch["pos_ids"], device=dev))


def oracle_run(shp, params, batch, steps=1, store_bf16=False, masters=True, **kw):
    """The oracle's update of one micro-batch, `steps` times: losses, h_out
    and dL/dh_out of the first step, gradients and parameters of every
    step.  store_bf16 rounds stored intermediates to bf16 (the storage
    floor of reading r4)."""
    cfg = oracle_cfg(shp, store_bf16=store_bf16, **kw)
    mb = dict(h_in=batch["h_in"], labels=batch["labels"], seq_lens=batch["seq_lens"],
              pos_ids=batch["pos_ids"])
    P, st = {k: np.asarray(v, np.float64) for k, v in params.items()}, init_opt_state()
    keep = _trainable(shp) if masters else []
    res = dict(grads=[], masters=[{k: P[k] for k in keep}], losses=[])
    for _ in range(steps):
        r = oracle.chunk_update_ref(cfg, P, st, [mb], batch["head_w"], batch["head_norm_w"],
                                    batch["head_norm_b"], grad_scale=1.0)
        if not res["grads"]:
            res["h_out"] = r["runs"][0]["h_out"]
            res["dh_out"] = r["runs"][0]["dh_out"]
        res["losses"].append(r["losses"][0])
        res["grads"].append(r["grads"])
        P, st = r["params"], r["state"]
        res["masters"].append({k: P[k] for k in keep})
        del r
    return res


def oracle_window(shp, params, batches, store_bf16=False, **kw):
    """One window of micro-batches (grad_scale 1/m, accumulate) and one step."""
    cfg = oracle_cfg(shp, store_bf16=store_bf16, **kw)
    b1 = batches[0]
    mbs = [dict(h_in=b["h_in"], labels=b["labels"], seq_lens=b["seq_lens"], pos_ids=b["pos_ids"])
           for b in batches]
    r = oracle.chunk_update_ref(cfg, params, init_opt_state(), mbs, b1["head_w"], b1["head_norm_w"],
                                b1["head_norm_b"])
    return dict(losses=r["losses"], grads=[r["grads"]], h_out=r["runs"][-1]["h_out"],
                dh_out=r["runs"][-1]["dh_out"],
                masters=[{k: np.asarray(params[k], np.float64) for k in _trainable(shp)},
                         {k: r["params"][k] for k in _trainable(shp)}])


def _trainable(shp):
    return [k for k, _, _ in workload.param_specs(shp)]


# ------------------------------------------------------- bf16 parity cases
# Each bf16 parity case by name: its workload shape and the arguments of its
# inputs and objective.  The bf16 storage floor of every case is stored in
# tests/golden/bf16_floor.json under the same name.
def _cfg(name, **kw):
    return workload.get_config(name).with_(**kw)


GPT2 = workload.get_config("gpt2")
BF16_CASES = {
    "gpt2_reduced": dict(shape=GPT2.with_(batch=2, seq=128), seq_lens=[128, 90], drop=10),
    "gpt2_sgd_forward_kl": dict(shape=GPT2.with_(batch=2, seq=64), optimizer="sgd", lr=1e-2,
                                alpha=0.7, consis="forward"),
    "gpt2_full": dict(shape=GPT2),
    "1b_slice": dict(shape=_cfg("1b", n_layers=1, batch=1, seq=512)),
    "8b_slice": dict(shape=_cfg("8b", n_layers=1, batch=1, seq=256)),
    "8b_two_layers_sgd": dict(shape=_cfg("8b", n_layers=2, batch=1, seq=256), alpha=1.0,
                              optimizer="sgd", lr=1e-3),
    "gpt2_adapter": dict(shape=GPT2.with_(batch=2, seq=128, adapter_rank=64)),
    "1b_adapter": dict(shape=_cfg("1b", n_layers=1, batch=1, seq=512, adapter_rank=256)),
    "gpt2_lora": dict(shape=GPT2.with_(batch=2, seq=128, lora_rank=8), seq_lens=[128, 90], drop=10),
    "1b_lora": dict(shape=_cfg("1b", n_layers=1, batch=1, seq=512, lora_rank=16)),
    "8b_two_layers_lora": dict(shape=_cfg("8b", n_layers=2, batch=1, seq=256, lora_rank=8)),
    # the paper's LoRA setting (rank 4, scaling factor 16), stored padded to 8
    "1b_lora_r4": dict(shape=_cfg("1b", n_layers=1, batch=1, seq=512, lora_rank=4, lora_alpha=16.0),
                       steps=3, lr=1e-3),
    "1b_lora_window": dict(shape=_cfg("1b", n_layers=1, batch=1, seq=512, lora_rank=16),
                           window=(1, 6)),
    # confident readout: the head scaled so the largest logits are about 30
    # and every label is its row's most likely token (p_y mostly 0.5-0.95)
    "1b_confident_logits": dict(shape=_cfg("1b", n_layers=1, batch=1, seq=512), head_scale=5.0,
                                argmax_labels=True),
    # a token count off every tile and 32-row epilogue block (200 rows): the
    # epilogues' partial-block paths in bf16
    "1b_ragged": dict(shape=_cfg("1b", n_layers=1, batch=1, seq=200)),
}


def argmax_labels(shp, params, batch, **kw):
    """Labels set to each row's most likely token under the oracle's readout
    of h_out (inputs only: nothing here comes from the device)."""
    cfg = oracle_cfg(shp, **kw)
    h_out, fw = chunk_forward_ref(cfg, params, batch["h_in"], batch["seq_lens"], batch["pos_ids"])
    W = oracle.bf16_round(batch["head_w"]) if shp.dtype == "bf16" else batch["head_w"]
    z = oracle.head_logits_ref(h_out.reshape(-1, shp.d_model), W, shp.arch,
                               np.asarray(batch["head_norm_w"], np.float64),
                               None if batch["head_norm_b"] is None
                               else np.asarray(batch["head_norm_b"], np.float64), shp.norm_eps)
    return np.argmax(z, axis=1).astype(np.int32).reshape(batch["labels"].shape)


def case_inputs(name):
    """(shape, kwargs of the objective, params, batch or [batches]) of a
    named bf16 case."""
    c = dict(BF16_CASES[name])
    shp = c.pop("shape")
    steps = c.pop("steps", 1)
    window = c.pop("window", None)
    head_scale = c.pop("head_scale", None)
    amax = c.pop("argmax_labels", False)
    seq_lens = c.pop("seq_lens", None)
    drop = c.pop("drop", 0)
    kw = dict(alpha=c.pop("alpha", 0.5), consis=c.pop("consis", "reverse"),
              optimizer=c.pop("optimizer", "adamw"), lr=c.pop("lr", 1e-4), wd=c.pop("wd", 0.01))
    assert not c, c
    if window:  # two micro-batches with their own tokens, one parameter set
        params, b1 = make_inputs(shp, seed=0, tokens_seed=window[0])
        _, b2 = make_inputs(shp, seed=0, tokens_seed=window[1])
        for k in ("head_w", "head_norm_w", "head_norm_b"):
            b2[k] = b1[k]
        return shp, kw, steps, params, [b1, b2]
    params, batch = make_inputs(shp, seq_lens=seq_lens, drop=drop)
    if head_scale:
        hw = batch["head_w"].astype(np.float64) * head_scale
        batch["head_w"] = workload.gen.bf16_round_trip_input(hw.astype(np.float32)) \
            if shp.dtype == "bf16" else hw.astype(np.float32)
    if amax:
        batch["labels"] = argmax_labels(shp, params, batch, **kw)
    return shp, kw, steps, params, batch


def case_oracle(name, store_bf16=False, masters=True):
    """The oracle's result of a named bf16 case (and its inputs)."""
    shp, kw, steps, params, batch = case_inputs(name)
    if isinstance(batch, list):
        return oracle_window(shp, params, batch, store_bf16=store_bf16, **kw), (params, batch[0])
    return oracle_run(shp, params, batch, steps=steps, store_bf16=store_bf16, masters=masters,
                      **kw), (params, batch)
