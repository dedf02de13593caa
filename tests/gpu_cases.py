"""Builders shared by the GPU tests (not collected by pytest).

Every GPU result comes from libzl through the C ABI; every expected value
comes from oracle/ on the same seeded inputs (workload/)."""
import numpy as np

import oracle
import workload
from oracle.chunk import init_opt_state

ARCH = {"llama": 0, "gpt2": 1}


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def zl_cfg(shp, **kw):
    from paper_2608_07974_amd.chunk import config_from_shape
    return config_from_shape(shp, **kw)


def oracle_cfg(shp, alpha=0.5, consis="reverse", optimizer="adamw", lr=1e-4, wd=0.01):
    return oracle.OracleConfig.from_shape(shp, alpha=alpha, consis=consis, optimizer=optimizer,
                                          lr=lr, weight_decay=wd)


def make_inputs(shp, seed=0, stress=True, seq_lens=None, drop=0):
    """Seeded parameters and batch; parity cases perturb norms/biases and use
    the stress scale so the consistency term is exercised."""
    params = workload.init_params(workload.param_specs(shp), seed=seed, perturb=True, stress=stress)
    if getattr(shp, "lora_rank", 0):  # the frozen base of a LoRA chunk
        params.update(workload.init_params(workload.base_specs(shp), seed=seed + 50, perturb=True,
                                           stress=stress))
    batch = workload.make_batch(shp, stress=stress, seq_lens=seq_lens, perturb_head=True)
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
