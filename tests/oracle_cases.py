"""Small shared builders for the oracle CPU tests (not collected by pytest)."""
import numpy as np

import workload
from oracle import OracleConfig
from workload.configs import ChunkShape


def tiny_shape(arch="llama", gqa=False, L=2, d=8, hd=4, ff=16, V=11, B=2, S=5, adapter_rank=0,
               lora_rank=0, lora_alpha=16.0):
    hq, hkv = (4, 2) if gqa else (2, 2)
    return ChunkShape("fd", arch, L, d, hq, hkv, hd, ff, V, B, S, "f32",
                      1e4 if arch == "llama" else 0.0, 2, adapter_rank=adapter_rank,
                      lora_rank=lora_rank, lora_alpha=lora_alpha)


def tiny_case(arch="llama", gqa=False, alpha=0.5, consis="reverse", seed=0, std=0.3,
              head_std=0.5, pad=True, drop_labels=True, **shape_kw):
    shp = tiny_shape(arch, gqa, **shape_kw)
    cfg = OracleConfig.from_shape(shp, alpha=alpha, consis=consis)
    specs = workload.param_specs(shp)
    P = {k: v.astype(np.float64) for k, v in
         workload.init_params(specs, seed=seed, std=std, perturb=True).items()}
    trainable = list(P)
    if shp.lora_rank:  # the frozen base joins the forward's parameters
        base = workload.init_params(workload.base_specs(shp), seed=seed + 50, std=std, perturb=True)
        P.update({k: v.astype(np.float64) for k, v in base.items()})
    rng = np.random.default_rng(seed + 100)
    B, S, d, V = shp.batch, shp.seq, shp.d_model, shp.vocab
    tok = rng.integers(0, V, size=(B, S)).astype(np.int32)
    lens = np.array([S, max(1, S - 2)] + [S] * (B - 2), np.int32)[:B] if pad else np.full(B, S, np.int32)
    labels = workload.labels_from_tokens(tok, lens)
    if drop_labels:
        labels[0, 0] = -100  # a prompt position
    h_in = rng.standard_normal((B, S, d))
    head_w = rng.standard_normal((V, d)) * head_std
    hn_w = 1.0 + 0.1 * rng.standard_normal(d)
    hn_b = 0.05 * rng.standard_normal(d) if arch == "gpt2" else None
    pos = np.tile(np.arange(S, dtype=np.int32), (B, 1))
    return dict(cfg=cfg, shape=shp, P=P, h_in=h_in, labels=labels, seq_lens=lens, pos_ids=pos,
                head_w=head_w, hn_w=hn_w, hn_b=hn_b, trainable=trainable)


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))
