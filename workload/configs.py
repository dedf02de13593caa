"""The five chunk workloads and the per-layer parameter naming.

Shapes follow the paper's setting of a decoder split into chunks of
consecutive layers (Sec. II.A, Eq. (1)); the concrete widths are the
GPT-2-small, Llama-1B and Llama-3-8B shapes plus a tiny parity model.
"""
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class ChunkShape:
    name: str
    arch: str            # "llama" (RMSNorm, RoPE, SwiGLU) or "gpt2" (LayerNorm, GELU, biases)
    n_layers: int        # layers in the chunk
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    batch: int
    seq: int
    dtype: str           # "f32" or "bf16" (bf16 compute, fp32 master/grad/state)
    rope_theta: float
    n_chunks: int        # chunks the whole model is split into
    norm_eps: float = 1e-5
    adapter_rank: int = 0  # readout adapter width r (0 = static head only)
    lora_rank: int = 0     # LoRA rank (0 = the whole chunk is trained)
    lora_alpha: float = 16.0  # LoRA scale s = lora_alpha / lora_rank

    @property
    def tokens(self):
        return self.batch * self.seq

    def with_(self, **kw):
        return replace(self, **kw)


CONFIGS = {
    "tiny": ChunkShape("tiny", "llama", 2, 64, 4, 4, 16, 256, 256, 4, 32, "f32", 1e4, 2),
    "gpt2": ChunkShape("gpt2", "gpt2", 3, 768, 12, 12, 64, 3072, 50257, 8, 512, "bf16", 0.0, 4),
    "1b": ChunkShape("1b", "llama", 4, 2048, 32, 8, 64, 8192, 128256, 4, 2048, "bf16", 5e5, 4),
    "1b-long": ChunkShape("1b-long", "llama", 4, 2048, 32, 8, 64, 8192, 128256, 1, 8192, "bf16", 5e5, 4),
    "8b": ChunkShape("8b", "llama", 8, 4096, 32, 8, 128, 14336, 128256, 4, 4096, "bf16", 5e5, 4),
}


def get_config(name, **overrides):
    cfg = CONFIGS[name]
    return cfg.with_(**overrides) if overrides else cfg


def base_specs(cfg):
    """The chunk's layer tensors, in order: list of (key, shape, kind).

    key is "L{layer}.{name}"; kind is one of "norm_w", "norm_b", "weight",
    "bias".  Linear weights are [out, in] (y = x W^T, as in Eq. (2)).  With
    LoRA these are the frozen base of the chunk.
    """
    d, hd = cfg.d_model, cfg.head_dim
    dq, dkv, ff = cfg.n_heads * hd, cfg.n_kv_heads * hd, cfg.d_ff
    out = []
    for l in range(cfg.n_layers):
        p = f"L{l}."
        if cfg.arch == "llama":
            out += [
                (p + "ln1_w", (d,), "norm_w"),
                (p + "wq", (dq, d), "weight"),
                (p + "wk", (dkv, d), "weight"),
                (p + "wv", (dkv, d), "weight"),
                (p + "wo", (d, dq), "weight"),
                (p + "ln2_w", (d,), "norm_w"),
                (p + "wg", (ff, d), "weight"),
                (p + "wu", (ff, d), "weight"),
                (p + "wd", (d, ff), "weight"),
            ]
        elif cfg.arch == "gpt2":
            out += [
                (p + "ln1_w", (d,), "norm_w"),
                (p + "ln1_b", (d,), "norm_b"),
                (p + "wqkv", (dq + 2 * dkv, d), "weight"),
                (p + "bqkv", (dq + 2 * dkv,), "bias"),
                (p + "wo", (d, dq), "weight"),
                (p + "bo", (d,), "bias"),
                (p + "ln2_w", (d,), "norm_w"),
                (p + "ln2_b", (d,), "norm_b"),
                (p + "wfc", (ff, d), "weight"),
                (p + "bfc", (ff,), "bias"),
                (p + "wproj", (d, ff), "weight"),
                (p + "bproj", (d,), "bias"),
            ]
        else:
            raise ValueError(cfg.arch)
    return out


LORA_TARGETS = {"llama": ("wq", "wk", "wv", "wo", "wg", "wu", "wd"),
                "gpt2": ("wqkv", "wo", "wfc", "wproj")}


def param_specs(cfg):
    """The chunk's trainable tensors, in order: list of (key, shape, kind).

    Without LoRA: base_specs.  With LoRA (Eq. (6), rank r): per layer the
    factors A [r, in] ("{name}_la", kind "lora_a") and B [out, r]
    ("{name}_lb", kind "lora_b", zero-initialised so training starts from
    the base model) of every linear in LORA_TARGETS, with the A factors of
    q/k/v and of g/u adjacent.  Then, with adapter_rank r > 0, the readout
    adapter as a pseudo-layer after the chunk's layers: ad_w1 [r, d] and
    ad_w2 [d, r] (kind "adapter_out", zero-initialised: identity adapter).
    """
    d = cfg.d_model
    if not cfg.lora_rank:
        out = base_specs(cfg)
    else:
        shapes = {k[len("L0."):]: s for k, s, _ in base_specs(cfg.with_(n_layers=1))}
        r = cfg.lora_rank
        if cfg.arch == "llama":
            order = [("wq", "a"), ("wk", "a"), ("wv", "a"), ("wq", "b"), ("wk", "b"), ("wv", "b"),
                     ("wo", "a"), ("wo", "b"), ("wg", "a"), ("wu", "a"), ("wg", "b"), ("wu", "b"),
                     ("wd", "a"), ("wd", "b")]
        else:
            order = [(n, f) for n in LORA_TARGETS["gpt2"] for f in ("a", "b")]
        out = []
        for l in range(cfg.n_layers):
            for name, f in order:
                o, i = shapes[name]
                out.append((f"L{l}.{name}_l{f}", (r, i) if f == "a" else (o, r), "lora_" + f))
    if cfg.adapter_rank:
        # readout adapter h' = h + gelu(h W1^T) W2^T before the frozen head,
        # listed as one extra pseudo-layer after the chunk's layers
        p = f"L{cfg.n_layers}."
        out += [(p + "ad_w1", (cfg.adapter_rank, d), "weight"),
                (p + "ad_w2", (d, cfg.adapter_rank), "adapter_out")]
    return out
