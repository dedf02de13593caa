"""Seeded generators: token ids, labels, embeddings, weights.

Token ids: uniform for the tiny model, otherwise Zipf(s=1.1) truncated to the
vocabulary and sampled by inverse CDF.  Labels are the next token (the head
predicts the next token, Sec. II.A after Eq. (2)); positions with no next
token inside the valid length are -100 (outside the labelled set).
"""
import numpy as np

IGNORE = -100


def uniform_tokens(batch, seq, vocab, seed=1):
    rng = np.random.default_rng(seed)
    return rng.integers(0, vocab, size=(batch, seq), dtype=np.int64).astype(np.int32)


def zipf_tokens(batch, seq, vocab, s=1.1, seed=1):
    """P(rank r) proportional to r^-s for r = 1..vocab; id = r - 1."""
    rng = np.random.default_rng(seed)
    w = np.arange(1, vocab + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = rng.random(batch * seq)
    ids = np.searchsorted(cdf, u, side="right")
    ids = np.minimum(ids, vocab - 1)
    return ids.reshape(batch, seq).astype(np.int32)


def labels_from_tokens(tokens, seq_lens=None):
    """y[b, i] = x[b, i+1] when i+1 < seq_len[b], else -100."""
    B, S = tokens.shape
    lens = np.full(B, S, np.int32) if seq_lens is None else np.asarray(seq_lens, np.int32)
    y = np.full((B, S), IGNORE, np.int32)
    for b in range(B):
        n = int(lens[b])
        if n > 1:
            y[b, : n - 1] = tokens[b, 1:n]
    return y


def embed_tokens(tokens, table, pos_table=None):
    """h_0 = E(x): a row gather (plus learned positions for GPT-2)."""
    h = table[tokens]
    if pos_table is not None:
        h = h + pos_table[None, : tokens.shape[1]]
    return h


def bf16_round_trip_input(x):
    """Round an fp32 array to bf16 (nearest-even) and back, as plain bit work.

    Used to make the fp32 host copy of an input that is handed to the device
    in bf16, so both sides start from identical values.
    """
    a = np.ascontiguousarray(x, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    return np.where(np.isnan(a), a, out)


def init_params(specs, seed=0, std=0.02, perturb=False, stress=False):
    """N(0, std) linears; norm weights 1 and biases 0.

    LoRA factors: A ~ N(0, std), B = 0 (the chunk starts as its base).
    perturb=True draws norm weights 1 + N(0, 0.1), biases N(0, 0.02), and a
    non-zero readout-adapter output projection and LoRA B, so every term of
    the update is exercised (unperturbed, those are zero: identity adapter,
    base model);
    stress=True widens the output projections (wo, wd, wproj) to
    N(0, 0.2 * sqrt(64 / fan_in)), i.e. 0.2 at fan-in 64, so their
    contribution keeps the same scale at every width.
    """
    rng = np.random.default_rng(seed)
    out = {}
    for key, shape, kind in specs:
        name = key.split(".", 1)[1]
        if kind == "weight":
            s = 0.2 * np.sqrt(64.0 / shape[1]) if (stress and name in ("wo", "wd", "wproj")) else std
            out[key] = (rng.standard_normal(shape) * s).astype(np.float32)
        elif kind == "lora_a":
            out[key] = (rng.standard_normal(shape) * std).astype(np.float32)
        elif kind in ("adapter_out", "lora_b"):
            # zero (identity adapter / base model) unless perturbed, so
            # parity exercises it
            sd = 0.2 * np.sqrt(64.0 / shape[1]) if (stress and kind == "adapter_out") else std
            out[key] = (rng.standard_normal(shape) * sd if perturb
                        else np.zeros(shape)).astype(np.float32)
        elif kind == "norm_w":
            out[key] = (1.0 + (rng.standard_normal(shape) * 0.1 if perturb else 0.0)) * np.ones(shape, np.float32)
            out[key] = out[key].astype(np.float32)
        else:  # norm_b, bias
            out[key] = (rng.standard_normal(shape) * 0.02 if perturb else np.zeros(shape)).astype(np.float32)
    return out


def make_batch(cfg, seed_tokens=1, seed_embed=2, seed_head=3, stress=False,
               seq_lens=None, batch=None, seq=None, perturb_head=False):
    """Everything a chunk update of `cfg` needs besides its own parameters.

    Returns dict with tokens, labels, seq_lens, pos_ids, h_in (fp32; already
    bf16-representable when cfg.dtype == "bf16"), head_w [V, d] (same),
    head_norm_w, head_norm_b (None for llama).
    """
    B = batch or cfg.batch
    S = seq or cfg.seq
    if cfg.name == "tiny" or cfg.vocab <= 256:
        tok = uniform_tokens(B, S, cfg.vocab, seed=seed_tokens)
    else:
        tok = zipf_tokens(B, S, cfg.vocab, seed=seed_tokens)
    lens = np.full(B, S, np.int32) if seq_lens is None else np.asarray(seq_lens, np.int32)
    labels = labels_from_tokens(tok, lens)
    rng_e = np.random.default_rng(seed_embed)
    table = (rng_e.standard_normal((cfg.vocab, cfg.d_model)) * 0.02).astype(np.float32)
    pos_table = None
    if cfg.arch == "gpt2":
        pos_table = (rng_e.standard_normal((S, cfg.d_model)) * 0.02).astype(np.float32)
    h_in = embed_tokens(tok, table, pos_table).astype(np.float32)
    rng_h = np.random.default_rng(seed_head)
    # stress: head logits with std about 1.6 at any width (0.2 at d = 64)
    head_std = 0.2 * np.sqrt(64.0 / cfg.d_model) if stress else 0.02
    head_w = (rng_h.standard_normal((cfg.vocab, cfg.d_model)) * head_std).astype(np.float32)
    if perturb_head:
        hn_w = (1.0 + 0.1 * rng_h.standard_normal(cfg.d_model)).astype(np.float32)
        hn_b = (0.02 * rng_h.standard_normal(cfg.d_model)).astype(np.float32) if cfg.arch == "gpt2" else None
    else:
        hn_w = np.ones(cfg.d_model, np.float32)
        hn_b = np.zeros(cfg.d_model, np.float32) if cfg.arch == "gpt2" else None
    if cfg.dtype == "bf16":
        h_in = bf16_round_trip_input(h_in)
        head_w = bf16_round_trip_input(head_w)
    pos = np.tile(np.arange(S, dtype=np.int32), (B, 1))
    return dict(tokens=tok, labels=labels, seq_lens=lens, pos_ids=pos, h_in=h_in,
                head_w=head_w, head_norm_w=hn_w, head_norm_b=hn_b, embed_table=table)
