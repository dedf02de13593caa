"""Benchmark: chunk-local update tokens/s on one MI355X, and MFMA utilisation.

One step = one whole zl_chunk_update (forward, local objective on the frozen
head, chunk-local backward, AdamW step) over one synthetic micro-batch whose
inputs are already resident in HBM.  Default workload: the Llama-3-8B-shaped
chunk (8 layers, d 4096, 32/8 heads x 128, MLP 14336, vocab 128256),
B = 4, S = 4096, bf16 with fp32 master weights, alpha = 0.5.

Prints one JSON line.  `roofline` covers the kernel with the largest share
of the step time (timed with HIP events on the launch stream inside the
timed steps); `cpu_baseline` times the fp64 oracle on a bounded slice of the
same workload on the host.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "chunk-local update tokens/sec on 1 MI355X; MFMA util % of bf16 peak"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16: 256 CU x 2.4 GHz x 4096 FLOP/clk/CU
PEAK_HBM_GBS = 8000.0


def algorithmic_flops(shp, T, S, alpha):
    """FLOPs the method must compute per update (no recompute counted):
    6 * P_lin * T for the chunk linears (forward, dgrad, wgrad); causal
    attention 2 * d_q * (S + 1) per token forward and twice that backward;
    head: readout of h_out, readout of h_in (alpha < 1), and the dgrad into
    h_out, 2 * d * V per token each (the head is frozen: no wgrad).
    With LoRA rank r the base linears are frozen: 4 * P_lin * T (no wgrad,
    and no data gradient of layer 0's QKV projection, which feeds only the
    detached input), plus per linear (in, out) 6 * r * (in + out) per token
    (x A^T and its B^T product forward; dy B, its A product, dA, dB
    backward; layer 0's QKV dx product excepted)."""
    d, hd, ff = shp.d_model, shp.head_dim, shp.d_ff
    dq, dkv = shp.n_heads * hd, shp.n_kv_heads * hd
    if shp.arch == "llama":
        p_lin = d * (dq + 2 * dkv) + dq * d + 3 * d * ff
        lins = [(d, dq), (d, dkv), (d, dkv), (dq, d), (d, ff), (d, ff), (ff, d)]
    else:
        p_lin = d * (dq + 2 * dkv) + dq * d + 2 * d * ff
        lins = [(d, dq + 2 * dkv), (dq, d), (d, ff), (ff, d)]
    lr = getattr(shp, "lora_rank", 0)
    if lr:
        nq = 3 if shp.arch == "llama" else 1
        lin = 4.0 * p_lin * T * shp.n_layers - 2.0 * T * d * (dq + 2 * dkv)
        lora = 6.0 * lr * T * shp.n_layers * sum(i + o for i, o in lins) - 2.0 * T * nq * lr * d
    else:
        lin = 6.0 * p_lin * T * shp.n_layers
    attn = 3.0 * 2.0 * dq * (S + 1) * T * shp.n_layers
    head = (3.0 if alpha < 1.0 else 2.0) * 2.0 * d * shp.vocab * T
    parts = dict(linear=lin, attention=attn, head=head)
    if lr:
        parts["lora"] = lora
    r = getattr(shp, "adapter_rank", 0)
    if r:  # readout adapter: 2 GEMMs forward, 4 backward (dU, dh, dW2, dW1)
        parts["adapter"] = 6.0 * 2.0 * d * r * T
    return sum(parts.values()), parts


def cpu_baseline(shp, alpha):
    """The oracle, as it stands, timed on a bounded slice of the workload:
    one update (forward, objective with the full head, chunk-local backward,
    AdamW) of one of the chunk's layers at full width, B = 1, S = 256.  The
    value is that slice's own tokens/s, labelled as a slice; it is not
    scaled to the whole chunk."""
    import numpy as np
    import oracle
    import workload
    from oracle.chunk import init_opt_state
    S = 256
    sl = shp.with_(n_layers=1, batch=1, seq=S)
    params = workload.init_params(workload.param_specs(sl), seed=0)
    batch = workload.make_batch(sl)
    cfg = oracle.OracleConfig.from_shape(sl, alpha=alpha)
    mb = dict(h_in=batch["h_in"], labels=batch["labels"])
    t0 = time.perf_counter()
    oracle.chunk_update_ref(cfg, params, init_opt_state(), [mb], batch["head_w"],
                            batch["head_norm_w"], batch["head_norm_b"])
    t_slice = time.perf_counter() - t0
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    threads = int(os.environ.get("OMP_NUM_THREADS", cores) or cores)
    try:
        blas = np.show_config(mode="dicts")["Build Dependencies"]["blas"]["name"]
    except Exception:  # numpy without the dict form
        blas = "unknown"
    return {"value": S / t_slice, "unit": "tokens/s", "cores": min(cores, threads), "kind": "oracle",
            "blas": blas, "slice": True,
            "sample": (f"slice: fp64 NumPy oracle, one update of 1 of the {shp.n_layers} layers at "
                       f"full width with the full head and AdamW, B=1 S={S}: {t_slice:.1f} s "
                       f"for {S} tokens; not scaled to the chunk")}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
GEMM_SOURCE = os.path.join(ROOT, "paper_2608_07974_amd", "csrc", "gemm.hip")


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed counter runs
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain-copy calibration), or None if
    none were taken for this kernel and workload or its source has changed
    since."""
    import hashlib
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        with open(GEMM_SOURCE, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
    except OSError:
        return None
    for r in rec.get("kernels", []):
        if r["kernel"] == kernel and r["workload"] == workload and r["source_sha256"] == sha:
            return r["hbm_bytes_per_launch"]
    return None


def copy_calibration(nbytes=1 << 30, reps=3):
    """A plain device-to-device copy of known size, for scaling the
    FETCH_SIZE / WRITE_SIZE counters (profiled separately), and the device's
    copy bandwidth (read + write bytes over the copy's event-timed duration,
    median of `reps`): the practical ceiling of the HBM-bound kernels."""
    import numpy as np
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        torch.cuda.synchronize()
        ms.append(a.elapsed_time(b))
    med = float(np.median(ms))
    print(json.dumps({"copy_calibration_bytes": nbytes, "reps": reps, "copy_ms": round(med, 4),
                      "copy_gbs": round(2 * nbytes / (med / 1e3) / 1e9, 1)}))


def gemm_compare(shape, reps=5):
    """One bf16 GEMM C[M, N] = A[M, K] B[N, K]^T (both operands K-major, the
    layout of the chunk's forward linears and head) with libzl's kernel and
    with torch.matmul (hipBLASLt), `reps` times each, event-timed: the
    reference for profiling the two kernels side by side."""
    import torch
    from paper_2608_07974_amd import zl
    M, N, K = (int(x) for x in shape.split(","))
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(0)
    A = torch.randn(M, K, device=dev, generator=g).bfloat16()
    B = torch.randn(N, K, device=dev, generator=g).bfloat16()
    C = torch.empty(M, N, device=dev)
    s = torch.cuda.current_stream().cuda_stream
    runs = {"libzl": lambda: zl.zl_kernel_gemm(M, N, K, A.data_ptr(), K, True, B.data_ptr(), K,
                                               True, C.data_ptr(), N, zl.ZL_BF16, s),
            "torch.matmul": lambda: torch.matmul(A, B.t())}
    out = {"gemm": [M, N, K]}
    for name, f in runs.items():
        f()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            f()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        out[name] = {"ms": round(ms, 4), "tflops": round(2.0 * M * N * K / ms / 1e9, 1)}
    print(json.dumps(out))


def pipeline_bench(args):
    """K chunks of `--config` chained as a stage pipeline on one GPU (one
    stream per stage, early forwarding, update window `--window`) against
    the same chunks run one after another on one stream.  One JSON line."""
    import numpy as np
    import torch

    import workload
    from paper_2608_07974_amd import zl
    from paper_2608_07974_amd.chunk import TorchChunk, config_from_shape
    from paper_2608_07974_amd.pipeline import Pipeline

    shp = workload.get_config(args.config)
    K, W = args.pipeline, args.window
    B, S, T = shp.batch, shp.seq, shp.batch * shp.seq
    dev = torch.device("cuda:0")
    torch.manual_seed(0)
    cfg = config_from_shape(shp, alpha=args.alpha)
    pipe = Pipeline([cfg] * K, window=W, depth=2, device=dev)
    head = (pipe.chunks[0].head_w, pipe.chunks[0].head_norm_w, pipe.chunks[0].head_norm_b)
    head[0].normal_(0.0, 0.02)
    for ch in pipe.chunks:
        ch.master.normal_(0.0, 0.02)
        for t in ch.layout:
            v = ch.view(ch.master, f"L{t['layer']}.{t['name']}")
            if t["name"].startswith("ln") and t["name"].endswith("_w"):
                v.fill_(1.0)
            elif len(t["shape"]) == 1:
                v.zero_()
        zl.zl_refresh_shadow(ch.handle, torch.cuda.current_stream().cuda_stream)
    tokens = workload.zipf_tokens(B, S, shp.vocab, seed=1) if shp.vocab > 256 else \
        workload.uniform_tokens(B, S, shp.vocab, seed=1)
    labels = torch.tensor(workload.labels_from_tokens(tokens), device=dev)
    table = torch.empty(shp.vocab, shp.d_model, dtype=pipe.dtype, device=dev).normal_(0.0, 0.02)
    h0 = table[torch.tensor(tokens, device=dev, dtype=torch.long)].contiguous()
    del table
    torch.cuda.synchronize()

    def timed(run, n):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run(n)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / n

    losses = torch.zeros(K, dtype=torch.float32, device=dev)

    def run_pipe(n):
        for _ in range(n):
            pipe.submit(h0, labels, losses=losses)
        pipe.sync()

    run_pipe(args.warmup * W)
    t_pipe = timed(run_pipe, args.steps * W)
    # the same chunks, sequentially on one stream (no early forwarding)
    outs = [torch.empty_like(h0) for _ in range(K)]
    count = [0]

    def run_seq(n):
        for _ in range(n):
            h = h0
            i = count[0]
            for k, ch in enumerate(pipe.chunks):
                h = ch.forward(h, h_out=outs[k])
                ch.objective(labels)
                ch.backward(1.0 / W, 0 if i % W == 0 else 1)
                if i % W == W - 1:
                    ch.step()
            count[0] += 1

    run_seq(args.warmup * W)
    t_seq = timed(run_seq, args.steps * W)
    flops, _ = algorithmic_flops(shp, T, S, args.alpha)
    out = {"metric": "stage-pipeline tokens/sec on 1 MI355X (K chunks, early forwarding)",
           "value": round(T / t_pipe, 1), "unit": "tokens/s", "n_gpus": 1,
           "ms_per_microbatch": round(t_pipe * 1e3, 3),
           "sequential_tokens_per_s": round(T / t_seq, 1),
           "sequential_ms_per_microbatch": round(t_seq * 1e3, 3),
           "speedup_vs_sequential": round(t_seq / t_pipe, 4),
           "mfma_util_pct": round(100.0 * K * flops / t_pipe / (PEAK_BF16_TFLOPS * 1e12), 2),
           "config": {"workload": f"{K} x {shp.name} chunks ({K * shp.n_layers} layers)",
                      "global_batch": B, "seq_len": S, "window": W, "depth": 2,
                      "alpha": args.alpha},
           "steps": args.steps * W, "warmup": args.warmup * W, "dtype": "bf16",
           "data": "synthetic (Zipf(1.1) token ids, random-init N(0,0.02) weights)"}
    print(json.dumps(out))
    pipe.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="8b")
    ap.add_argument("--alpha", type=float, default=0.5)
    ap.add_argument("--adapter-rank", type=int, default=0,
                    help="readout adapter width r (0 = static head)")
    ap.add_argument("--lora-rank", type=int, default=0,
                    help="LoRA rank r (0 = the whole chunk is trained)")
    ap.add_argument("--lora-alpha", type=float, default=16.0, help="LoRA scale s = alpha / r")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-json", default=None, help="write the per-kernel profile here")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration) and exit")
    ap.add_argument("--gemm-compare", default=None,
                    help="M,N,K: time one K-major bf16 GEMM with libzl and with torch.matmul")
    ap.add_argument("--pipeline", type=int, default=0,
                    help="K > 0: time K chunks as a stage pipeline instead (one JSON line)")
    ap.add_argument("--window", type=int, default=1, help="update window (with --pipeline)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gemm_compare:
        gemm_compare(args.gemm_compare, reps=args.steps)
        return
    if args.pipeline > 0:
        if args.gpus != 1:
            print("bench.py: --pipeline runs on one GPU", file=sys.stderr)
            sys.exit(2)
        pipeline_bench(args)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: this build runs one chunk on one GPU; --gpus {args.gpus} "
              f"(WORLD_SIZE={world}) is not supported. A K-GPU pipeline would run one "
              "chunk per GPU and exchange only hidden states.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workload
    from paper_2608_07974_amd import zl
    from paper_2608_07974_amd.chunk import TorchChunk, config_from_shape, current_stream

    shp = workload.get_config(args.config, adapter_rank=args.adapter_rank,
                              lora_rank=args.lora_rank, lora_alpha=args.lora_alpha)
    B, S = shp.batch, shp.seq
    T = B * S
    dev = torch.device("cuda:0")
    torch.manual_seed(0)
    cfg = config_from_shape(shp, alpha=args.alpha)
    ch = TorchChunk(cfg, device=dev)
    # random-init weights of the architecture, on device: N(0, 0.02) linears
    # (and LoRA factors), norm weights 1, biases 0; frozen head N(0, 0.02),
    # head norm 1 / 0
    for buf, layout in ((ch.master, ch.layout), (ch.base_master, ch.base_layout)):
        if buf is None:
            continue
        buf.normal_(0.0, 0.02)
        for t in layout:
            v = buf[t["offset"]: t["offset"] + t["numel"]]
            if t["name"].startswith("ln") and t["name"].endswith("_w"):
                v.fill_(1.0)
            elif len(t["shape"]) == 1:
                v.zero_()
    ch.head_w.normal_(0.0, 0.02)
    zl.zl_refresh_shadow(ch.handle, current_stream())
    tokens = workload.zipf_tokens(B, S, shp.vocab, seed=1) if shp.vocab > 256 else \
        workload.uniform_tokens(B, S, shp.vocab, seed=1)
    labels = torch.tensor(workload.labels_from_tokens(tokens), device=dev)
    table = torch.empty(shp.vocab, shp.d_model, dtype=ch.dtype, device=dev).normal_(0.0, 0.02)
    h_in = table[torch.tensor(tokens, device=dev, dtype=torch.long)].contiguous()
    if shp.arch == "gpt2":
        pos = torch.empty(S, shp.d_model, dtype=ch.dtype, device=dev).normal_(0.0, 0.02)
        h_in = (h_in + pos[None]).contiguous()
    del table
    h_out = torch.empty_like(h_in)
    torch.cuda.synchronize()

    loss_first = None
    for i in range(args.warmup):
        ch.update(h_in, labels, h_out=h_out)
        if i == 0:
            loss_first = float(ch.loss.item())   # loss of the initial weights
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    zl.zl_profile_begin(ch.handle, 1024 * max(1, args.steps))
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(args.steps):
        ch.update(h_in, labels, h_out=h_out)
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    prof = zl.zl_profile_end(ch.handle, 512)
    step_ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    total_ms = ev[0].elapsed_time(ev[-1])
    loss = float(ch.loss.item())
    med = float(np.median(step_ms))

    flops, parts = algorithmic_flops(shp, T, S, args.alpha)
    tokens_s = T / (med / 1e3)
    mfma_pct = 100.0 * flops / (med / 1e3) / (PEAK_BF16_TFLOPS * 1e12)

    # dominant kernel by summed time over the timed steps
    prof.sort(key=lambda e: -e["total_ms"])
    dom = prof[0]
    per_launch_ms = dom["total_ms"] / dom["launches"]
    if dom["flops"] > 0:
        achieved = dom["flops"] / (dom["total_ms"] / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None}
    else:
        achieved = dom["bytes"] / (dom["total_ms"] / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None}
    roof["traffic"] = measured_traffic(dom["name"], shp.name)
    roof["kernel"] = dom["name"]
    roof["launches_per_step"] = dom["launches"] / args.steps
    roof["avg_launch_ms"] = round(per_launch_ms, 4)
    roof["share_of_step"] = round(dom["total_ms"] / total_ms, 4)

    kernels = []
    for e in prof:
        k = {"name": e["name"], "ms_per_step": round(e["total_ms"] / args.steps, 3),
             "launches_per_step": e["launches"] / args.steps}
        if e["flops"] > 0:
            k["tflops"] = round(e["flops"] / (e["total_ms"] / 1e3) / 1e12, 1)
        if e["bytes"] > 0:
            k["gbs"] = round(e["bytes"] / (e["total_ms"] / 1e3) / 1e9, 1)
        kernels.append(k)
    if args.profile_json:
        with open(args.profile_json, "w") as f:
            json.dump(dict(kernels=kernels, step_ms=step_ms), f, indent=1)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(shp, args.alpha)

    out = {
        "metric": METRIC, "value": round(tokens_s, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(med, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (Zipf(1.1) token ids, random-init N(0,0.02) weights)",
        "config": {"workload": f"{shp.name}: llama-3-8B-shaped chunk of {shp.n_layers} layers, "
                               f"d={shp.d_model}, heads {shp.n_heads}/{shp.n_kv_heads}x"
                               f"{shp.head_dim}, ff={shp.d_ff}, vocab={shp.vocab}"
                               if shp.name == "8b" else shp.name,
                   "global_batch": B, "seq_len": S, "tokens_per_step": T,
                   "alpha": args.alpha, "optimizer": "adamw", "parallelism": "none (1 GPU)",
                   "adapter_rank": shp.adapter_rank, "lora_rank": shp.lora_rank},
        "mfma_util_pct": round(mfma_pct, 2),
        "device": dict(zl.zl_device_info(0), peak_bf16_tflops_used=PEAK_BF16_TFLOPS),
        "algorithmic_tflop_per_step": round(flops / 1e12, 2),
        "flop_split": {k: round(v / flops, 4) for k, v in parts.items()},
        "ms_per_step_min": round(min(step_ms), 3),
        "loss_initial_and_last": [None if loss_first is None else round(loss_first, 4), round(loss, 4)],
        "roofline": roof,
        "kernels": kernels[:16],
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))
    ch.close()


if __name__ == "__main__":
    main()
