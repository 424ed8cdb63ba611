"""Benchmark: one Llama-style decoder block, forward + backward, on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config 3b] [--no-cpu-baseline]
    python bench.py --config 3b_stack [--no-recompute]     (the whole 28-block model)

A step is one ls_block_fwd_bwd call (RMSNorm, QKV + RoPE, causal GQA flash
attention, output projection, RMSNorm, SwiGLU MLP, and the whole backward with
all weight gradients accumulated in fp32) on the Llama-3.2-3B-shaped block at
batch 4 x seq 2048 with seeded synthetic bf16 inputs already resident in HBM.
Prints one JSON line (the last line of stdout).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decoder-block fwd+bwd TFLOP/s and MFU (bf16), 3B shape seq 2048, 1 MI355X"  # the default --config 3b
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 matrix peak (256 CUs x 4096 FLOP/clk x 2.4 GHz)
PEAK_HBM_GBS = 8000.0
STACK_DOMINANT = "gate/up projection"  # the stack's roofline launch: the largest product of each block
COPY_BYTES = 1 << 30  # size of the plain device copy used to calibrate the HBM byte counters


def log(*a):
    print(*a, file=sys.stderr, flush=True)


LAUNCH_DESC = {
    "qkv projection": "bf16 MFMA GEMM [T,H]x[H,Dq+2Dkv] + fused RoPE",
    "output projection": "bf16 MFMA GEMM [T,Dq]x[Dq,H] + fused residual",
    "gate/up projection": "bf16 MFMA GEMM [T,H]x[H,2I] + fused SwiGLU",
    "down projection": "bf16 MFMA GEMM [T,I]x[I,H] + fused residual",
    "dact": "bf16 MFMA GEMM [T,H]x[H,I] + fused SwiGLU backward",
    "dWd": "bf16 MFMA GEMM [H,T]x[T,I], fp32 accumulate",
    "dh2": "bf16 MFMA GEMM [T,2I]x[2I,H] (input gradient of the gate/up projection)",
    "dWg/dWu": "bf16 MFMA GEMM [2I,T]x[T,H], fp32 accumulate",
    "dO": "bf16 MFMA GEMM [T,H]x[H,Dq]",
    "dWo": "bf16 MFMA GEMM [H,T]x[T,Dq], fp32 accumulate",
    "dh1": "bf16 MFMA GEMM [T,Dq+2Dkv]x[Dq+2Dkv,H]",
    "dWqkv": "bf16 MFMA GEMM [Dq+2Dkv,T]x[T,H], fp32 accumulate",
    "attention fwd": "causal GQA flash attention forward (bf16 MFMA)",
    "attention bwd": "causal GQA flash attention backward (bf16 MFMA)",
}


def traffic_key(label: str, config: str) -> str:
    return f"{label.replace('/', '_').replace(' ', '_')}_{config}"


def launch_traffic(label: str, config: str):
    """HBM bytes per launch of a labelled launch from the committed counter
    runs, or None when there are none or the kernel sources changed since."""
    from paper_2510_02483_amd import profiling

    path = profiling.TRAFFIC_JSON
    if not os.path.exists(path):
        return None
    with open(path) as f:
        entry = json.load(f).get(traffic_key(label, config))
    if not entry or entry.get("sources_hash") != profiling.sources_hash():
        return None
    return entry["traffic_bytes"]


def launch_breakdown(step_fn, labels, steps: int):
    """Mean duration (ms) and launches per step of every labelled launch,
    from HIP events the library records around it, over `steps` untimed steps
    per label."""
    import torch

    from paper_2510_02483_amd import lib

    out = {}
    for label in labels:
        lib.ls_timing_begin(label, 8 * steps)
        for _ in range(steps):
            step_fn()
        torch.cuda.synchronize()
        n, ms = lib.ls_timing_end()
        if n:
            out[label] = (n // steps, ms)
    return out


def calibrate_copy(iters: int = 5):
    """A plain device copy of COPY_BYTES (read once, written once) for the
    counter calibration run."""
    import torch

    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(iters):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "iters": iters}), flush=True)


def cpu_baseline(c, sequences: int):
    """The fp64 oracle on a bounded sample of the workload: its first
    `sequences` sequences (the block treats sequences independently)."""
    import numpy as np  # noqa: F401
    from threadpoolctl import threadpool_info

    from oracle import block as ob
    from paper_2510_02483_amd import flops, inputs

    n = min(sequences, c.batch)
    sample = c.with_(batch=n)
    host = inputs.make_inputs(c)
    f = inputs.to_f64({k: (v[:n] if k in ("x", "dy") else v) for k, v in host.items()})
    w = {k: f[k] for k in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm", "mlp_norm")}
    t0 = time.perf_counter()
    ob.block_fwd_bwd(f["x"], w, f["dy"], n_q_heads=c.n_q_heads, n_kv_heads=c.n_kv_heads,
                     rope_theta=c.rope_theta, eps=c.rms_eps)
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    return {"value": flops.block_fwd_bwd_flops(sample) / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{n} of {c.batch} sequences ({n * c.seq} tokens) of the same block, fp64 numpy oracle "
                      f"(BLAS matmuls), {dt:.1f} s wall",
            "host": host_record()}


def host_record() -> dict:
    """The CPU the oracle ran on: logical CPUs visible to this process, the
    machine's count and the model name."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count(), "cpu_model": model}


def kernel_only(args):
    """Time one kernel family through the C ABI on seeded inputs (for
    per-kernel counters): a plain bf16 product C = A B^T of --shape M,N,K, or
    causal attention forward + backward at the configuration's shape."""
    import torch

    from paper_2510_02483_amd import configs, flops, lib

    g = torch.Generator(device="cpu").manual_seed(1234)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, n):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        start.record()
        for _ in range(n):
            fn()
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / n

    if args.kernel in ("gemm_nt", "torch_nt"):
        M, N, K = (int(v) for v in args.shape.split(","))
        A = torch.randn(M, K, generator=g).to(torch.bfloat16).cuda()
        B = torch.randn(N, K, generator=g).to(torch.bfloat16).cuda()
        C = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        if args.kernel == "gemm_nt":
            fn = lambda: lib.ls_gemm_nt(A, B, C)  # noqa: E731
        else:  # yardstick only: the vendor library's product of the same shape, timed, never part of the path
            fn = lambda: torch.mm(A, B.t(), out=C)  # noqa: E731
        ms = timed(fn, args.steps)
        out = {"kernel": args.kernel, "shape": [M, N, K], "ms": round(ms, 4),
               "tflops": round(2.0 * M * N * K / (ms * 1e-3) / 1e12, 2)}
    else:
        c = configs.PRESETS[args.config]
        T, Dq, Dkv = c.tokens, c.dq, c.dkv
        qkv = torch.randn(T, Dq + 2 * Dkv, generator=g).to(torch.bfloat16).cuda()
        do = torch.randn(T, Dq, generator=g).to(torch.bfloat16).cuda()
        o = torch.empty(T, Dq, dtype=torch.bfloat16, device="cuda")
        lse = torch.empty(c.batch, c.n_q_heads, c.seq, dtype=torch.float32, device="cuda")
        dqkv = torch.empty_like(qkv)
        ws = torch.empty(lib.ls_attn_core_bwd_workspace(c), dtype=torch.uint8, device="cuda")
        fwd = timed(lambda: lib.ls_attn_core_fwd(c, qkv, o, lse), args.steps)
        bwd = timed(lambda: lib.ls_attn_core_bwd(c, qkv, o, lse, do, dqkv, ws), args.steps)
        fl = flops.attention_fwd_flops(c)
        out = {"kernel": "attention", "config": c.name, "fwd_ms": round(fwd, 4), "bwd_ms": round(bwd, 4),
               "fwd_tflops": round(fl / (fwd * 1e-3) / 1e12, 2), "bwd_tflops_model": round(2 * fl / (bwd * 1e-3) / 1e12, 2)}
    print(json.dumps(out), flush=True)


WORKLOAD_NAMES = {"3b": "Llama-3.2-3B-shaped", "3b_8k": "Llama-3.2-3B-shaped", "30b": "Llama-30B-shaped (52 x 128 heads)",
                  "paper_3b": "Table-1 3B-shaped (hidden 2048, 16q/2kv, SwiGLU 11008)", "tiny": "tiny"}
ADAMW_BYTES_PER_PARAM = 34  # norm pass: read the fp32 gradient (4); update: read 16, write 14


def energy_of(step_fn, tokens_per_step: int, args):
    """GPU energy of repeated steps over about --energy-seconds (None figures
    when the energy counter cannot be read)."""
    import torch

    from paper_2510_02483_amd import energy

    if args.energy_seconds <= 0:
        return None
    meter = energy.EnergyMeter()

    def one():
        step_fn()
        torch.cuda.synchronize()

    calls, secs, joules, sclk = meter.measure(one, args.energy_seconds)
    out = energy.report(calls, secs, joules, tokens_per_step)
    out["sclk_mhz"] = sclk  # mean shader clock over the same loop
    if meter.error:
        out["error"] = meter.error
    return out


def stack_bench(args):
    """--config 3b_stack: the whole model (28 blocks, tied embedding and LM
    head, cross-entropy) forward + backward per step, inputs drawn on the GPU."""
    import torch

    from paper_2510_02483_amd import configs, flops, inputs, lib

    sc = configs.STACK_PRESETS[args.config].with_(recompute=not args.no_recompute)
    log(f"config {sc}")
    st = lib.Stack(sc, inputs.make_stack_inputs(sc, device="cuda"))
    for _ in range(args.warmup):
        st.step(accumulate=True)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    per_step = sc.n_layers * (2 if sc.recompute else 1)
    lib.ls_timing_begin(STACK_DOMINANT, args.steps * per_step)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        st.step(accumulate=True)
    stop.record(stream)
    torch.cuda.synchronize()
    n_dom, dom_ms = lib.ls_timing_end()
    ms = start.elapsed_time(stop) / args.steps
    # the optimizer step (once per global batch in training): clipped AdamW over every parameter
    st.init_optimizer()
    st.optimizer_step(lr=1e-5)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        st.optimizer_step(lr=1e-5)
    stop.record(stream)
    torch.cuda.synchronize()
    opt_ms = start.elapsed_time(stop) / args.steps
    energy = energy_of(lambda: st.step(accumulate=True), sc.tokens, args)
    fl = flops.stack_fwd_bwd_flops(sc)
    tflops = fl / (ms * 1e-3) / 1e12
    dom_tflops = flops.launch_flops(sc.block)[STACK_DOMINANT] / (dom_ms * 1e-3) / 1e12 if n_dom else None
    c = sc.block
    result = {
        "metric": f"model fwd+bwd TFLOP/s and MFU (bf16), {sc.name} ({sc.n_layers} blocks), 1 MI355X",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{sc.name}: {sc.n_layers}-block stack fwd+bwd with tied embedding, LM head and "
                               f"cross-entropy, micro-batch {c.batch} x seq {c.seq}, vocab {sc.vocab}, "
                               f"{'per-block recompute' if sc.recompute else 'no recompute (all saved states kept)'}",
                   "n_layers": sc.n_layers, "vocab": sc.vocab, "batch": c.batch, "seq": c.seq,
                   "hidden": c.hidden, "recompute": sc.recompute, "parallelism": "single GPU"},
        "mfu": round(tflops / PEAK_BF16_TFLOPS, 4),
        "tokens_per_s": round(sc.tokens / (ms * 1e-3), 1),
        "model_flops_per_step": fl,
        "tflops_paper_convention": round(flops.training_flops_per_token(
            sc.n_layers, c.hidden, c.n_q_heads, c.n_kv_heads, c.intermediate, sc.vocab, c.seq) * sc.tokens
            / (ms * 1e-3) / 1e12, 2),
        "loss": round(st.loss.item(), 4),
        "optimizer": {"kernel": "clipped AdamW over flat fp32 arrays (ls_adamw_step)", "bound": "hbm",
                      "params": st.n_params, "ms": round(opt_ms, 3),
                      "bytes_per_param": ADAMW_BYTES_PER_PARAM,
                      "achieved_gbs": round(ADAMW_BYTES_PER_PARAM * st.n_params / (opt_ms * 1e-3) / 1e9, 1),
                      "peak_gbs": PEAK_HBM_GBS,
                      "frac": round(ADAMW_BYTES_PER_PARAM * st.n_params / (opt_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
        "energy": energy,
        "roofline": {
            "kernel": f"{STACK_DOMINANT} ({LAUNCH_DESC[STACK_DOMINANT]})",
            "bound": "mfma",
            "achieved": round(dom_tflops, 2) if dom_tflops else None,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(dom_tflops / PEAK_BF16_TFLOPS, 4) if dom_tflops else None,
            "traffic": None,
            "launches": n_dom,
            "mean_ms": round(dom_ms, 4),
        },
    }
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="3b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sequences", type=int, default=4, help="sequences in the oracle's timed sample")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain 1 GiB device copy (for counter calibration) and exit")
    ap.add_argument("--kernel", choices=("gemm_nt", "torch_nt", "attention"),
                    help="time one kernel family instead of the block step (for per-kernel counters); torch_nt: "
                         "the vendor library's product of the same shape through torch, as a yardstick")
    ap.add_argument("--shape", default="8192,16384,3072", help="M,N,K of --kernel gemm_nt")
    ap.add_argument("--energy-seconds", type=float, default=2.0,
                    help="seconds of extra steps read against the GPU energy counter (0: skip)")
    ap.add_argument("--no-recompute", action="store_true",
                    help="stack configurations: keep every block's saved state instead of recomputing it")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library runs on a single MI355X "
              "(no sharding or collectives); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.kernel:
        kernel_only(args)
        return
    from paper_2510_02483_amd import configs as _configs

    if args.config in _configs.STACK_PRESETS:
        stack_bench(args)
        return

    import torch

    from paper_2510_02483_amd import configs, flops, inputs, lib

    c = configs.PRESETS[args.config]
    log(f"config {c}")
    host = inputs.make_inputs(c)
    blk = lib.Block(c, host)
    del host

    for _ in range(args.warmup):
        blk.step(accumulate=True)
    torch.cuda.synchronize()

    # untimed: every labelled launch's duration; the roofline launch is the one
    # that takes the largest share of the step
    lfl = flops.launch_flops(c)
    breakdown = launch_breakdown(lambda: blk.step(accumulate=True), flops.BLOCK_LAUNCHES, max(2, args.warmup))
    dominant = max((lb for lb in breakdown if lb in lfl), key=lambda lb: breakdown[lb][0] * breakdown[lb][1])
    per_step = breakdown[dominant][0]

    stream = torch.cuda.current_stream()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    lib.ls_timing_begin(dominant, args.steps * per_step)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        blk.step(accumulate=True)
    stop.record(stream)
    torch.cuda.synchronize()
    n_dom, dom_ms = lib.ls_timing_end()
    ms = start.elapsed_time(stop) / args.steps

    energy = energy_of(lambda: blk.step(accumulate=True), c.tokens, args)
    sclk = energy.get("sclk_mhz") if energy else None
    fl = flops.block_fwd_bwd_flops(c)
    tflops = fl / (ms * 1e-3) / 1e12
    dom_tflops = lfl[dominant] / (dom_ms * 1e-3) / 1e12 if n_dom else None
    launches = {}
    for lb, (n, lms) in breakdown.items():
        e = {"per_step": n, "us": round(lms * 1e3, 1)}
        if lb in lfl:
            tf = lfl[lb] / (lms * 1e-3) / 1e12
            e.update(tflops=round(tf, 1), frac=round(tf / PEAK_BF16_TFLOPS, 4))
        launches[lb] = e
    result = {
        "metric": METRIC if args.config == "3b" else f"decoder-block fwd+bwd TFLOP/s and MFU (bf16), {c.name}, 1 MI355X",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{WORKLOAD_NAMES.get(c.name, c.name)} decoder block fwd+bwd, batch {c.batch} x seq {c.seq}",
                   "batch": c.batch, "seq": c.seq, "hidden": c.hidden, "n_q_heads": c.n_q_heads,
                   "n_kv_heads": c.n_kv_heads, "head_dim": c.head_dim, "intermediate": c.intermediate,
                   "rope_theta": c.rope_theta, "parallelism": "single GPU"},
        "mfu": round(tflops / PEAK_BF16_TFLOPS, 4),
        "tokens_per_s": round(c.tokens / (ms * 1e-3), 1),
        "model_flops_per_step": fl,
        "tflops_noncausal_convention": round(flops.block_fwd_bwd_flops(c, causal=False) / (ms * 1e-3) / 1e12, 2),
        "energy": energy,
        "roofline": {
            "kernel": f"{dominant} ({LAUNCH_DESC.get(dominant, dominant)}): the launch with the largest share of the step",
            "bound": "mfma",
            "achieved": round(dom_tflops, 2) if dom_tflops else None,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(dom_tflops / PEAK_BF16_TFLOPS, 4) if dom_tflops else None,
            "traffic": launch_traffic(dominant, c.name),
            "launches": n_dom,
            "mean_ms": round(dom_ms, 4),
            "flops_per_launch": lfl[dominant],
            # the shader clock measured over the energy loop (same steps, right
            # after the timed ones) and the peak at that clock
            "sclk_mhz": sclk,
            "peak_at_sclk": round(PEAK_BF16_TFLOPS * sclk / 2400.0, 1) if sclk else None,
        },
        "launches": launches,
    }
    if not args.no_cpu_baseline and args.config == "3b":
        log("timing the fp64 oracle on a sample of the workload ...")
        result["cpu_baseline"] = cpu_baseline(c, args.cpu_sequences)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
