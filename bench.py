"""Benchmark of the SJD-PAC step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload verify]

Prints ONE JSON line. Workloads (synthetic, seeded; see synth_inputs.py):
  verify : sjd_verify over 4096 independent windows of 32 rows x 16384 logits
           (current logits N(0, 2^2), draft = current + N(0, 0.5^2), drafts
           drawn from top-2000 softmax of the draft logits), one launch per
           step; value = committed image tokens per second over all windows.
Inputs are resident in HBM before the timed region starts. The roofline
object reports the dominant kernel's algorithmic bytes per launch over its
average duration measured with HIP events on the launch stream; the
cpu_baseline object times the oracle on a bounded sample of the same
workload on this host's cores.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="verify", choices=["verify"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=0, help="oracle sample size (trials); 0 = default")
    return ap.parse_args()


def cpu_cores():
    try:
        return len(os.sched_getaffinity(0))
    except Exception:
        return os.cpu_count() or 1


def bench_verify(args):
    import numpy as np
    import torch

    import paper_2603_18599_amd as sjd
    from paper_2603_18599_amd.sjd import verify_outputs
    from synth_inputs import CONFIGS, verify_inputs

    c = CONFIGS["verify"]
    B, L, V, K, D, top_k = c["B"], c["L"], c["V"], c["K"], c["D"], c["top_k"]
    inp = verify_inputs(B, L, V, top_k=top_k, seed=2026, logit_std=c["logit_std"], draft_noise=c["draft_noise"],
                        device="cuda")
    out = verify_outputs(B, L, K, D)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    seed = 7

    def step(t):
        sjd.sjd_verify(inp["cur"], inp["draft"], inp["draft_tok"], inp["meta"], out, K=K, D=D, top_k=top_k,
                       temperature=c["temperature"], seed=seed, step=t, sib=inp["sib"], stream=stream)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    nc_sum = torch.zeros((), dtype=torch.int64, device="cuda")
    t0 = time.perf_counter()
    for t in range(args.steps):
        evs[t][0].record(stream)
        step(1000 + t)
        evs[t][1].record(stream)
        nc_sum += out["meta"][:, 0].sum()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = [a.elapsed_time(b) for a, b in evs]
    avg_ms = sum(kern_ms) / len(kern_ms)
    total_nc = int(nc_sum.item())
    mean_nc = total_nc / (args.steps * B)
    bytes_per_launch = 2.0 * B * L * V * 4  # current + draft logits, read once
    achieved = bytes_per_launch / (avg_ms * 1e-3) / 1e9
    ms_per_step = wall * 1e3 / args.steps
    value = total_nc / wall

    # closed form of E[n_c] for these inputs (positions independent given the logits)
    res = dict(metric="image tokens/sec on 1 MI355X; mean accept length/step; verify HBM GB/s",
               value=value, unit="image tokens/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
               ms_per_step=ms_per_step, higher_is_better=True, scaling="weak", vs_baseline=None, dtype="f32",
               data="synthetic",
               config={"workload": f"verify: {B} windows x {L} rows x {V} logits, top-{top_k}, T=1, "
                                   f"chain drafts, K={K} D={D} drafting",
                       "global_batch": B, "seq_len": L},
               mean_accept_length=mean_nc, verify_GBps=achieved,
               roofline={"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                         "kernel": "k_verify_rows + k_verify_finalize", "bytes_per_launch": bytes_per_launch,
                         "avg_launch_ms": avg_ms})
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_verify(args, inp, K, D, top_k, c["temperature"], seed, B, L)
    return res


def cpu_baseline_verify(args, inp, K, D, top_k, T, seed, B, L):
    """The oracle (plain C, OpenMP over trials) on a bounded sample of the same
    windows, scaled to committed tokens per second."""
    import numpy as np

    from oracle import oracle as orc
    n = args.cpu_sample or 2048
    idx = np.arange(n)
    cpu = {k: (v[:n].cpu().numpy() if v is not None else None) for k, v in inp.items()}
    t0 = time.perf_counter()
    r = orc.verify(cpu["cur"], cpu["draft"], cpu["draft_tok"], cpu["meta"], K=K, D=D, top_k=top_k, T=T, seed=seed,
                   step=1000, sib=cpu["sib"])
    dt = time.perf_counter() - t0
    toks = int(r["meta"][:, 0].sum())
    return {"value": toks / dt, "unit": "image tokens/s", "cores": int(os.environ.get("OMP_NUM_THREADS", cpu_cores())),
            "kind": "oracle", "sample": f"{len(idx)} of {B} windows (one verification step), {dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    if args.workload == "verify":
        res = bench_verify(args)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
