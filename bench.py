"""Benchmark of the SJD-PAC step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 7b|8b|mid|tiny|verify]

Prints ONE JSON line. Workloads (synthetic, seeded; see synth_inputs.py):
  7b (default): one SJD-PAC iteration per step (window forward of L = 32
           slots over the KV cache, verification, KV commit) of a 7B-shaped
           decoder (32 layers, d = 4096, 32 heads x 128, SwiGLU 11008, vocab
           65536, bf16 random-init weights), generating a 48x48 image with
           row-end tokens after a 64-token random prompt; top-2000, T = 1,
           K = 4, D = 3. value = committed image tokens per second. The same
           line carries the verify workload's numbers under "verify".
  8b, mid, tiny: the other decoder shapes.
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
    ap.add_argument("--workload", default="7b", choices=["7b", "8b", "mid", "tiny", "verify"])
    ap.add_argument("--no-verify", action="store_true", help="skip the verify workload section")
    ap.add_argument("--context", default="mid", choices=["mid", "start"],
                    help="mid: time the steps half-way through an image (prompt + n_gen/2 tokens cached); "
                         "start: right after the prompt")
    ap.add_argument("--mode", default="sjd-pac", choices=["sjd-pac", "sjd", "ac", "pd"],
                    help="verification mode (Sec. 5.3 ablation): both adaptive continuation and proactive "
                         "drafting, vanilla SJD, AC only, PD only")
    ap.add_argument("--L", type=int, default=0, help="window slots (0 = the workload's)")
    ap.add_argument("--K", type=int, default=0, help="drafting candidates per tree row (0 = the workload's)")
    ap.add_argument("--D", type=int, default=-1, help="tree depth (-1 = the workload's)")
    ap.add_argument("--batch", type=int, default=1, choices=[1, 2],
                    help="images per step (2: both windows in one forward, one pass over the weights)")
    ap.add_argument("--no-batch2", action="store_true", help="skip the two-images-per-step section")
    ap.add_argument("--cfg-w", type=float, default=0.0,
                    help="classifier-free guidance weight (Sec. 5.1 samples with 3): a text-prompt and an "
                         "unconditional stream in one window forward; 0 = unguided")
    ap.add_argument("--no-guided", action="store_true", help="skip the guided (CFG weight 3) section")
    ap.add_argument("--eager", action="store_true", help="enqueue every kernel directly (no captured graph)")
    ap.add_argument("--tune", action="store_true",
                    help="time candidate GEMM plans at init (SJD_TUNE) instead of the recorded / closed-form plan")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=0, help="oracle sample size (trials); 0 = default")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one 256 MiB device-to-device copy before the timed region (the reference kernel "
                         "of known size for HBM counter runs) and mark copy + timed region as the profiler's "
                         "selected region (rocprofv3 --selected-regions)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="read two rocprofv3 --pmc output directories (FETCH_SIZE, WRITE_SIZE) of a "
                         "--calibrate-copy run of this workload and record the measured HBM bytes per launch "
                         "in profiles/traffic_<workload>.txt")
    return ap.parse_args()


CALIB_BYTES = 256 << 20


def kernel_source_hash():
    """sha256 over the HIP/C++ sources of the library: a recorded traffic
    figure is reported only while the kernels it was measured on are
    unchanged."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2603_18599_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".cpp", ".h")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")


def recorded_traffic(workload):
    """Measured HBM bytes per launch (FETCH + WRITE) from the counter record,
    or None if there is none or the kernels changed since."""
    try:
        with open(traffic_file(workload)) as fh:
            rec = dict(l.strip().split("=", 1) for l in fh if "=" in l and not l.startswith("#"))
    except OSError:
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    try:
        return float(rec["fetch_bytes_per_launch"]) + float(rec["write_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def profiler_region(on):
    """Resume (on) or pause the profiler's collection (rocprofv3
    --selected-regions); a no-op when the ROCtx library is absent."""
    import ctypes
    for name in ("librocprofiler-sdk-roctx.so.1", "librocprofiler-sdk-roctx.so"):
        try:
            lib = ctypes.CDLL(name)
        except OSError:
            continue
        fn = lib.roctxProfilerResume if on else lib.roctxProfilerPause
        fn.argtypes = [ctypes.c_uint64]
        fn(0)
        return


def calibration_copy():
    import torch
    a = torch.empty(CALIB_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    del a, b


def read_counter(dirname, counter):
    """{dispatch id: (kernel name, summed value)} from a rocprofv3 counter_collection.csv"""
    import csv
    import glob
    files = glob.glob(os.path.join(dirname, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {dirname}")
    files = [max(files, key=os.path.getmtime)]  # the newest run only (dispatch ids restart per run)
    out = {}
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                d = int(r["Dispatch_Id"])
                name, v = out.get(d, (r["Kernel_Name"], 0.0))
                out[d] = (name, v + float(r["Counter_Value"]))
    return out


def traffic_from(args):
    """Per-launch HBM bytes from FETCH_SIZE / WRITE_SIZE (KiB per dispatch),
    each scaled by the counter's reading on the calibration copy of known
    size; written to profiles/traffic_<workload>.txt."""
    per = {}
    facs = {}
    for counter, d in (("FETCH_SIZE", args.traffic_from[0]), ("WRITE_SIZE", args.traffic_from[1])):
        c = read_counter(d, counter)
        ids = sorted(c)
        # the calibration copy is the last large device-to-device copy before
        # the timed launches (the model set-up may copy earlier)
        copies = [i for i in ids if "copyBuffer" in c[i][0] and c[i][1] * 1024.0 >= CALIB_BYTES / 8]
        if args.workload == "verify":
            launches_all = [i for i in ids if "k_verify_rows" in c[i][0]]
        else:
            launches_all = [i for i in ids if "k_build_window" in c[i][0]]
        copies = [i for i in copies if any(j > i for j in launches_all)]
        if not copies:
            raise SystemExit(f"{counter}: no calibration copy found (run with --calibrate-copy)")
        cal = max(copies)
        fac = CALIB_BYTES / (c[cal][1] * 1024.0)
        facs[counter] = fac
        if args.workload == "verify":
            launches = [i for i in ids if "k_verify_rows" in c[i][0] and i > cal]
            tot = []
            for i in launches:
                fin = [j for j in ids if j > i and "k_verify_finalize" in c[j][0]]
                tot.append(c[i][1] + (c[fin[0]][1] if fin else 0.0))
        else:
            starts = [i for i in ids if "k_build_window" in c[i][0] and i > cal]
            tot = []
            for a, b in zip(starts, starts[1:]):
                tot.append(sum(c[j][1] for j in ids if a <= j < b))
        if not tot:
            raise SystemExit(f"{counter}: no launches of the {args.workload} workload found")
        per[counter] = sum(tot) / len(tot) * 1024.0 * fac
    wl = "" if args.workload == "7b" else f" --workload {args.workload}"
    run = (f"python3 bench.py{wl} --steps 3 --warmup 1 --no-cpu-baseline --no-verify --calibrate-copy"
           if args.workload != "verify" else "python3 bench.py --workload verify --steps 2 --warmup 1 "
                                              "--no-cpu-baseline --calibrate-copy")
    lines = ["# Measured HBM traffic per launch (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE; KiB per dispatch",
             "# summed over the dispatches of one launch, scaled by the counter's reading on a 256 MiB",
             "# device-to-device copy in the same run). Reported by bench.py while source_hash matches.",
             "# Commands (repository root; cd /tmp && export TMPDIR=/tmp first):",
             f"#   rocprofv3 --pmc FETCH_SIZE --output-format csv -d <fetch_dir> -- {run}",
             f"#   rocprofv3 --pmc WRITE_SIZE --output-format csv -d <write_dir> -- {run}",
             f"#   python3 bench.py{' --workload ' + args.workload} --traffic-from <fetch_dir> <write_dir>",
             f"workload={args.workload}",
             f"source_hash={kernel_source_hash()}",
             f"fetch_bytes_per_launch={per['FETCH_SIZE']:.0f}",
             f"write_bytes_per_launch={per['WRITE_SIZE']:.0f}",
             f"fetch_calibration={facs['FETCH_SIZE']:.4f}",
             f"write_calibration={facs['WRITE_SIZE']:.4f}"]
    with open(traffic_file(args.workload), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def progress(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


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
    if getattr(args, "calibrate_copy", False):
        profiler_region(True)
        calibration_copy()
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
    if getattr(args, "calibrate_copy", False):
        profiler_region(False)
    kern_ms = [a.elapsed_time(b) for a, b in evs]
    avg_ms = sum(kern_ms) / len(kern_ms)
    total_nc = int(nc_sum.item())
    mean_nc = total_nc / (args.steps * B)
    bytes_per_launch = 2.0 * B * L * V * 4  # current + draft logits, read once
    achieved = bytes_per_launch / (avg_ms * 1e-3) / 1e9
    ms_per_step = wall * 1e3 / args.steps
    value = total_nc / wall

    res = dict(metric="image tokens/sec on 1 MI355X; mean accept length/step; verify HBM GB/s",
               value=value, unit="image tokens/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
               ms_per_step=ms_per_step, higher_is_better=True, scaling="weak", vs_baseline=None, dtype="f32",
               data="synthetic",
               config={"workload": f"verify: {B} windows x {L} rows x {V} logits, top-{top_k}, T=1, "
                                   f"chain drafts, K={K} D={D} drafting",
                       "global_batch": B, "seq_len": L},
               mean_accept_length=mean_nc, verify_GBps=achieved,
               roofline={"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBPS, "traffic": recorded_traffic("verify"),
                         "kernel": "k_verify_rows + k_verify_finalize", "bytes_per_launch": bytes_per_launch,
                         "avg_launch_ms": avg_ms})
    res["expected_accept_length"], res["expected_accept_length_over_drafts"] = chain_expected_nc(
        inp["cur"], inp["draft"], inp["draft_tok"], top_k, c["temperature"])
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_verify(args, inp, K, D, top_k, c["temperature"], seed, B, L)
    return res


def chain_expected_nc(cur, draft, draft_tok, top_k, T, chunk=128):
    """Closed-form mean committed length of these chain windows, reported
    beside the measured mean. A step commits the accepted prefix plus one
    token, at most L, and given the logits the rows are independent:
    E[n_c] = 1 + sum_{i=1}^{L-1} prod_{j<i} a_j, averaged over the windows.
    Returns (a_j given the drafted tokens x_j: min(1, p_j(x_j) / q_j(x_j)),
    the exact expectation of the timed steps, whose accept draws are fresh
    each step while the drafts are fixed; a_j over draft draws from q_j:
    sum_x min(p_j, q_j), one minus the total-variation distance, Sec. 3).
    p and q are the top-k softmaxes of the current and draft logits at
    temperature T (plain torch ops: a statistic of the inputs, not part of
    the measured path)."""
    import torch

    B, L, V = cur.shape
    k = V if top_k <= 0 or top_k >= V else top_k

    def topk_softmax(x):
        vals, idx = torch.topk(x / T, k, dim=1)
        return torch.zeros_like(x).scatter_(1, idx, torch.softmax(vals.double(), dim=1).float())

    def expect(a):
        return (1.0 + torch.cumprod(a[:, :L - 1], dim=1).sum(1)).sum().item()

    given, over = 0.0, 0.0
    for w0 in range(0, B, chunk):
        p = topk_softmax(cur[w0:w0 + chunk].reshape(-1, V).float())
        q = topk_softmax(draft[w0:w0 + chunk].reshape(-1, V).float())
        x = draft_tok[w0:w0 + chunk].reshape(-1, 1).long()
        px, qx = p.gather(1, x).double(), q.gather(1, x).double()
        given += expect(torch.clamp(px / qx, max=1.0).view(-1, L))
        over += expect(torch.minimum(p, q).double().sum(1).view(-1, L))
    return given / B, over / B


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


def step_bytes(cfg, n_mean, B=1, streams=None):
    """Algorithmic HBM bytes of one step: every weight streamed once (bf16),
    the LM head rows of the sampled range only, the cached keys and values
    read once (hi/lo bf16 planes, 4 bytes per element), the window's K/V
    written, and the logits written and read back by the verification; B
    images share the weight stream, each has its own cache and logits
    (n_mean: mean cached rows per image); a guided step has two streams
    (two caches) and one image's logits."""
    d, H, Hkv, hd, F, V, L = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "V", "L"))
    per_layer = (H * hd * d + 2 * Hkv * hd * d + d * H * hd + 3 * F * d) * 2
    weights = cfg["n_layers"] * per_layer + V * d * 2
    kv = (streams or B) * cfg["n_layers"] * 2 * Hkv * hd * 4 * (n_mean + L)
    logits = B * 2 * L * V * 4 * 2  # written once, current + draft rows read once
    return weights + kv + logits, weights, kv


def bench_step(args):
    import numpy as np
    import torch

    from paper_2603_18599_amd.sjd import Engine, SjdError
    from synth_inputs import image_history, model_config, model_weights, prompt_tokens

    over = {"flags": {"sjd-pac": 3, "sjd": 0, "ac": 1, "pd": 2}[args.mode] | (4 if args.eager else 0)
            | (16 if getattr(args, "tune", False) else 0)}
    if args.L > 0:
        over["L"] = args.L
    if args.K > 0:
        over["K"] = args.K
    if args.D >= 0:
        over["D"] = args.D
    if args.mode in ("sjd", "ac") and args.K <= 0:
        over["K"], over["D"] = 1, 0  # no drafting tree without PD
    B = args.batch
    over["batch"] = B
    guided = args.cfg_w != 0.0
    if guided:
        if B != 1:
            raise SystemExit("guidance runs one image per step (--batch 1)")
        over["cfg_w"] = args.cfg_w
    cfg = model_config(args.workload, **over)
    seed = 11
    w = model_weights(cfg, 1, device="cuda")
    prompts = []
    for b in range(B):  # image b: its own prompt (and image so far)
        p = prompt_tokens(cfg, 2 + 10 * b)
        if args.context == "mid":
            p = torch.cat([p, image_history(cfg, cfg["n_gen"] // 2, 3 + 10 * b)])
        prompts.append(p.cuda())
    prompt = prompts[0]
    uncond = None
    if guided:  # the unconditional stream: its own prompt ids, the same image so far
        u = prompt_tokens(cfg, 77)
        if args.context == "mid":
            u = torch.cat([u, image_history(cfg, cfg["n_gen"] // 2, 3)])
        uncond = u.cuda()
    eng = Engine(cfg, w)
    stream = torch.cuda.current_stream()
    K, W = args.steps, args.warmup
    metas = torch.zeros(W + K, B, 8, dtype=torch.int32, device="cuda")

    def prefill_all(sd):
        if guided:
            eng.prefill_cfg(prompts[0], uncond, sd, stream=stream)
            return
        for b in range(B):
            eng.prefill_image(b, prompts[b], sd + 1000 * b, stream=stream)

    if not args.calibrate_copy:  # (counter runs: one prefill only, each dispatch is slow there)
        prefill_all(seed)
    torch.cuda.synchronize()
    progress(f"model ready; prefill of {B} x {prompt.numel()} tokens")
    t_pre = time.perf_counter()
    prefill_all(seed)
    torch.cuda.synchronize()
    prefill_ms = (time.perf_counter() - t_pre) * 1e3
    restarts = 0

    def one(t):
        nonlocal restarts
        try:
            eng.step(cfg["temperature"], cfg["top_k"], seed, t, out_meta=metas[t], stream=stream)
        except SjdError as e:
            if e.code != -4:
                raise
            restarts += 1  # an image is complete: its cache is full, start the next images
            prefill_all(seed + restarts)
            eng.step(cfg["temperature"], cfg["top_k"], seed, t, out_meta=metas[t], stream=stream)

    progress("prefill done")
    for t in range(W):
        one(t)
    torch.cuda.synchronize()
    progress("warmup done")
    if args.calibrate_copy:
        profiler_region(True)
        calibration_copy()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    host_s = 0.0  # host time spent enqueueing steps
    t0 = time.perf_counter()
    for i in range(K):
        evs[i][0].record(stream)
        th = time.perf_counter()
        one(W + i)
        host_s += time.perf_counter() - th
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if args.calibrate_copy:
        profiler_region(False)
    m = metas.cpu().numpy()
    ncs = m[W:, :, 0]  # [step][image]
    ns = m[W:, :, 7]
    step_ms = [a.elapsed_time(b) for a, b in evs]
    avg_ms = float(np.mean(step_ms))
    n_mean = float(np.mean(ns - ncs))
    total, weights, kv = step_bytes(cfg, n_mean, B, streams=2 if guided else None)
    achieved = total / (avg_ms * 1e-3) / 1e9
    res = dict(metric="image tokens/sec on 1 MI355X; mean accept length/step; verify HBM GB/s",
               value=float(ncs.sum()) / wall, unit="image tokens/s", n_gpus=1, steps=K, warmup=W,
               ms_per_step=wall * 1e3 / K, higher_is_better=True, scaling="weak", vs_baseline=None, dtype="bf16",
               data="synthetic (random-init weights, random prompt ids)",
               config={"workload": f"{args.workload}-shaped decoder: {cfg['n_layers']} layers, d={cfg['d_model']}, "
                                   f"{cfg['n_heads']}q/{cfg['n_kv_heads']}kv heads x {cfg['head_dim']}, "
                                   f"SwiGLU {cfg['ffn_dim']}, vocab {cfg['vocab_size']} (sampled {cfg['V']}), "
                                   f"L={cfg['L']} K={cfg['K']} D={cfg['D']}, mode {args.mode}, "
                                   + (f"{B} images per step, " if B > 1 else "") +
                                   (f"CFG weight {args.cfg_w:g} (text + unconditional stream), " if guided else "") +
                                   f"top-{cfg['top_k']}, T=1, "
                                   f"{cfg['n_prompt']}-token prompt, {cfg['n_gen']}-token image, "
                                   f"steps timed from KV length {prompt.numel() - 1}",
                       "global_batch": B, "seq_len": cfg["L"]},
               mean_accept_length=float(ncs.mean()), step_latency_ms=avg_ms,
               step_latency_p50_ms=float(np.percentile(step_ms, 50)),
               step_latency_p99_ms=float(np.percentile(step_ms, 99)),
               prefill_ms=prefill_ms, kv_rows_mean=n_mean, image_restarts=restarts,
               host_enqueue_ms_per_step=host_s * 1e3 / K, split_plan=eng.plan(), split_pin=eng.plan_pin(),
               roofline={"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBPS, "traffic": recorded_traffic(args.workload),
                         "kernel": "sjd_step (window forward + verification + KV commit)",
                         "bytes_per_launch": total, "weight_bytes": weights, "kv_bytes": kv,
                         "avg_launch_ms": avg_ms,
                         "mfma_tflops": 2.0 * weights / 2 * cfg["L"] * B / (avg_ms * 1e-3) / 1e12})
    eng.close()
    del w
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_step(args, cfg, seed)
    return res


def cpu_baseline_step(args, cfg, seed):
    """The oracle (plain C, fp64 accumulation, OpenMP) on one SJD-PAC step of
    the same model at the same start: weights regenerated from the same seed,
    prompt prefilled untimed, then the first window's forward + verification
    timed. Scaled to committed tokens per second."""
    import numpy as np
    import torch

    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from model_util import oracle_model, oracle_prefill, placeholders, weights_numpy
    from oracle import oracle as orc
    from synth_inputs import model_weights, prompt_tokens

    w = model_weights(cfg, 1, device="cuda")
    w = dict(embed=w["embed"].cpu(), final_norm=w["final_norm"].cpu(), lm_head=w["lm_head"].cpu(),
             layers=[{k: v.cpu() for k, v in l.items()} for l in w["layers"]])
    prompt = prompt_tokens(cfg, 2).numpy().astype(np.int32)
    m = oracle_model(orc, cfg, weights_numpy(w))
    n = oracle_prefill(m, prompt)
    L, V = cfg["L"], cfg["V"]
    spine = placeholders(orc, cfg, seed)
    t0 = time.perf_counter()
    logits = m.forward(n, [int(prompt[-1])] + spine[:L - 1], [n + i for i in range(L)],
                       [(1 << (a + 1)) - 1 for a in range(L)])
    meta = np.array([[0, 0, 0, 0]], np.int32)
    r = orc.verify(logits[None], logits[None], np.array([spine], np.int32), meta, K=cfg["K"], D=cfg["D"],
                   top_k=cfg["top_k"], T=cfg["temperature"], flags=cfg.get("flags", 3), seed=seed, step=0,
                   vis_lo=cfg["vis_lo"],
                   eol_id=cfg["eol_id"], row_len=cfg["row_len"])
    dt = time.perf_counter() - t0
    m.close()
    n_c = int(r["meta"][0, 0])
    return {"value": n_c / dt, "unit": "image tokens/s", "cores": int(os.environ.get("OMP_NUM_THREADS", cpu_cores())),
            "kind": "oracle",
            "sample": f"first SJD-PAC step after a {cfg['n_prompt']}-token prefill (prefill untimed): "
                      f"{L}-slot window forward + verification, {dt:.1f} s, n_c={n_c}"}


def main():
    args = parse()
    if args.traffic_from:
        traffic_from(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    if args.workload == "verify":
        res = bench_verify(args)
    else:
        res = bench_step(args)
        if not args.no_verify:
            v = bench_verify(argparse.Namespace(steps=10, warmup=2, no_cpu_baseline=True, cpu_sample=0,
                                                calibrate_copy=False))
            res["verify"] = {k: v[k] for k in ("value", "unit", "ms_per_step", "mean_accept_length",
                                               "expected_accept_length", "expected_accept_length_over_drafts",
                                               "verify_GBps", "roofline", "config")}
        if args.batch == 1 and not args.no_batch2 and not args.calibrate_copy:
            # the same workload with two images per step (serving several requests)
            b2 = bench_step(argparse.Namespace(**dict(vars(args), batch=2, no_cpu_baseline=True)))
            res["batch2"] = {k: b2[k] for k in ("value", "unit", "ms_per_step", "mean_accept_length",
                                                "step_latency_ms", "config")}
            res["batch2"]["roofline_frac"] = b2["roofline"]["frac"]
        if args.batch == 1 and args.cfg_w == 0.0 and not args.no_guided and not args.calibrate_copy:
            # the paper's sampling setting: guidance weight 3 (Sec. 5.1), both streams in one forward
            gd = bench_step(argparse.Namespace(**dict(vars(args), cfg_w=3.0, no_cpu_baseline=True)))
            res["guided"] = {k: gd[k] for k in ("value", "unit", "ms_per_step", "mean_accept_length",
                                                "step_latency_ms", "config")}
            res["guided"]["roofline_frac"] = gd["roofline"]["frac"]
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
