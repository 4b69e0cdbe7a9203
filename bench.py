"""Benchmark of the SJD-PAC step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 7b|8b|mid|tiny|verify]

Prints ONE JSON line. Workloads (synthetic, seeded; see synth_inputs.py):
  7b (default): one SJD-PAC iteration per step (window forward of L = 32
           slots over the KV cache, verification, KV commit) of a 7B-shaped
           decoder (32 layers, d = 4096, 32 heads x 128, SwiGLU 11008, vocab
           65536, bf16 random-init weights), generating a 48x48 image with
           row-end tokens after a 64-token random prompt; top-2000, T = 1,
           K = 4, D = 3. value = committed image tokens per second. The same
           line carries the other workloads under "verify", "tiny", "mid" and
           "8b" (each with its roofline fraction and oracle baseline), the
           7B step with two and four images per step ("batch2", "batch4"),
           with guidance weight 3 ("guided") and with two guided images per
           step ("guided_batch2", four streams in one forward).
  8b, mid, tiny: the other decoder shapes.
  --sweep: ablation modes and the K/D/L grid on a small model (one JSON line
           per configuration).
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
    ap.add_argument("--batch", type=int, default=1, choices=[1, 2, 3, 4],
                    help="images per step (all windows in one forward, one pass over the weights; "
                         "at most 2 with --cfg-w)")
    ap.add_argument("--no-batch2", action="store_true",
                    help="skip the batched sections (2 and 4 images per step, 2 guided images per step)")
    ap.add_argument("--cfg-w", type=float, default=0.0,
                    help="classifier-free guidance weight (Sec. 5.1 samples with 3): a text-prompt and an "
                         "unconditional stream in one window forward; 0 = unguided")
    ap.add_argument("--no-guided", action="store_true", help="skip the guided (CFG weight 3) section")
    ap.add_argument("--top-k", type=int, default=-1, help="sampler top-k (-1 = the workload's; 1 = greedy)")
    ap.add_argument("--eager", action="store_true", help="enqueue every kernel directly (no captured graph)")
    ap.add_argument("--tune", action="store_true",
                    help="time candidate GEMM plans at init (SJD_TUNE) instead of the recorded / closed-form plan")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip the tiny, mid and 8b sections of the 7b line")
    ap.add_argument("--sweep", action="store_true",
                    help="ablation modes and K in 2..5 x D in 2..4 x L in {32, 64} on --workload (tiny or mid)")
    ap.add_argument("--sweep-images", type=int, default=4, help="whole images generated per sweep configuration")
    ap.add_argument("--cpu-sample", type=int, default=0, help="oracle sample size (verify windows); 0 = 1024")
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


def default_step_config(args):
    """True for the step configuration the traffic records measure (one
    image, no guidance, the workload's window, tree, mode, sampler and
    cache point; graph replay, recorded plan): a record does not apply to
    any other."""
    return (args.batch == 1 and args.cfg_w == 0.0 and args.L == 0 and args.K == 0 and args.D == -1
            and args.mode == "sjd-pac" and args.top_k == -1 and args.context == "mid" and not args.eager
            and not args.tune)


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


_HBM_REF = None


def hbm_reference():
    """This device's measured copy rate, for a fraction beside the one of the
    published 8 TB/s peak: a 2 GiB device-to-device copy through the HIP
    runtime, read + write bytes, best of five, measured once per run outside
    every timed region (a yardstick, not the measured path; a plain
    streaming-read kernel reaches more, about 6.6-7.0 TB/s on 100-540 MB)."""
    global _HBM_REF
    if _HBM_REF is not None:
        return _HBM_REF
    import torch

    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    a = torch.empty(1 << 29, dtype=torch.float32, device="cuda").fill_(1.0)  # 2 GiB
    b = torch.empty_like(a)
    b.copy_(a)
    t = []
    for _ in range(5):
        ev[0].record()
        b.copy_(a)
        ev[1].record()
        torch.cuda.synchronize()
        t.append(ev[0].elapsed_time(ev[1]))
    del a, b
    torch.cuda.empty_cache()
    _HBM_REF = {"copy_GBps": 2.0 * (1 << 29) * 4 / (min(t) * 1e-3) / 1e9}
    return _HBM_REF


def with_measured(roof):
    """roofline dict + the achieved rate over this device's measured copy rate"""
    ref = hbm_reference()
    roof["measured_copy_GBps"] = ref["copy_GBps"]
    roof["frac_of_copy"] = roof["achieved"] / ref["copy_GBps"]
    return roof


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


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for l in fh:
                if l.startswith("model name"):
                    return l.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


class omp_threads:
    """Sets the OpenMP thread count of the oracle's parallel regions (called
    from this thread) for the duration of a with-block."""

    def __init__(self, n):
        import ctypes
        self.n = n
        self.gomp = None
        for name in ("libgomp.so.1", "libgomp.so"):
            try:
                self.gomp = ctypes.CDLL(name)
                break
            except OSError:
                continue

    def __enter__(self):
        if self.gomp is not None:
            self.prev = self.gomp.omp_get_max_threads()
            self.gomp.omp_set_num_threads(self.n)
        return self

    def __exit__(self, *a):
        if self.gomp is not None:
            self.gomp.omp_set_num_threads(self.prev)


def all_threads():
    return int(os.environ.get("OMP_NUM_THREADS", cpu_cores()))


def nc_histogram(ncs, L):
    """counts of the committed lengths 1 .. L (index 0 = n_c of 1)"""
    import numpy as np
    h = np.bincount(np.asarray(ncs, dtype=np.int64).ravel(), minlength=L + 1)[1:L + 1]
    return [int(v) for v in h]


# ---------------------------------------------------------------------------- verify workload
def bench_verify(args, cpu=True):
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

    def step(t, rows=None):
        sjd.sjd_verify(inp["cur"], inp["draft"], inp["draft_tok"], inp["meta"], out, K=K, D=D, top_k=top_k,
                       temperature=c["temperature"], seed=seed, step=t, sib=inp["sib"], stream=stream,
                       out_rows=rows)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    if getattr(args, "calibrate_copy", False):
        profiler_region(True)
        calibration_copy()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    ncs = torch.zeros(args.steps, B, dtype=torch.int32, device="cuda")
    t0 = time.perf_counter()
    for t in range(args.steps):
        evs[t][0].record(stream)
        step(1000 + t)
        evs[t][1].record(stream)
        ncs[t].copy_(out["meta"][:, 0])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if getattr(args, "calibrate_copy", False):
        profiler_region(False)
    kern_ms = [a.elapsed_time(b) for a, b in evs]
    avg_ms = sum(kern_ms) / len(kern_ms)
    nc = ncs.cpu().numpy()
    total_nc = int(nc.sum())
    bytes_per_launch = 2.0 * B * L * V * 4  # current + draft logits, each read once
    achieved = bytes_per_launch / (avg_ms * 1e-3) / 1e9
    res = dict(metric="image tokens/sec on 1 MI355X; mean accept length/step; verify HBM GB/s",
               value=total_nc / wall, unit="image tokens/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
               ms_per_step=wall * 1e3 / args.steps, higher_is_better=True, scaling="weak", vs_baseline=None,
               dtype="f32", data="synthetic",
               config={"workload": f"verify: {B} windows x {L} rows x {V} logits, top-{top_k}, T=1, "
                                   f"chain drafts, K={K} D={D} drafting",
                       "global_batch": B, "seq_len": L},
               mean_accept_length=total_nc / nc.size, nc_hist=nc_histogram(nc, L), verify_GBps=achieved,
               roofline={"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBPS, "traffic": recorded_traffic("verify"),
                         "kernel": "k_verify_rows + k_verify_finalize", "bytes_per_launch": bytes_per_launch,
                         "avg_launch_ms": avg_ms})
    if not getattr(args, "calibrate_copy", False):
        with_measured(res["roofline"])
    res["expected_accept_length"], res["expected_accept_length_over_drafts"] = chain_expected_nc(
        inp["cur"], inp["draft"], inp["draft_tok"], top_k, c["temperature"])
    if cpu and not args.no_cpu_baseline:
        # the GPU's decisions of step 1000 on the sampled windows, for the
        # parity report beside the oracle's timing
        rows = torch.zeros(B, L, 2, dtype=torch.int32, device="cuda")
        step(1000, rows)
        torch.cuda.synchronize()
        gpu = {k: v.cpu().numpy() for k, v in out.items()}
        gpu["rows"] = rows.cpu().numpy()
        res["cpu_baseline"], res["parity_sample"] = cpu_baseline_verify(args, inp, gpu, K, D, top_k,
                                                                        c["temperature"], seed, B, L, V)
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


def cpu_baseline_verify(args, inp, gpu, K, D, top_k, T, seed, B, L, V):
    """The oracle (plain C, OpenMP over windows) on a bounded sample of the
    same windows and step, on all host cores and on one core, scaled to
    committed tokens per second; its decisions on the sample are compared
    with the GPU's (near-tie report)."""
    import numpy as np

    from oracle import oracle as orc
    from oracle.parity import compare_verify
    n = args.cpu_sample or 1024
    n1 = max(8, n // 16)
    cpu = {k: (v[:n].cpu().numpy() if v is not None else None) for k, v in inp.items()}

    def run(m):
        sub = {k: (v[:m] if v is not None else None) for k, v in cpu.items()}
        t0 = time.perf_counter()
        r = orc.verify(sub["cur"], sub["draft"], sub["draft_tok"], sub["meta"], K=K, D=D, top_k=top_k, T=T,
                       seed=seed, step=1000, sib=sub["sib"])
        return r, time.perf_counter() - t0

    cores = all_threads()
    with omp_threads(cores):
        r, dt = run(n)
    with omp_threads(1):
        r1, dt1 = run(n1)
    toks, toks1 = int(r["meta"][:, 0].sum()), int(r1["meta"][:, 0].sum())
    rep = []
    sub_gpu = {k: v[:n] for k, v in gpu.items()}
    compare_verify(sub_gpu, r, K=K, D=D, report=rep, label=f"verify workload, first {n} windows")
    base = {"value": toks / dt, "unit": "image tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"first {n} of {B} windows (step 1000), {dt:.1f} s on {cores} threads ({cpu_model()}); "
                      f"full {B}-window step extrapolated: {dt * B / n:.1f} s",
            "one_thread": {"value": toks1 / dt1, "unit": "image tokens/s", "cores": 1,
                           "sample": f"first {n1} windows, {dt1:.1f} s"},
            "bytes_per_s": 2.0 * n * L * V * 4 / dt}
    return base, rep[0]


# ---------------------------------------------------------------------------- decoder step
def step_bytes(cfg, n_mean, B=1, streams=None):
    """Algorithmic HBM bytes of one step (the per-unit figures of the
    method's byte model): every weight streamed once (bf16), the LM head
    rows of the sampled range only; the cached keys and values read once in
    bf16, 2 * layers * Hkv * hd * 2 bytes per cached row at the mean fill;
    the logits written once and read once as current rows and once as draft
    rows (3 * L * V * 4 bytes). B images share the weight stream, each with
    its own cache and logits; a guided step has two streams (two caches) and
    one image's logits. Returns (total, weights, kv, logits, kv_hilo): kv_hilo
    is what the cache actually moves, two bf16 planes per element (the
    precision design), reported beside the algorithmic figure."""
    d, H, Hkv, hd, F, V, L = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "V", "L"))
    per_layer = (H * hd * d + 2 * Hkv * hd * d + d * H * hd + 3 * F * d) * 2
    weights = cfg["n_layers"] * per_layer + V * d * 2
    kv_row = cfg["n_layers"] * 2 * Hkv * hd * 2
    kv = (streams or B) * kv_row * n_mean
    logits = B * 3 * L * V * 4
    return weights + kv + logits, weights, kv, logits, 2 * kv


def decoder_inputs(cfg, B, context, guided, device="cuda"):
    import torch

    from synth_inputs import image_history, prompt_tokens
    prompts, uncond = [], []
    for b in range(B):  # image b: its own prompt (and image so far)
        p = prompt_tokens(cfg, 2 + 10 * b)
        if context == "mid":
            p = torch.cat([p, image_history(cfg, cfg["n_gen"] // 2, 3 + 10 * b)])
        prompts.append(p.to(device))
        if guided:  # the unconditional stream: its own prompt ids, the same image so far
            u = prompt_tokens(cfg, 77 + 10 * b)
            if context == "mid":
                u = torch.cat([u, image_history(cfg, cfg["n_gen"] // 2, 3 + 10 * b)])
            uncond.append(u.to(device))
    return prompts, uncond


def workload_config(args, workload=None):
    from synth_inputs import model_config
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
    if getattr(args, "top_k", -1) >= 0:
        over["top_k"] = args.top_k
    over["batch"] = args.batch
    if args.cfg_w != 0.0:
        if args.batch > 2:
            raise SystemExit("guidance runs at most two images per step (four streams)")
        over["cfg_w"] = args.cfg_w
    return model_config(workload or args.workload, **over)


def bench_step(args, cpu=True):
    import numpy as np
    import torch

    from paper_2603_18599_amd.sjd import Engine, SjdError
    from synth_inputs import model_weights

    cfg = workload_config(args)
    B = args.batch
    guided = args.cfg_w != 0.0
    seed = 11
    w = model_weights(cfg, 1, device="cuda")
    prompts, uncond = decoder_inputs(cfg, B, args.context, guided)
    prompt = prompts[0]
    eng = Engine(cfg, w)
    stream = torch.cuda.current_stream()
    K, W = args.steps, args.warmup
    metas = torch.zeros(W + K, B, 8, dtype=torch.int32, device="cuda")

    def prefill_all(sd):
        for b in range(B):
            if guided:
                eng.prefill_cfg(prompts[b], uncond[b], sd + 1000 * b, stream=stream, image=b)
            else:
                eng.prefill_image(b, prompts[b], sd + 1000 * b, stream=stream)

    if not args.calibrate_copy:  # (counter runs: one prefill only, each dispatch is slow there)
        prefill_all(seed)
    torch.cuda.synchronize()
    progress(f"{args.workload}: model ready; prefill of {B} x {prompt.numel()} tokens")
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

    for t in range(W):
        one(t)
    torch.cuda.synchronize()
    progress(f"{args.workload}: warmup done")
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
    total, weights, kv, logit_b, kv_hilo = step_bytes(cfg, n_mean, B, streams=2 * B if guided else None)
    achieved = total / (avg_ms * 1e-3) / 1e9
    moved = total - kv + kv_hilo
    res = dict(metric="image tokens/sec on 1 MI355X; mean accept length/step; verify HBM GB/s",
               value=float(ncs.sum()) / wall, unit="image tokens/s", n_gpus=1, steps=K, warmup=W,
               ms_per_step=wall * 1e3 / K, higher_is_better=True, scaling="weak", vs_baseline=None, dtype="bf16",
               data="synthetic (random-init weights, random prompt ids)",
               config={"workload": f"{args.workload}-shaped decoder: {cfg['n_layers']} layers, d={cfg['d_model']}, "
                                   f"{cfg['n_heads']}q/{cfg['n_kv_heads']}kv heads x {cfg['head_dim']}, "
                                   f"SwiGLU {cfg['ffn_dim']}, vocab {cfg['vocab_size']} (sampled {cfg['V']}), "
                                   f"L={cfg['L']} K={cfg['K']} D={cfg['D']}, mode {args.mode}, "
                                   + (f"{B} images per step, " if B > 1 else "") +
                                   (f"CFG weight {args.cfg_w:g} (text + unconditional stream per image), "
                                    if guided else "") +
                                   f"top-{cfg['top_k']}, T=1, "
                                   f"{cfg['n_prompt']}-token prompt, {cfg['n_gen']}-token image, "
                                   f"steps timed from KV length {prompt.numel() - 1}",
                       "global_batch": B, "seq_len": cfg["L"]},
               mean_accept_length=float(ncs.mean()), nc_hist=nc_histogram(ncs, cfg["L"]), step_latency_ms=avg_ms,
               step_latency_p50_ms=float(np.percentile(step_ms, 50)),
               step_latency_p99_ms=float(np.percentile(step_ms, 99)),
               prefill_ms=prefill_ms, kv_rows_mean=n_mean, image_restarts=restarts,
               host_enqueue_ms_per_step=host_s * 1e3 / K, split_plan=eng.plan(), split_pin=eng.plan_pin(),
               roofline={"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBPS,
                         "traffic": recorded_traffic(args.workload) if default_step_config(args) else None,
                         "kernel": "sjd_step (window forward + verification + KV commit)",
                         "bytes_per_launch": total, "weight_bytes": weights, "kv_bytes": kv,
                         "logit_bytes": logit_b, "avg_launch_ms": avg_ms,
                         "bytes_moved_hilo_kv": moved,
                         "frac_hilo_kv": moved / (avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                         "mfma_tflops": 2.0 * weights / 2 * cfg["L"] * B / (avg_ms * 1e-3) / 1e12,
                         "mfma_frac": 2.0 * weights / 2 * cfg["L"] * B / (avg_ms * 1e-3) / 2.5e15})
    eng.close()
    del w
    torch.cuda.empty_cache()
    if not getattr(args, "calibrate_copy", False):
        with_measured(res["roofline"])
    if cpu and not args.no_cpu_baseline and B == 1 and not guided:
        res["cpu_baseline"] = cpu_baseline_step(args, cfg, seed, n_mean, prompt)
    return res


def cpu_baseline_step(args, cfg, seed, n_target, gpu_prompt):
    """The oracle (plain C, fp64 accumulation, OpenMP over output rows and
    heads) on the same model (weights regenerated from the same seed) and
    the same kind of step (window forward + verification of the context's
    window), on all host cores, plus a one-thread figure.

    Small models (tiny, mid): the GPU line's context is prefilled (untimed)
    and a few steps are timed at its cache length. Large models (7b, 8b): a
    full prefill of the GPU line's ~1240 or ~4160 tokens would take minutes,
    so one step is timed after a 64-token prefill and scaled by the step's
    flop count to the GPU line's mean fill (only the attention grows with
    it: +5% at 1240 rows on the 7B shape); labelled as extrapolated.
    One thread: a one-layer slice (same shapes, same LM head) is timed on
    one thread and on all threads; the ratio scales the all-thread step."""
    import numpy as np
    import torch

    from oracle import oracle as orc
    from oracle.harness import causal, oracle_model, oracle_prefill, placeholders, weights_numpy
    from synth_inputs import model_weights

    w = model_weights(cfg, 1, device="cuda" if torch.cuda.is_available() else "cpu")
    w = dict(embed=w["embed"].cpu(), final_norm=w["final_norm"].cpu(), lm_head=w["lm_head"].cpu(),
             layers=[{k: v.cpu() for k, v in l.items()} for l in w["layers"]])
    if torch.cuda.is_available():
        torch.cuda.empty_cache()
    w_np = weights_numpy(w)
    L, V = cfg["L"], cfg["V"]
    spine = placeholders(orc, cfg, seed)
    cores = all_threads()
    large = cfg["d_model"] >= 4096

    def one_step(m, n, pending):
        t0 = time.perf_counter()
        logits = m.forward(n, [int(pending)] + spine[:L - 1], [n + i for i in range(L)], causal(L))
        meta = np.array([[0, 0, 0, 0]], np.int32)
        r = orc.verify(logits[None], logits[None], np.array([spine], np.int32), meta, K=cfg["K"], D=cfg["D"],
                       top_k=cfg["top_k"], T=cfg["temperature"], flags=cfg.get("flags", 3) & 3, seed=seed,
                       step=0, vis_lo=cfg["vis_lo"], eol_id=cfg["eol_id"], row_len=cfg["row_len"])
        return time.perf_counter() - t0, int(r["meta"][0, 0])

    prompt = gpu_prompt.cpu().numpy().astype(np.int32)
    with omp_threads(cores):
        if large:
            m = oracle_model(orc, cfg, w_np, max_seq=160)
            n = oracle_prefill(m, prompt[:65])
            t1, nc = one_step(m, n, prompt[n])
            m.close()
            nc = float(nc)

            def flops(rows):
                # GEMMs (every weight once per slot) + attention over the
                # cached rows and the window
                d, H, Hkv, hd, F = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim"))
                params = cfg["n_layers"] * (2 * H * hd * d + 2 * Hkv * hd * d + 3 * F * d) + V * d
                return 2.0 * params * L + 4.0 * cfg["n_layers"] * H * hd * L * (rows + L / 2)

            t_step = t1 * flops(n_target) / flops(n)
            how = (f"one SJD-PAC step (32-slot window forward + verification) timed after a {n}-token prefill: "
                   f"{t1:.1f} s on {cores} threads ({cpu_model()}); scaled by the step's flop count to the GPU "
                   f"line's mean cache of {n_target:.0f} rows (only the attention grows with it): "
                   f"{t_step:.1f} s per step (extrapolated)")
        else:
            m = oracle_model(orc, cfg, w_np)
            n = oracle_prefill(m, prompt)
            reps = 3 if cfg["d_model"] >= 1024 else 8
            dts, ncs = [], []
            for _ in range(reps):
                dt, c = one_step(m, n, prompt[n])
                dts.append(dt)
                ncs.append(c)
            m.close()
            t_step = float(np.mean(dts))
            nc = float(np.mean(ncs))
            how = (f"{reps} SJD-PAC steps (window forward + verification) at the GPU line's cache of {n} rows, "
                   f"{t_step:.2f} s per step on {cores} threads ({cpu_model()})")
    # one thread: a one-layer slice of the same shapes (and the same LM
    # head) over a 4-slot window, on one thread and on all of them
    one = dict(cfg, n_layers=1)
    w1 = dict(w_np, layers=w_np["layers"][:1])
    times = {}
    for th in (cores, 1):
        with omp_threads(th):
            m = oracle_model(orc, one, w1, max_seq=128)
            oracle_prefill(m, prompt[:65])
            t0 = time.perf_counter()
            m.forward(64, [int(prompt[64])] + spine[:3], [64 + i for i in range(4)], causal(4))
            times[th] = time.perf_counter() - t0
            m.close()
    ratio = times[1] / times[cores]
    return {"value": nc / t_step, "unit": "image tokens/s", "cores": cores, "kind": "oracle", "sample": how,
            "step_s": t_step,
            "one_thread": {"value": nc / (t_step * ratio), "unit": "image tokens/s", "cores": 1,
                           "sample": f"one-layer slice, 4-slot window forward: {times[1]:.2f} s on 1 thread vs "
                                     f"{times[cores]:.2f} s on {cores}; the all-thread step scaled by that ratio "
                                     f"({ratio:.1f}x, extrapolated)"}}


# ---------------------------------------------------------------------------- sweep (ablation, K/D/L grid)
def run_sweep(args):
    """Ablation modes and the drafting tree / window grid (Tabs. 2-3 of the
    paper) on a small model where random-init weights still accept tokens:
    whole generations of the workload's image from its prompt, per
    configuration: mean committed tokens per step, the n_c histogram and the
    step time. One JSON line per configuration."""
    import numpy as np
    import torch

    from paper_2603_18599_amd.sjd import Engine
    from synth_inputs import model_config, model_weights, prompt_tokens

    grid = []
    for mode in ("sjd", "ac", "pd", "sjd-pac"):
        grid.append((mode, 32, 4, 3))
    for L in (32, 64):
        for K in (2, 3, 4, 5):
            for D in (2, 3, 4):
                grid.append(("sjd-pac", L, K, D))
    base = model_config(args.workload)
    w = model_weights(base, 1, device="cuda")
    prompt = prompt_tokens(base, 2).cuda()
    for mode, L, K, D in grid:
        flags = {"sjd-pac": 3, "sjd": 0, "ac": 1, "pd": 2}[mode]
        if mode in ("sjd", "ac"):
            K, D = 1, 0
        if K * D > L:
            continue
        cfg = model_config(args.workload, L=L, K=K, D=D, flags=flags)
        eng = Engine(cfg, w)
        meta = torch.zeros(8, dtype=torch.int32, device="cuda")
        ncs, ms = [], []
        for img in range(args.sweep_images):
            eng.prefill(prompt, 100 + img)
            gen, t = 0, 0
            ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            while gen < cfg["n_gen"]:
                ev0.record()
                eng.step(cfg["temperature"], cfg["top_k"], 100 + img, t, out_meta=meta)
                ev1.record()
                torch.cuda.synchronize()
                n_c = int(meta[0])
                ncs.append(n_c)
                ms.append(ev0.elapsed_time(ev1))
                gen += n_c
                t += 1
        eng.close()
        print(json.dumps({"workload": args.workload, "mode": mode, "L": L, "K": K, "D": D,
                          "images": args.sweep_images, "steps": len(ncs), "mean_accept_length": float(np.mean(ncs)),
                          "nc_hist": nc_histogram(ncs, L), "step_ms": float(np.median(ms))}), flush=True)


def section(res, keys=("value", "unit", "ms_per_step", "mean_accept_length", "nc_hist", "step_latency_ms",
                       "kv_rows_mean", "config", "roofline", "cpu_baseline")):
    return {k: res[k] for k in keys if k in res}


def main():
    args = parse()
    if args.traffic_from:
        traffic_from(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only (one process, one device); "
                                   "--gpus must be 1"}))
        sys.exit(2)
    if args.sweep:
        run_sweep(args)
        return
    if args.workload == "verify":
        res = bench_verify(args)
    else:
        res = bench_step(args)
        quick = argparse.Namespace(**dict(vars(args), steps=10, warmup=2))
        if not args.no_verify:
            v = bench_verify(quick, cpu=not args.no_cpu_baseline)
            res["verify"] = section(v, ("value", "unit", "ms_per_step", "mean_accept_length", "nc_hist",
                                        "expected_accept_length", "expected_accept_length_over_drafts",
                                        "verify_GBps", "roofline", "config", "cpu_baseline", "parity_sample"))
        if args.workload == "7b" and args.batch == 1 and args.cfg_w == 0.0 and not args.no_configs \
                and not args.calibrate_copy:
            # the other decoder shapes of the byte model, each with its own
            # oracle baseline
            for wl in ("tiny", "mid", "8b"):
                r = bench_step(argparse.Namespace(**dict(vars(args), workload=wl)))
                res[wl] = section(r)
        # several streams per forward (images, or guided pairs) take windows
        # of at most 32 slots; a longer window skips those sections
        multi = args.L <= 32
        if args.batch == 1 and not args.no_batch2 and not args.calibrate_copy and multi:
            # the same workload with two and four images per step (serving
            # several requests per weight pass)
            for nb in (2, 4):
                bn = bench_step(argparse.Namespace(**dict(vars(args), batch=nb)), cpu=False)
                res[f"batch{nb}"] = section(bn)
        if args.batch == 1 and args.cfg_w == 0.0 and not args.no_guided and not args.calibrate_copy and multi:
            # the paper's sampling setting: guidance weight 3 (Sec. 5.1), both streams in one forward
            gd = bench_step(argparse.Namespace(**dict(vars(args), cfg_w=3.0)), cpu=False)
            res["guided"] = section(gd)
            if not args.no_batch2:
                # two guided images per step (four streams in one forward)
                gd2 = bench_step(argparse.Namespace(**dict(vars(args), cfg_w=3.0, batch=2)), cpu=False)
                res["guided_batch2"] = section(gd2)

    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
