"""Benchmark: contrastive-decoding tree verification on one MI355X.

One step = one dcd_verify_greedy call (LM heads of both models, softmax
partials and candidates, mask + cd score + argmax + log Z per row, draft-token
statistics, tree walk) over one Llama-3-8B/1B-shaped 64-node draft tree with
every input resident in HBM.  Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload b8_tree64]
                  [--theta T] [--mode greedy|sample|propose] [--final-norm]
                  [--no-cpu-baseline] [--no-probes] [--calibrate-copy BYTES]

The default is the greedy verification of the workload.  --mode sample times
dcd_verify_sample on the workload's tree (chains or trees; proposals from the
expert's parent-row logits plus noise, as the tests draw them), --mode propose
times dcd_propose on the workload's two heads, and --final-norm makes every call
start with the models' final RMS normalisation.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA, TFLOP/s

METRIC = "verified draft nodes/sec (8B/1B-shaped, 64-node tree); % of HBM peak"
# the same metric on the other workloads, named by what each is
METRICS = {
    "b8_tree64": METRIC,
    "tiny_chain8": "verified draft nodes/sec (tiny fp32 chain of 8 nodes)",
    "s8_chain16x8": "verified draft nodes/sec (8B/1B-shaped, 16 sampled chains of 8 nodes); % of HBM peak",
    "b8_batch32x64": "verified draft nodes/sec (8B/1B-shaped, 32 x 64-node trees); % of MFMA peak",
    "b70_tree64": "verified draft nodes/sec (70B/8B-shaped, 64-node tree); % of HBM peak",
}


def algorithmic_bytes(case) -> int:
    """Bytes the method must move per verification: each LM head once, the hidden
    states, both bias vectors, the tree inputs and the outputs."""
    esz = 2 if case.dtype == "bf16" else 4
    R, V = case.R, case.V
    weights = V * (case.dp + case.dq) * esz
    hidden = R * (case.dp + case.dq) * esz
    bias = 2 * V * 4
    tree_io = R * 4 * 2 + R * 4 + case.B * 4 * 3   # parents, tokens, path, len/next/status
    return weights + hidden + bias + tree_io


def lmhead_bytes(case) -> int:
    """Algorithmic bytes of the LM-head kernel alone: weights, hidden states, biases."""
    esz = 2 if case.dtype == "bf16" else 4
    return case.V * (case.dp + case.dq) * esz + case.R * (case.dp + case.dq) * esz + 2 * case.V * 4


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="b8_tree64")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--theta", type=float, default=None,
                    help="override the workload's plausibility cutoff (0 = untruncated target)")
    ap.add_argument("--mode", choices=("greedy", "sample", "propose"), default=None,
                    help="what to time (default: the workload's own mode)")
    ap.add_argument("--final-norm", action="store_true",
                    help="start every call with the models' final RMS normalisation")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probes", action="store_true",
                    help="skip the measured read-bandwidth and MFMA-rate ceilings")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes 10 times (for "
                         "scaling the HBM byte counters of a profiler run) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the verification step runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.calibrate_copy:
        src = torch.ones(args.calibrate_copy // 4, dtype=torch.int32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": src.numel() * 4, "copies": 10}), flush=True)
        return

    from paper_2608_12913_amd import dcd, synth
    from paper_2608_12913_amd.runner import DeviceProblem

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    over = {} if args.theta is None else {"theta": args.theta}
    case = synth.make_case(args.workload, args.seed, **over)
    mode = args.mode or case.mode
    own_mode = mode == case.mode
    if mode == "sample" and case.mode != "sample":  # the drafter's noise and draws
        case = synth.make_case(args.workload, args.seed, mode="sample", **over)
    log(f"{args.workload}: B={case.B} N={case.N} V={case.V} dp={case.dp} dq={case.dq} "
        f"mode={mode} final_norm={args.final_norm}")
    norm = {}
    if args.final_norm:
        # the synthetic rows taken as the models' last states before their final norm
        rng = np.random.default_rng(args.seed + 1)
        for key, d in (("norm_p", case.dp), ("norm_q", case.dq)):
            norm[key] = synth.bf16_bits((1 + 0.1 * rng.standard_normal(d)).astype(np.float32)) \
                if case.dtype == "bf16" else (1 + 0.1 * rng.standard_normal(d)).astype(np.float32)
        norm["norm_eps"] = 1e-5

    stream = torch.cuda.current_stream()
    probs = None
    if mode == "sample":
        # proposals of node i: softmax(z_p of its parent row + N(0,1)), its token drawn from it
        dev0 = DeviceProblem.from_case(case, np.zeros((case.B, case.N), np.int32), row_outputs=False)
        hp = dev0.hp.float()
        z = (hp @ dev0.wp.float().T + dev0.bias_p).double().cpu().numpy()
        del hp, dev0
        parents = case.parents.reshape(-1) + np.repeat(np.arange(case.B) * case.N, case.N)
        parent_logits = z[np.maximum(parents, 0)]
        probs, tokens = synth.sampled_draft(case, parent_logits)
        dev = DeviceProblem.from_case(case, tokens, draft_probs=probs, **norm)
    else:
        # draft tokens: half copy the target argmax of the parent row (taken from a first
        # verification call on the GPU), half are uniform; in a tree, the nodes of one
        # deepest path all copy it, so the walk accepts a full-depth path
        dev = DeviceProblem.from_case(case, np.zeros((case.B, case.N), np.int32), **norm)
        first = dev.run("greedy")
        tokens = synth.greedy_tokens(case, first["row_argmax"], spine=case.cfg["tree"] == "tree")
        dev.set_tokens(tokens)
    if mode == "propose":
        u = torch.from_numpy(case.u_res.astype(np.float32)).to(dev.device)
        ptoks = torch.empty(case.R, dtype=torch.int32, device=dev.device)
        pargmax = torch.empty(case.R, dtype=torch.int32, device=dev.device)
        pprobs = torch.empty(case.R, case.V, dtype=torch.float32, device=dev.device)

        def step():
            dcd.propose(dev.problem, dev.inputs, u, ptoks, pprobs, pargmax, dev.workspace,
                        dev.ws_bytes, stream)
    else:
        def step():
            dev.launch(mode, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K full steps
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = ev0.elapsed_time(ev1) / args.steps
    out = dev.run("greedy" if mode == "propose" else mode)

    norm_cost = None
    if args.final_norm and mode != "propose":
        # the normalisation's own cost: the same step without the flag on rows already
        # normalised the same way (fp32 statistics, bf16 roundings; the last bit of an
        # element may differ from the library's, which does not matter for timing)
        plain = {}
        for key, hkey, d in (("hp", "norm_p", case.dp), ("hq", "norm_q", case.dq)):
            x = getattr(case, key)
            xf = synth.bf16_to_f32(x) if case.dtype == "bf16" else np.asarray(x, np.float32)
            gf = synth.bf16_to_f32(norm[hkey]) if case.dtype == "bf16" else norm[hkey]
            r = (1.0 / np.sqrt(np.mean(xf * xf, axis=1, dtype=np.float32) + np.float32(norm["norm_eps"])))
            t = xf * r[:, None].astype(np.float32)
            if case.dtype == "bf16":
                plain[key] = synth.bf16_bits(gf[None, :] * synth.bf16_to_f32(synth.bf16_bits(t)))
            else:
                plain[key] = (gf[None, :] * t).astype(np.float32)
        dev_plain = DeviceProblem.from_case(case, tokens, draft_probs=probs, **plain)
        for _ in range(args.warmup):
            dev_plain.launch(mode, stream)
        torch.cuda.synchronize()
        p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        p0.record(stream)
        for _ in range(args.steps):
            dev_plain.launch(mode, stream)
        p1.record(stream)
        torch.cuda.synchronize()
        ms_plain = p0.elapsed_time(p1) / args.steps
        del dev_plain
        norm_cost = {"step_us_without_norm": round(ms_plain * 1e3, 2),
                     "cost_us": round((ms_step - ms_plain) * 1e3, 2)}
        log(f"final normalisation: step {ms_step * 1e3:.1f} us with it, {ms_plain * 1e3:.1f} us "
            f"on the same rows normalised beforehand")

    # the dominant kernel alone (LM heads + partials), same stream, HIP events
    lm_mode = "greedy" if mode == "greedy" else "sample"
    for _ in range(5):
        dev.launch_lmhead(lm_mode, stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        dev.launch_lmhead(lm_mode, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_lmhead = e0.elapsed_time(e1) / args.steps
    log(f"step {ms_step * 1e3:.1f} us, lm-head kernel {ms_lmhead * 1e3:.1f} us, "
        f"wall {wall:.3f} s, accept lengths {out['accept_len'].tolist()}")

    R = case.R
    nodes_per_s = R / (ms_step * 1e-3)
    kbytes = lmhead_bytes(case)
    flops = 2 * R * (case.dp + case.dq) * case.V
    # many rows (bf16, with or without the mask) go to the compute-shaped LM-head kernel
    kernel = "lmhead_wide_kernel" if case.dtype == "bf16" and R >= 512 else "lmhead_kernel"
    ridge = MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    # committed counters: per kernel and workload, and per mode and theta where they
    # differ from the workload's own
    variant = "" if own_mode and not over else f"_{mode}_theta{case.theta:g}"
    traffic, traffic_src = (counted_traffic(kernel, args.workload + variant)
                            if not args.final_norm else (None, "no counters for this workload"))
    if case.dtype == "bf16" and flops / kbytes > ridge:
        achieved = flops / (ms_lmhead * 1e-3) / 1e12
        roofline = dict(bound="mfma", achieved=round(achieved, 1), peak=MFMA_BF16_PEAK_TFLOPS,
                        unit="TFLOP/s", frac=round(achieved / MFMA_BF16_PEAK_TFLOPS, 4))
    else:
        achieved = kbytes / (ms_lmhead * 1e-3) / 1e9
        roofline = dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                        frac=round(achieved / HBM_PEAK_GBS, 4))
    roofline.update(traffic=traffic, kernel=kernel, algorithmic_bytes=kbytes, flops=flops,
                    avg_us=round(ms_lmhead * 1e3, 2), traffic_source=traffic_src)
    util = counted_utilisation(kernel, args.workload + variant) if not args.final_norm else None
    if util:
        roofline["counters"] = util
    if not args.no_probes:
        measured = measured_ceilings(torch, stream, log)
        roofline["measured_peak"] = measured
        key = "mfma_bf16_TFLOPs" if roofline["bound"] == "mfma" else "stream_read_GBs"
        roofline["frac_of_measured"] = round(roofline["achieved"] / measured[key], 4)

    cpu = None
    if mode != "greedy" or args.final_norm:
        log("cpu baseline: only for the greedy verification of the workload's own rows")
    elif not args.no_cpu_baseline:
        cpu = cpu_baseline(case, tokens, log)
        cpu["single_core"] = cpu_single_core(case, tokens, log)

    step_bytes = algorithmic_bytes(case)
    metric = METRICS.get(args.workload, f"verified draft nodes/sec ({args.workload})")
    line = {
        "metric": metric if mode != "propose" else "proposal rows/sec (recombined heads)",
        "value": round(nodes_per_s, 1),
        "unit": "nodes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if case.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "batch": case.B, "nodes": case.N, "vocab": case.V,
                   "d_expert": case.dp, "d_amateur": case.dq, "plaus_thresh": case.theta,
                   "cd_strength": case.s, "rows": R, "seed": args.seed, "mode": mode,
                   "final_norm": bool(args.final_norm)},
        "hbm_frac_step": round(step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        # rows scored per second without the roots (each sequence's root is the last
        # committed token, not a drafted one), and what the timed calls accepted
        "drafted_nodes_per_s": round((R - case.B) / (ms_step * 1e-3), 1),
        "accept_len": out["accept_len"].tolist() if mode != "propose" else None,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if norm_cost:
        line["final_norm_cost"] = norm_cost
    print(json.dumps(line), flush=True)


def measured_ceilings(torch, stream, log):
    """What this device delivers to a plain streaming read (4 GiB, far above the
    256 MB MALL) and to a register-only bf16 MFMA loop (include/dcd_probe.h), each
    timed with HIP events on the bench stream."""
    from paper_2608_12913_amd import dcd

    def timed(fn, n):
        fn()
        fn()  # the first launches also ramp the clocks
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n * 1e-3

    nbytes = 4 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    sink = torch.zeros(256 * 1024, dtype=torch.float32, device="cuda:0")
    t_read = timed(lambda: dcd.probe_stream_read(buf, nbytes, sink, stream), 10)
    del buf
    wg, iters = 1024, 4000
    flops = dcd.probe_mfma_bf16(wg, iters, sink, stream)
    t_mfma = timed(lambda: dcd.probe_mfma_bf16(wg, iters, sink, stream), 5)
    out = {"stream_read_GBs": round(nbytes / t_read / 1e9, 1),
           "mfma_bf16_TFLOPs": round(flops / t_mfma / 1e12, 1)}
    log(f"measured ceilings: {out}")
    return out


def code_sha256(root, rels):
    """SHA-256 of the code of the listed sources: comments, blank lines and the
    indentation of lines removed, so that a change to comments alone keeps committed
    counters valid."""
    import hashlib
    import re

    h = hashlib.sha256()
    for rel in rels:
        text = open(os.path.join(root, rel), encoding="utf-8").read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        for line in text.splitlines():
            line = line.strip()
            if line:
                h.update(line.encode() + b"\n")
    return h.hexdigest()


def read_profile_fields(path, root):
    """The key: value fields of a committed profiler summary, or None when the code of
    its listed sources no longer hashes to the recorded digest."""
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith(" "):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    rels = fields.get("sources", "").split()
    if not rels or code_sha256(root, rels) != fields.get("sources_code_sha256"):
        return None
    return fields


def counted_utilisation(kernel, workload):
    """MFMA-busy and LDS-busy fractions of the LM-head kernel and its waves' wait
    share, from the committed SQ-counter summary of this kernel and workload (None when
    there is none or the kernel has changed since)."""
    root = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(root, "profiles", f"{kernel}_{workload}_sq_counters.txt")
    if not os.path.exists(path):
        return None
    f = read_profile_fields(path, root)
    if f is None:
        return None
    return {"mfma_busy": float(f["mfma_busy"]), "lds_busy": float(f["lds_busy"]),
            "wave_wait": float(f["wave_wait"]), "source": os.path.relpath(path, root)}


def counted_traffic(kernel, workload):
    """HBM bytes per LM-head launch from the committed profiler counter summary of this
    kernel and workload, or None when there is none or the kernel sources have changed
    since the counters were taken."""
    root = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(root, "profiles", f"{kernel}_{workload}_hbm_counters.txt")
    if not os.path.exists(path):
        return None, "no counters for this workload"
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith(" "):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    rels = fields.get("sources", "").split()
    if not rels or code_sha256(root, rels) != fields.get("sources_code_sha256"):
        return None, "stale counters (kernel changed since they were taken)"
    fetch = float(fields["fetch_kib_per_dispatch"]) * float(fields["fetch_scale"])
    write = float(fields["write_kib_per_dispatch"]) * float(fields["write_scale"])
    return round((fetch + write) * 1024.0), os.path.relpath(path, root)


def cpu_baseline(case, tokens, log, min_seconds=10.0):
    """The oracle, untuned, on the host cores: complete verifications of the same
    workload (every row's LM heads in fp64, mask, cd target, walk), repeated until
    min_seconds have passed; the rate is the mean over the repetitions."""
    import oracle

    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    hp, hq = oracle.as_f32(case.hp), oracle.as_f32(case.hq)
    wp, wq = oracle.as_f32(case.wp), oracle.as_f32(case.wq)
    log(f"cpu baseline: oracle over {case.R} rows on {threads} threads")
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.verify("greedy", case.B, case.N, hp, hq, wp, wq, case.bias, case.bias,
                      case.parents, tokens, theta=case.theta, s=case.s, nthreads=threads)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    log(f"cpu baseline: {reps} verifications in {dt:.2f} s")
    return {"value": round(reps * case.R / dt, 3), "unit": "nodes/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{reps} full {case.name} verifications ({case.R} rows each, fp64 "
                      f"oracle) in {dt:.2f} s"}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_single_core(case, tokens, log, max_macs=8e9):
    """The oracle on one thread: complete verifications when one takes at most
    max_macs multiply-adds, else the first rows of the workload (the LM-head dot
    products are nearly all of a row's work and the walk is negligible), timed and
    scaled to nodes/s."""
    import oracle

    hp, hq = oracle.as_f32(case.hp), oracle.as_f32(case.hq)
    wp, wq = oracle.as_f32(case.wp), oracle.as_f32(case.wq)
    per_row = case.V * (case.dp + case.dq)
    t0 = time.perf_counter()
    if per_row * case.R <= max_macs:
        oracle.verify("greedy", case.B, case.N, hp, hq, wp, wq, case.bias, case.bias,
                      case.parents, tokens, theta=case.theta, s=case.s, nthreads=1)
        n, what = case.R, f"1 full {case.name} verification ({case.R} rows)"
    else:
        n = max(1, int(max_macs // per_row))
        oracle.eval_rows(hp, hq, wp, wq, case.bias, case.bias, theta=case.theta, s=case.s,
                         rows=np.arange(n), nthreads=1)
        what = f"the first {n} of {case.R} rows of {case.name} (row evaluation only)"
    dt = time.perf_counter() - t0
    log(f"cpu baseline, 1 thread: {what} in {dt:.2f} s")
    return {"value": round(n / dt, 3), "unit": "nodes/s", "cores": 1,
            "sample": f"{what} in {dt:.2f} s"}


if __name__ == "__main__":
    main()
