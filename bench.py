"""Throughput of the pose-inversion hot path on one MI355X.

A step is one pass of the whole hot path over one batch: render -> Huber loss
-> pose gradient for K hypotheses (pnerf_render_loss_grad), the pose update
(pnerf_step_momentum, or pnerf_step_adam at the setting of Sec. IV-D with
--optimizer adam) and, at the workload's resampling interval, Monte Carlo
resampling (pnerf_resample_hypotheses).  Inputs (field, observation, pixel
batches, poses) are resident in HBM before timing starts.

Prints one JSON line.  value = ray-samples/s (samples composited and
back-propagated to the pose gradient, summed over the timed steps, divided by
the timed wall time).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2210_10108_amd import synth  # noqa: E402

PEAK_BF16_MFMA = 2.5e15       # MI355X dense bf16 MFMA, FLOP/s (the MLP kernels' instructions)
PEAK_HBM = 8.0e12             # MI355X HBM3E, bytes/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    # default: the largest single-GPU workload (1024 x 512 rays in the [-2,2]^3
    # box, T = 2^21, 256^3 occupancy, up to 2048 samples per ray)
    ap.add_argument("--workload", default="large4m_occ256", choices=synth.ORDER)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--optimizer", default="momentum", choices=("momentum", "adam"),
                    help="pose update: the workload's momentum SGD, or Adam with the "
                         "learning rates and decay of Sec. IV-D")
    ap.add_argument("--sh-dir-grad", type=int, default=0, choices=(0, 1),
                    help="1: also carry the gradient through the view-direction (SH) input")
    ap.add_argument("--paper-run", action="store_true",
                    help="instead of the step benchmark, time one whole pose estimate: the "
                         "Monte Carlo schedule of Sec. IV-B/IV-D (64 hypotheses, 2560 Adam "
                         "steps, 4 resampling rounds) on the workload's field and pixel count")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-calibration", action="store_true",
                    help="skip the on-box copy and bf16 GEMM reference rates")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--backward", type=int, default=0, choices=(0, 1),
                    help="0: separate composite, network backward and reduction kernels; "
                         "1: the fused per-ray backward kernel")
    ap.add_argument("--graph", action="store_true",
                    help="also record one step (loss gradient + optimizer step) into a HIP graph "
                         "and time its replays (workloads without resampling whose batch fits "
                         "one sample buffer)")
    ap.add_argument("--mlp-precision", type=int, default=0, choices=(0, 1),
                    help="0: split-bf16 MFMA (three products, fp32-equivalent); "
                         "1: fp16 MFMA (one product, fp32 accumulation)")
    ap.add_argument("--overlap-chunks", type=int, default=0,
                    help="field option: loss-gradient chunks pipelined over two streams "
                         "(0 = library default, 1 = off)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first run a plain device copy of this many MiB (3 times), whose "
                         "FETCH_SIZE / WRITE_SIZE calibrate the profiler's byte counters")
    return ap.parse_args()


def render_observation(field, w, gt, dev):
    """Observed image = the field rendered at the ground-truth pose (HIP path)."""
    import torch
    n = w.width * w.height
    out = torch.empty(n, 3, dtype=torch.float32, device=dev)
    chunk = 1 << 16
    pose = torch.from_numpy(gt[None]).to(dev)
    intr = synth.intrinsics(w)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        ids = torch.arange(s, e, dtype=torch.int32, device=dev)[None]
        out[s:e] = field.render(pose, ids, intr)[0]
    return out.reshape(w.height, w.width, 3)


def graph_replay(field, w, obs, intr, pix, fresh, adam, loss, dpose, S, W):
    """One step -- the loss gradient and the momentum step -- recorded into a
    HIP graph by stream capture and replayed W + S times from the initial
    poses (S timed), each replay's pixel ids copied into the recorded buffer
    first: the eager steps' work without a host launch per kernel."""
    import torch
    from paper_2210_10108_amd import pnerf
    if w.resample_every:
        return {"unsupported": "the workload resamples between steps"}
    if adam is not None:
        return {"unsupported": "the Adam step takes its step number from the host"}
    poses, mom = fresh()
    pix_buf = pix[0].clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    try:
        with torch.cuda.graph(g):
            field.render_loss_grad(poses, pix_buf, obs, intr, loss, dpose)
            pnerf.step_momentum(poses, mom, dpose, w.lr, w.beta)
    except pnerf.PnerfError as e:
        torch.cuda.synchronize()
        return {"unsupported": str(e)}
    for i in range(W):
        pix_buf.copy_(pix[i % len(pix)])
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(W, W + S):
        pix_buf.copy_(pix[i % len(pix)])
        g.replay()
    torch.cuda.synchronize()
    return {"ms_per_step": (time.perf_counter() - t0) / S * 1e3}


def dtype_label(w, args):
    """The path's arithmetic: fp32 (or fp16-stored) table and weights, fp32
    encoding and compositing, and the networks' MFMA arithmetic."""
    storage = "f16-storage" if w.param_dtype == "f16" else "f32"
    return storage + ("+f16-mfma" if args.mlp_precision else "+split-bf16x3-mfma")


def measured_traffic(workload, kernel_key):
    """HBM bytes per launch of one kernel from the committed rocprofv3 counter
    summary (profiles/traffic_<workload>.md), or None when there is none or the
    kernel sources have changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    if "```json" not in text:
        return None
    rec = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    src = os.path.join(ROOT, "paper_2210_10108_amd", "csrc")
    h = hashlib.sha256()
    for fn in sorted(os.listdir(src)):
        with open(os.path.join(src, fn), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != rec.get("csrc_sha256"):
        return None
    k = rec["kernels"].get(kernel_key)
    return None if k is None else k["fetch_bytes"] + k["write_bytes"]


def cpu_baseline(w, spec, gt, poses, pix_batches, budget_s):
    """The oracle, untuned, on a bounded sample of the same workload: whole
    hypotheses (all P pixels of one batch each), cycling through the pixel
    batches, until about `budget_s` seconds of timed work.  The oracle renders
    its own observation and builds its own occupancy grid (both untimed)."""
    import dataclasses
    from oracle import oracle as O
    threads = O.n_threads_default()
    intr = synth.intrinsics(w)
    if spec.occ_res > 0 and spec.occ_bits is None:
        plain = O.OracleField(dataclasses.replace(spec, occ_res=0, occ_bits=None))
        bits = plain.build_occupancy(spec.occ_res, spec.occ_threshold, threads=threads)
        spec = dataclasses.replace(spec, occ_bits=bits)
    of = O.OracleField(spec)
    done_s, samples, hyps = 0.0, 0, 0
    while done_s < budget_s and hyps < w.K * len(pix_batches):
        k, b = hyps % w.K, hyps // w.K
        pix = pix_batches[b][k:k + 1]
        obs = np.zeros((w.height, w.width, 3), np.float32)
        flat = np.unique(pix)
        obs.reshape(-1, 3)[flat] = of.render(gt[None], flat[None].astype(np.int32), intr,
                                             threads=threads)[0]
        t0 = time.perf_counter()
        out = of.render_loss_grad(poses[k:k + 1], pix, obs, intr, threads=threads)
        done_s += time.perf_counter() - t0
        samples += int(out["march"][0][-1])
        hyps += 1
    # the same oracle on one thread, over one hypothesis
    pix = pix_batches[0][0:1]
    obs = np.zeros((w.height, w.width, 3), np.float32)
    flat = np.unique(pix)
    obs.reshape(-1, 3)[flat] = of.render(gt[None], flat[None].astype(np.int32), intr,
                                         threads=threads)[0]
    t0 = time.perf_counter()
    out = of.render_loss_grad(poses[0:1], pix, obs, intr, threads=1)
    one = int(out["march"][0][-1]) / (time.perf_counter() - t0)
    return {"value": samples / done_s, "unit": "ray-samples/s", "cores": threads,
            "kind": "oracle", "single_thread_value": one,
            "sample": f"{hyps} hypotheses x {w.P} pixels (of {w.K} per batch; "
                      f"{samples} samples, {done_s:.1f} s timed, fp64 oracle, {threads} threads)"}


def calibrate(dev):
    """On-box reference rates, reported beside the published peaks: a 1 GiB
    device-to-device copy (bytes read + written per second), a large bf16
    library GEMM (hipBLASLt through torch; 2 m n k flop per product), and
    random 16-byte reads counted at the 128-byte line each one fetches."""
    import torch
    out = {}
    n = (1 << 30) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    out["copy_TBps"] = 10 * 2 * n * 4 / (time.perf_counter() - t0) / 1e12
    del src, dst
    m = 8192
    a = torch.randn(m, m, dtype=torch.bfloat16, device=dev)
    b = torch.randn(m, m, dtype=torch.bfloat16, device=dev)
    for _ in range(3):
        c = a @ b
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(10):
        c = a @ b
    torch.cuda.synchronize()
    out["bf16_gemm_TFLOPs"] = 10 * 2 * m ** 3 / (time.perf_counter() - t0) / 1e12
    del a, b, c
    # random 16-byte reads from a table of `mib` MiB (torch's indexing kernel):
    # each touches its own 128-byte line, the encoding's pattern on its fine
    # levels; reported as lines fetched per second x 128 B
    n_idx = 1 << 24
    for mib in (256, 1024):
        table = torch.ones(mib * (1 << 20) // 16, 4, dtype=torch.float32, device=dev)
        g = torch.Generator(device=dev).manual_seed(0)
        idx = torch.randint(0, table.shape[0], (n_idx,), generator=g, device=dev)
        for _ in range(2):
            torch.index_select(table, 0, idx)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(10):
            torch.index_select(table, 0, idx)
        torch.cuda.synchronize()
        out[f"random_line_read_{mib}MiB_TBps"] = 10 * n_idx * 128 / (time.perf_counter() - t0) / 1e12
        del table, idx
    torch.cuda.empty_cache()
    return out


def paper_run(args):
    """One whole pose estimate with the paper's schedule (P_N = 64, s1 = s2 = 512,
    S = 4, r = 0.25 halved; Adam at 5e-3 / 3e-3 decaying by 0.33 per 256 steps),
    P pixels per hypothesis per step from 8 seeded batches in turn.  Prints one
    JSON line: wall seconds of the run, with its inputs resident in HBM."""
    import torch
    from paper_2210_10108_amd import driver, pnerf
    dev = torch.device("cuda:0")
    w = synth.WORKLOADS[args.workload]
    sched = driver.PAPER_SCHEDULE
    K = sched.n_hypotheses
    fa = synth.make_field(w, args.seed)
    field = pnerf.Field(synth.field_spec(w, fa, sh_dir_grad=args.sh_dir_grad),
                        backward=args.backward, mlp_precision=args.mlp_precision)
    gt = synth.ground_truth_pose(w, args.seed)
    obs = render_observation(field, w, gt, dev)
    poses0 = synth.perturb_poses(gt, K, w.max_rot_deg, w.max_trans, args.seed)
    pix = [torch.from_numpy(synth.pixel_batch(args.seed, i, K, w.P, w.width, w.height)).to(dev)
           for i in range(8)]
    intr = synth.intrinsics(w)
    sr = math.radians(w.resample_sigma_rot_deg)

    def run():
        poses = torch.from_numpy(poses0.copy()).to(dev)
        loss, _ = driver.invert(field, poses, obs, intr, lambda it: pix[it % 8], sched,
                                pnerf.AdamParams(), sigma_rot=sr,
                                sigma_trans=w.resample_sigma_trans, seed=args.seed)
        return poses, loss

    run()  # warm-up run
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    poses, loss = run()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    best = int(torch.argmin(loss).item())
    p = poses[best].cpu().numpy().astype(np.float64)
    rot_err = math.degrees(np.arccos(np.clip((np.trace(p[:, :3].T @ gt[:, :3]) - 1) / 2, -1, 1)))
    print(json.dumps({
        "metric": "seconds per pose estimate (paper schedule)", "value": elapsed, "unit": "s",
        "n_gpus": 1, "higher_is_better": False, "data": "synthetic",
        "dtype": dtype_label(w, args),
        "steps": sched.total_steps, "hypotheses": K,
        "hypothesis_iters_per_sec": K * sched.total_steps / elapsed,
        "config": {"workload": w.name, "P": w.P, "rays_per_step": K * w.P,
                   "optimizer": "adam (lr 5e-3 / 3e-3, decay 0.33 per 256 steps)",
                   "schedule": "P_N=64, s1=s2=512, S=4, r=0.25 halved"},
        "best_hypothesis": {"loss": float(loss[best].item()), "rotation_error_deg": rot_err,
                            "translation_error": float(np.linalg.norm(p[:, 3] - gt[:, 3]))}}))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path shards "
              "over hypotheses but no multi-GPU run is built", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2210_10108_amd import pnerf

    if args.paper_run:
        paper_run(args)
        return
    dev = torch.device("cuda:0")
    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    w = synth.WORKLOADS[args.workload]
    fa = synth.make_field(w, args.seed)
    spec = synth.field_spec(w, fa, sh_dir_grad=args.sh_dir_grad)  # occupancy built on the device
    field = pnerf.Field(spec, overlap_chunks=args.overlap_chunks, backward=args.backward,
                        mlp_precision=args.mlp_precision)
    gt = synth.ground_truth_pose(w, args.seed)
    obs = render_observation(field, w, gt, dev)
    poses0 = synth.perturb_poses(gt, w.K, w.max_rot_deg, w.max_trans, args.seed)
    n_batches = 8
    pix_host = [synth.pixel_batch(args.seed, i, w.K, w.P, w.width, w.height)
                for i in range(n_batches)]
    pix = [torch.from_numpy(p).to(dev) for p in pix_host]
    intr = synth.intrinsics(w)
    K = w.K
    loss = torch.empty(K, dtype=torch.float32, device=dev)
    dpose = torch.empty(K, 6, dtype=torch.float32, device=dev)
    sr = math.radians(w.resample_sigma_rot_deg)

    def run(n_steps, start, poses, mom, count=False, counts=None):
        for i in range(start, start + n_steps):
            field.render_loss_grad(poses, pix[i % n_batches], obs, intr, loss, dpose)
            if count:
                counts.append(field.last_sample_count())
            if adam is None:
                pnerf.step_momentum(poses, mom, dpose, w.lr, w.beta)
            else:
                pnerf.step_adam(poses, mom, dpose, i, adam)
            if w.resample_every and (i + 1) % w.resample_every == 0:
                pnerf.resample_hypotheses(poses, mom, loss, w.keep_frac, sr,
                                          w.resample_sigma_trans, args.seed,
                                          (i + 1) // w.resample_every)

    adam = pnerf.AdamParams() if args.optimizer == "adam" else None
    state_dim = 6 if adam is None else pnerf.ADAM_STATE

    def fresh():
        return (torch.from_numpy(poses0.copy()).to(dev),
                torch.zeros(K, state_dim, dtype=torch.float32, device=dev))

    W, S = args.warmup, args.steps
    # sample counts of the timed steps (deterministic replay, synchronising per step)
    poses, mom = fresh()
    counts = []
    run(W + S, 0, poses, mom, count=True, counts=counts)
    timed_samples = int(sum(counts[W:]))

    # timed run, with HIP events recorded around every kernel launch on the
    # stream it runs on (read once the clock has stopped): the per-kernel
    # times are those of the timed steps themselves
    poses, mom = fresh()
    run(W, 0, poses, mom)
    torch.cuda.synchronize()
    field.set_profiling(True)
    t0 = time.perf_counter()
    run(S, W, poses, mom)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = {name: {"launches": n, "avg_ms": ms / max(n, 1)} for name, n, ms in field.profile()}
    field.set_profiling(False)
    # the same steps again without the events: their cost on the device (a few
    # microseconds per launch) shows on workloads whose launches are short
    poses, mom = fresh()
    run(W, 0, poses, mom)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    run(S, W, poses, mom)
    torch.cuda.synchronize()
    elapsed_plain = time.perf_counter() - t1

    graph = None
    if args.graph:
        graph = graph_replay(field, w, obs, intr, pix, fresh, adam, loss, dpose, S, W)
        if "ms_per_step" in graph:
            graph["value"] = timed_samples / (graph["ms_per_step"] * 1e-3 * S)

    samples_per_step = timed_samples / S
    # roofline of every per-sample kernel: algorithmic units per sample x samples
    # per launch / average launch time (HIP events on the call's stream)
    elem = 2 if w.param_dtype == "f16" else 4
    gather_bytes = 8 * w.n_levels * w.n_features * elem      # one gather pass per sample
    din = w.n_levels * w.n_features
    # algorithmic multiply-accumulates per sample (input gradient only, frozen
    # field; the SH rows of the first colour layer count once per ray, not here):
    # density din*64 + 64*16, colour 16*64 + 64*64 + 64*3; backward colour
    # 3*64 + 64*64 + 64*15, density 16*64 + 64*din
    mac_fwd = din * 64 + 64 * 16 + 16 * 64 + 64 * 64 + 64 * 3
    mac_bwd = 3 * 64 + 64 * 64 + 64 * 15 + 16 * 64 + 64 * din
    # the MLP kernels run v_mfma_f32_16x16x32_bf16 on split (hi + lo) operands
    # (three bf16 products per fp32 product), or v_mfma_f32_16x16x32_f16 (two:
    # the weight's two fp16 parts times the fp16 activation); both priced
    # against the 16-bit peak
    units = {"encode": ("hbm", gather_bytes, PEAK_HBM, "GB/s", 1e9),
             "mlp_fwd": ("mfma", 2 * mac_fwd, PEAK_BF16_MFMA, "TFLOP/s", 1e12),
             "mlp_bwd": ("mfma", 2 * mac_bwd, PEAK_BF16_MFMA, "TFLOP/s", 1e12),
             "ray_bwd": ("mfma", 2 * mac_bwd, PEAK_BF16_MFMA, "TFLOP/s", 1e12)}
    rooflines = {}
    for kname, (bound, per, peak, unit, scale) in units.items():
        if kname not in prof:
            continue
        launches_per_step = prof[kname]["launches"] / S
        avg_s = prof[kname]["avg_ms"] * 1e-3
        ach = samples_per_step / launches_per_step * per / avg_s
        rooflines[kname] = {"bound": bound, "achieved": ach / scale, "peak": peak / scale,
                            "unit": unit, "frac": ach / peak, "traffic": None,
                            "avg_ms": prof[kname]["avg_ms"], "per_sample": per,
                            "_scale_bytes": 1e9 if bound == "hbm" else None}
        if bound == "mfma":
            # 16-bit products issued: three bf16 (split) or two fp16 (weights
            # as two parts) per fp32 product
            rooflines[kname]["executed_frac"] = (2 if args.mlp_precision else 3) * ach / peak
    dom_name = max(rooflines, key=lambda k: prof[k]["avg_ms"] * prof[k]["launches"])
    lpg = w.n_levels // 4
    tf = {0: "false", 1: "true"}
    h, dr = tf[args.mlp_precision], tf[args.sh_dir_grad]
    keys = {"encode": f"k_encode<{'true' if w.param_dtype == 'f16' else 'false'}, true>",
            "mlp_fwd": f"k_mlp_fwd<{lpg}, true, {h}>",
            "mlp_bwd": f"k_mlp_bwd<{lpg}, {dr}, {h}>",
            "ray_bwd": f"k_ray_bwd<{lpg}, {dr}, false, {h}>"}
    for kname, r in rooflines.items():
        tr = measured_traffic(w.name, keys[kname])
        # HBM bytes per launch (calibrated FETCH_SIZE + WRITE_SIZE), same units as achieved
        if tr is not None and r["_scale_bytes"]:
            r["traffic"] = tr / (r["avg_ms"] * 1e-3) / r["_scale_bytes"]
        r["traffic_bytes_per_launch"] = tr
    for r in rooflines.values():
        if r["_scale_bytes"] is None:
            r["traffic"] = None  # an MFMA kernel: traffic in GB/s is given under traffic_GBps
            tb = r.pop("traffic_bytes_per_launch", None)
            r["traffic_GBps"] = None if tb is None else tb / (r["avg_ms"] * 1e-3) / 1e9
        else:
            r.pop("traffic_bytes_per_launch", None)
        r.pop("_scale_bytes")
    roof = dict(kernel=dom_name, **rooflines[dom_name])

    res = {
        "metric": "ray-samples/sec fwd+bwd to pose grads",
        "value": timed_samples / elapsed,
        "unit": "ray-samples/s",
        "n_gpus": 1,
        "steps": S,
        "warmup": W,
        "ms_per_step": elapsed / S * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the path's arithmetic: fp32 (or fp16-stored) table and weights, fp32
        # encoding and compositing; the MLPs as three bf16 MFMA products per fp32
        # product (hi*hi + hi*lo + lo*hi), accumulated in fp32
        "dtype": dtype_label(w, args),
        "mlp_arithmetic": ("fp16 MFMA (weights as two fp16 parts, activations rounded to fp16, "
                           "two products), fp32 accumulation" if args.mlp_precision else
                           "bf16 MFMA on split hi/lo operands (3 products), fp32 accumulation"),
        "data": ("synthetic (seeded random frozen field" +
                 ("" if w.density == "random" else ", density shaped as one object in empty space") +
                 "; observation rendered at a seeded ground-truth pose)"),
        "config": {"workload": w.name, "K": K, "P": w.P, "levels": w.n_levels,
                   "table": f"2^{w.log2_table}", "image": f"{w.width}x{w.height}",
                   "sampling": "uniform" if w.march_mode == 0 else "lattice+occupancy",
                   "optimizer": args.optimizer, "sh_dir_grad": args.sh_dir_grad,
                   "backward": "separate-kernels" if args.backward == 0 else "fused-per-ray",
                   "parallelism": "single-gpu"},
        "hypothesis_iters_per_sec": K * S / elapsed,
        "graph_replay": graph,
        "without_kernel_events": {"value": timed_samples / elapsed_plain,
                                  "ms_per_step": elapsed_plain / S * 1e3},
        "samples_per_step": samples_per_step,
        "mean_samples_per_ray": samples_per_step / w.n_rays,
        "roofline": roof,
        "kernel_rooflines": rooflines,
        "kernels_avg_ms": {k: v["avg_ms"] for k, v in prof.items()},
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, spec, gt, poses0, pix_host, args.cpu_seconds)
    if not args.no_calibration:
        res["calibration"] = calibrate(dev)
    field.close()
    print(json.dumps(res))


if __name__ == "__main__":
    main()
