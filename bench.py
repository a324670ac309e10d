"""Throughput of the fused DendSN forward + backward scan on one MI355X.

One step = dendsn_forward + dendsn_backward over one batch of the layer
(default: the CIFAR-shaped spiking-conv activation, T=4, batch 128, C=128,
32x32 maps, 8 branches, fp32).  Inputs are synthetic (seeded normal draws) and
already resident in HBM when timing starts.  Prints one JSON line.

The rate is neuron-branch-steps per second: T * N * B / (time of one step).
The roofline object is for the dominant kernel (the backward scan): its
algorithmic bytes per launch divided by its mean launch time, timed with HIP
events on the stream the kernels run on, each timed call preceded by an untimed
512 MiB scratch read that evicts the MALL (so the bytes come from HBM), against
MI355X's 8 TB/s HBM peak; the same calls back to back are reported as
"unflushed".
"""

from __future__ import annotations

import argparse
import hashlib
import json
import multiprocessing as mp
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FLUSH_BYTES = 512 << 20   # untimed scratch read before each per-launch timed call: evicts the 256 MB MALL


def pmc_summary_path(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"pmc_dendsn_bwd_{workload}.txt")


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2412_06355_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if not name.endswith((".hip", ".h")):  # sources only (no caches or editor files)
            continue
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(digest: str, workload: str, key: str = "hbm_bytes_per_launch"):
    """HBM bytes per backward launch (key "fwd_hbm_bytes_per_launch": per forward
    launch) from the committed rocprofv3 counter summary of this workload, or None
    when there is none or the kernels changed since."""
    path = pmc_summary_path(workload)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.strip().split("=", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_src_sha256_16") != digest or vals.get("workload") != workload:
        return None
    try:
        return float(vals[key])
    except (KeyError, ValueError):
        return None


# ---------------------------------------------------------------------------
# CPU baseline: the float64 oracle, timed on a bounded sample of the workload
# ---------------------------------------------------------------------------
def _oracle_chunk(args):
    import numpy as np

    import oracle

    (T, C, S, B, k, x_mean, x_std, alpha, beta, vth, psi, sg, sg_scale, stateful, residual, seed) = args
    rng = np.random.default_rng(seed)
    N = C * S
    X = rng.normal(x_mean, x_std, size=(T, N, B * k))
    gS = rng.normal(size=(T, N))
    kappa = rng.uniform(0.0, 1.0, size=(C, B))
    t0 = time.perf_counter()
    rec = oracle.forward(X, alpha=alpha if stateful else 0.0, beta=beta, v_th=vth, kappa=kappa, C=C, S=S,
                         psi_kind=psi, stateful=stateful, residual=residual, comps_per_branch=k)
    oracle.backward(rec, gS, sg_kind=sg, sg_scale=sg_scale)
    return time.perf_counter() - t0, T * N * B


def _warm(_):
    import numpy  # noqa: F401

    import oracle  # noqa: F401

    return os.getpid()


def cpu_baseline(wl, target_nbs: float):
    """Oracle fwd+bwd throughput on a bounded sample: whole batch items of the
    layer (about target_nbs neuron-branch-steps), one task per item, spread
    over a process pool of up to 16 host cores; timed after the pool is up."""
    per_item = wl.T * wl.C * wl.S * wl.P
    items = int(max(1, min(wl.batch, round(target_nbs / per_item))))
    workers = int(min(16, len(os.sched_getaffinity(0)), items))
    args = [(wl.T, wl.C, wl.S, wl.B, wl.comps_per_branch, wl.x_mean, wl.x_std, wl.alpha, wl.beta, wl.v_th,
             wl.psi, wl.sg, wl.sg_scale, wl.stateful, wl.residual, 1000 + i) for i in range(items)]
    with mp.get_context("spawn").Pool(workers) as pool:
        pool.map(_warm, range(workers))
        t0 = time.perf_counter()
        res = pool.map(_oracle_chunk, args, chunksize=1)
        wall = time.perf_counter() - t0
    nbs = sum(r[1] for r in res)
    cpu_s = sum(r[0] for r in res)
    return {
        "value": nbs / wall,
        "unit": "neuron-branch-steps/s",
        "cores": workers,
        "kind": "oracle",
        "sample": f"{items} of {wl.batch} batch items of the layer (T={wl.T}, C={wl.C}, S={wl.S}, B={wl.B}, "
                  f"P={wl.P}), "
                  f"{nbs} neuron-branch-steps, float64 numpy forward+backward, one task per item on "
                  f"{workers} processes; {cpu_s:.1f} CPU-s in {wall:.2f} s wall",
    }


# ---------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=30)  # the clocks ramp over the first ~30 ms of work
    ap.add_argument("--workload", default="cifar")
    ap.add_argument("--batch-groups", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-nbs", type=float, default=4e8, help="oracle sample size")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 5 plain device copies of MIB MiB (scales the HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the library runs the "
              "DendSN scan on a single GPU.", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n * 4, "copy_calibration_bytes_written": n * 4,
                          "dispatches": 5}), flush=True)
        return

    import paper_2412_06355_amd as dendsn
    import workloads

    wl = workloads.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = dendsn.DendSNConfig(T=wl.T, batch=wl.batch, C=wl.C, S=wl.S, B=wl.B, stateful=wl.stateful,
                              detach_reset=wl.detach_reset, ckpt_every=wl.ckpt_every, io=wl.io, psi=wl.psi,
                              sg=wl.sg, sg_scale=wl.sg_scale, beta=wl.beta, v_th=wl.v_th,
                              batch_groups=args.batch_groups, comps_per_branch=wl.comps_per_branch,
                              residual=wl.residual, layout=wl.layout)
    X, gS = workloads.activations(wl, device=dev, seed=0)
    p = workloads.params(wl, seed=0)
    kappa = torch.from_numpy(p["kappa"]).to(dev)
    alpha = torch.tensor([wl.alpha], dtype=torch.float32, device=dev)
    masks = None
    if wl.tasks:
        masks = [torch.from_numpy(workloads.branch_mask(wl.C, wl.B, q, wl.mask_rho)).to(dev)
                 for q in range(1, wl.tasks + 1)]
    io_dt = X.dtype
    spikes = torch.empty((wl.T, wl.N), dtype=io_dt, device=dev)
    nck_bytes = dendsn.dendsn_ckpt_bytes(cfg)
    ckpt = torch.empty((max(1, nck_bytes // 4),), dtype=torch.float32, device=dev) if nck_bytes else None
    gX = torch.empty_like(X)
    g_alpha = torch.empty((1,), dtype=torch.float32, device=dev)
    g_beta = torch.empty((1,), dtype=torch.float32, device=dev)
    g_kappa = torch.empty_like(kappa)
    g_xi = torch.empty((wl.C, wl.P), dtype=torch.float32, device=dev)
    g_zeta = torch.empty_like(kappa)
    ws = torch.empty(((dendsn.dendsn_bwd_workspace_bytes(cfg) + 3) // 4,), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    tasks = masks if masks is not None else [None]

    def step():
        # one step: forward + backward of the layer (every task's mask for the gated layer)
        for m in tasks:
            dendsn.dendsn_forward(cfg, X, alpha, None, kappa, None, None, m, spikes, None, ckpt)
            dendsn.dendsn_backward(cfg, X, alpha, None, kappa, None, None, m, ckpt, gS, None, gX, g_alpha,
                                   g_beta, g_kappa, g_xi, g_zeta, ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)

    # whole-step timing: K steps between two events, synchronized on both sides
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    t_start.record(stream)
    for _ in range(args.steps):
        step()
    t_end.record(stream)
    torch.cuda.synchronize(dev)
    ms_per_step = t_start.elapsed_time(t_end) / args.steps

    # per-launch timing of each kernel call, with HIP events on the stream the
    # kernels run on.  Flushed (the default figures): before each timed call an
    # untimed read of 512 MiB of scratch (twice the 256 MB MALL) evicts whatever
    # the cache held, and writes back any dirty lines outside the timed region,
    # so every byte a call reads comes from HBM.  Unflushed: the calls back to
    # back, as in the whole step (a layer whose tensors fit the MALL may hit in it).
    flush_buf = torch.zeros((FLUSH_BYTES // 4,), dtype=torch.float32, device=dev)

    def timed_calls(flush: bool):
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps * len(tasks))]
        it = iter(evs)
        torch.cuda.synchronize(dev)
        for i in range(args.steps):
            for m in tasks:
                e = next(it)
                if flush:
                    flush_buf.sum()
                e[0].record(stream)
                dendsn.dendsn_forward(cfg, X, alpha, None, kappa, None, None, m, spikes, None, ckpt)
                e[1].record(stream)
                if flush:
                    flush_buf.sum()
                e[2].record(stream)
                dendsn.dendsn_backward(cfg, X, alpha, None, kappa, None, None, m, ckpt, gS, None, gX, g_alpha,
                                       g_beta, g_kappa, g_xi, g_zeta, ws)
                e[3].record(stream)
        torch.cuda.synchronize(dev)
        fwd = sum(e[0].elapsed_time(e[1]) for e in evs) / len(evs)
        bwd = sum(e[2].elapsed_time(e[3]) for e in evs) / len(evs)
        return fwd, bwd

    fwd_ms, bwd_ms = timed_calls(flush=True)
    fwd_ms_nf, bwd_ms_nf = timed_calls(flush=False)
    del flush_buf

    # sanity of the last outputs: spikes are exact 0/1, gradients finite
    sp = spikes.float()
    ok = bool(((sp == 0) | (sp == 1)).all().item()) and bool(torch.isfinite(gX.float()).all().item())
    rate = float(sp.mean().item())

    esz = X.element_size()
    nbs = wl.T * wl.N * wl.B
    ncs = wl.T * wl.N * wl.P                                        # compartment-steps: elements of X
    ck = nck_bytes
    fwd_bytes = ncs * esz + wl.T * wl.N * esz + ck                  # read X, write S, write checkpoints
    bwd_bytes = 2 * ncs * esz + wl.T * wl.N * esz + ck              # read X and gS, write gX, read checkpoints
    digest = kernel_source_digest()
    traffic = measured_traffic(digest, wl.name)
    bwd_gbs = bwd_bytes / (bwd_ms * 1e-3) / 1e9
    fwd_gbs = fwd_bytes / (fwd_ms * 1e-3) / 1e9
    n_tasks = len(tasks)
    value = nbs * n_tasks / (ms_per_step * 1e-3)

    out = {
        "metric": "DendSN fwd+bwd neuron-branch-steps/sec (T*N*B/s) and % of peak HBM GB/s",
        "value": value,
        "unit": "neuron-branch-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if wl.io == "f32" else "bf16 storage, f32 arithmetic",
        "data": "synthetic",
        "config": {"workload": wl.name, "T": wl.T, "batch": wl.batch, "C": wl.C, "S": wl.S, "B": wl.B,
                   "P": wl.P, "layout": wl.layout, "N": wl.N, "io": wl.io, "psi": wl.psi, "surrogate": f"{wl.sg}({wl.sg_scale})",
                   "dendrite": ("res" if wl.residual else "") + ("stateful" if wl.stateful else "stateless"),
                   "alpha": wl.alpha, "beta": wl.beta, "v_th": wl.v_th, "ckpt_every": wl.K,
                   "tasks": n_tasks},
        "roofline": {"bound": "hbm", "kernel": "dendsn_backward (scan + finalize)",
                     "achieved": bwd_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": bwd_gbs / HBM_PEAK_GBS, "traffic": traffic,
                     "algorithmic_bytes_per_launch": bwd_bytes, "ms_per_launch": bwd_ms,
                     "timing": "512 MiB scratch read (MALL eviction) before each timed call",
                     "unflushed": {"ms_per_launch": bwd_ms_nf,
                                   "frac": bwd_bytes / (bwd_ms_nf * 1e-3) / 1e9 / HBM_PEAK_GBS}},
        "roofline_fwd": {"achieved": fwd_gbs, "frac": fwd_gbs / HBM_PEAK_GBS, "unit": "GB/s",
                         "traffic": measured_traffic(digest, wl.name, "fwd_hbm_bytes_per_launch"),
                         "algorithmic_bytes_per_launch": fwd_bytes, "ms_per_launch": fwd_ms,
                         "unflushed": {"ms_per_launch": fwd_ms_nf,
                                       "frac": fwd_bytes / (fwd_ms_nf * 1e-3) / 1e9 / HBM_PEAK_GBS}},
        "step_hbm_frac": (fwd_bytes + bwd_bytes) * n_tasks / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "outputs_ok": ok,
        "firing_rate": rate,
        "kernel_src": digest,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_nbs)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
