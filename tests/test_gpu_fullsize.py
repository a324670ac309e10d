"""Parity at the benchmark's full layer sizes, in the launch configuration
bench.py times (same cfg, automatic batch groups): every batch item's spikes,
v_soma and grad_x are checked against the float64 oracle, run item by item in a
pool of host processes, and the parameter gradients against the oracle's sums
over all items.  Inputs are the benchmark's own seeded draws.  Tolerances are
those of tests/parity.py: rtol, or twice the error of a plain float32
evaluation of the same items where float32 itself cannot reach rtol (each
tensor's worst element over all items against the float32 evaluation's)."""

import multiprocessing as mp
import os

import numpy as np
import pytest

import paper_2412_06355_amd as dendsn
import workloads
from tests.fullsize import check_item, judge_elementwise
from tests import fp32_eval
from tests.parity import RTOL_BF16, RTOL_F32, announce, tolerance

pytestmark = pytest.mark.gpu


def _dump(t, path):
    a = t.float().cpu().numpy()
    mm = np.memmap(path, dtype=np.float32, mode="w+", shape=a.shape)
    mm[...] = a
    mm.flush()
    return (str(path), list(a.shape))


def _npb(t, wl):
    """X or grad_x in the oracle's [T, N, P] order: a channel-major tensor's memory
    is [T, batch, C, P, S], its compartments S elements apart."""
    if wl.layout != "channel_major":
        return t
    return t.reshape(wl.T, wl.batch, wl.C, wl.P, wl.S).permute(0, 1, 2, 4, 3).reshape(wl.T, wl.N, wl.P)


def _check_against_oracle(wl, cfg, X, gS, kappa, alpha, p, mask_np, xg_files, tmp_path, label):
    """Forward + backward of the layer on the GPU (mask_np: one task's gate, or
    None), then every batch item against the oracle in a pool of host processes
    and the parameter gradients against the oracle's sums over all items."""
    import torch

    dev = X.device
    mask = torch.from_numpy(mask_np).to(dev) if mask_np is not None else None
    # the forward as bench.py runs it (no v_soma), then again with v_soma for the
    # potential's comparison: the spikes and checkpoints agree bit for bit
    spikes, _, ckpt = dendsn.forward(cfg, X, alpha, kappa, None, None, mask)
    s2, v_soma, ck2 = dendsn.forward(cfg, X, alpha, kappa, None, None, mask, want_v_soma=True)
    assert torch.equal(s2.view(torch.uint8), spikes.view(torch.uint8))
    if ckpt is not None:
        assert torch.equal(ck2.view(torch.uint8), ckpt.view(torch.uint8))
    del s2, ck2
    g = dendsn.backward(cfg, X, alpha, kappa, None, None, mask, ckpt, gS)
    torch.cuda.synchronize(dev)
    files = dict(xg_files, S=_dump(spikes, tmp_path / "S.f32"), H=_dump(v_soma, tmp_path / "H.f32"),
                 gX=_dump(_npb(g["grad_x"], wl), tmp_path / "gX.f32"))
    grads = {k: g[k].cpu().numpy().astype(np.float64) for k in ("grad_kappa", "grad_xi", "grad_zeta")}
    g_alpha, g_beta = float(g["grad_alpha"].item()), float(g["grad_beta"].item())
    del spikes, v_soma, ckpt, g
    torch.cuda.empty_cache()

    params = dict(alpha=wl.alpha if wl.stateful else 0.0, beta=wl.beta, v_th=wl.v_th, kappa=p["kappa"],
                  xi=None, zeta=None, mask=mask_np, C=wl.C, S=wl.S, psi=wl.psi, stateful=wl.stateful,
                  residual=wl.residual, k=wl.comps_per_branch, sg=wl.sg, sg_scale=wl.sg_scale,
                  detach=wl.detach_reset)
    rtol_io = RTOL_BF16 if wl.io == "bf16" else RTOL_F32
    jobs = [dict(item=b, M=wl.C * wl.S, T=wl.T, params=params, rtol_io=rtol_io, **files) for b in range(wl.batch)]
    workers = int(min(16, len(os.sched_getaffinity(0)), wl.batch))
    with mp.get_context("spawn").Pool(workers) as pool:
        res = pool.map(check_item, jobs, chunksize=1)
    errors = [r["error"] for r in res if r["error"]]
    assert not errors, errors[:5]
    exempt = sum(r["exempt"] for r in res)
    announce(f"full-size parity {label}: {wl.batch} items, {exempt} near-threshold exemptions; worst elementwise "
             f"error/scale: v_soma {max(r['gpu_v_soma'] for r in res):.2e} (float32 evaluation "
             f"{max(r['fp32_v_soma'] for r in res):.2e}), grad_x {max(r['gpu_grad_x'] for r in res):.2e} "
             f"(float32 evaluation {max(r['fp32_grad_x'] for r in res):.2e})")
    errors = judge_elementwise(res, rtol_io)
    assert not errors, errors

    def summed(key):
        return sum(r[key] for r in res)

    def f32_sum(key):  # the float32 evaluation's per-item sums, added in float32
        acc = np.float32(0)
        for r in res:
            acc = acc + np.asarray(r[key], np.float32)
        return acc

    for k in ("kappa", "xi", "zeta"):
        o, a = summed("g_" + k), summed("abs_" + k)
        got = grads["grad_" + k]
        tol = tolerance(RTOL_F32, fp32_eval.summed_ratio(f32_sum("f32_" + k), o, a))
        scale = a + np.sqrt(np.mean(a * a))
        err = np.abs(got - o)
        assert np.all(err <= tol * scale), (k, float(np.max(err / scale)), tol)
        assert np.linalg.norm(got - o) <= RTOL_F32 * np.linalg.norm(o), k
    for k, got, on in (("alpha", g_alpha, wl.stateful), ("beta", g_beta, True)):
        if not on:
            continue
        o, a = summed("g_" + k), summed("abs_" + k)
        tol = tolerance(RTOL_F32, abs(float(f32_sum("f32_" + k)) - o) / a if a > 0 else 0.0)
        assert abs(got - o) <= tol * a, (k, got, o, a, tol)
    if mask_np is not None:
        off = mask_np == 0
        assert np.all(grads["grad_kappa"][off] == 0.0) and np.all(grads["grad_zeta"][off] == 0.0)
        assert np.all(grads["grad_xi"][np.repeat(off, wl.comps_per_branch, axis=1)] == 0.0)


# every benchmark layer (bench.py --workload W), in the launch configuration it
# times; the gated layer with each of its tasks' masks
@pytest.mark.parametrize("name", ["cifar", "imagenet_stem", "long_horizon", "dbg", "cifar_bf16", "cifar_p4b2",
                                  "cifar_p4b2_cm", "cifar_cm", "tiny_imagenet_res", "dvs_p10b5",
                                  "dvs_p10b5_stateful"])
def test_full_size_against_oracle(gpu_device, name, tmp_path):
    import torch

    wl = workloads.WORKLOADS[name]
    announce(f"full-size parity {name}: T={wl.T} batch={wl.batch} C={wl.C} S={wl.S} B={wl.B} {wl.io}")
    cfg = dendsn.DendSNConfig(T=wl.T, batch=wl.batch, C=wl.C, S=wl.S, B=wl.B, stateful=wl.stateful,
                              detach_reset=wl.detach_reset, ckpt_every=wl.ckpt_every, io=wl.io, psi=wl.psi,
                              sg=wl.sg, sg_scale=wl.sg_scale, beta=wl.beta, v_th=wl.v_th,
                              comps_per_branch=wl.comps_per_branch, residual=wl.residual, layout=wl.layout)
    X, gS = workloads.activations(wl, device=gpu_device, seed=0)
    p = workloads.params(wl, seed=0)
    kappa = torch.from_numpy(p["kappa"]).to(gpu_device)
    alpha = torch.tensor([wl.alpha], dtype=torch.float32, device=gpu_device)
    xg_files = dict(X=_dump(_npb(X, wl), tmp_path / "X.f32"), gS=_dump(gS, tmp_path / "gS.f32"))
    if not wl.tasks:
        _check_against_oracle(wl, cfg, X, gS, kappa, alpha, p, None, xg_files, tmp_path, name)
        return
    # Eq. methods-dbg-sampling: one fixed mask per task, q = 1 .. tasks, as bench.py times them
    for q in range(1, wl.tasks + 1):
        mask_np = workloads.branch_mask(wl.C, wl.B, q, wl.mask_rho)
        _check_against_oracle(wl, cfg, X, gS, kappa, alpha, p, mask_np, xg_files, tmp_path, f"{name} task {q}")
