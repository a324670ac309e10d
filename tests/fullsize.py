"""Per-batch-item oracle check for the full-size parity tests (runs in worker
processes).  Neurons of different batch items are independent in both
directions, so item b of a layer is checked on its own: spikes (forced-spike
protocol) and the norm-wise errors of v_soma and grad_x; their elementwise
errors, the kernel's and a plain float32 evaluation's, and the item's
parameter-gradient contributions are returned, to be judged and summed over all
items (judge_elementwise; sums in float64)."""

from __future__ import annotations

import numpy as np

import oracle
from tests import fp32_eval
from tests.parity import BAND, RTOL_F32, tolerance


def _open(spec):
    path, shape = spec
    return np.memmap(path, dtype=np.float32, mode="r", shape=tuple(shape))


def check_item(job: dict) -> dict:
    b, M, T = job["item"], job["M"], job["T"]
    sl = slice(b * M, (b + 1) * M)
    X = np.asarray(_open(job["X"])[:, sl, :], dtype=np.float64)
    gS = np.asarray(_open(job["gS"])[:, sl], dtype=np.float64)
    S_g = np.asarray(_open(job["S"])[:, sl], dtype=np.float64)
    H_g = np.asarray(_open(job["H"])[:, sl], dtype=np.float64)
    gX_g = np.asarray(_open(job["gX"])[:, sl, :], dtype=np.float64)
    p = job["params"]
    kw = dict(alpha=p["alpha"], beta=p["beta"], v_th=p["v_th"], kappa=p["kappa"], xi=p["xi"], zeta=p["zeta"],
              mask=p["mask"], C=p["C"], S=p["S"], psi_kind=p["psi"], stateful=p["stateful"],
              residual=p["residual"], comps_per_branch=p["k"])
    # forced-spike protocol: impose the kernel's decision only where the oracle's
    # potential is within BAND of the threshold
    force = -np.ones((T, M), dtype=np.int64)
    exempt = 0
    for _ in range(T + 1):
        rec = oracle.forward(X, force=force if exempt else None, **kw)
        diff = rec["S"] != S_g
        if not diff.any():
            break
        cols = np.nonzero(diff.any(axis=0))[0]
        t_first = diff[:, cols].argmax(axis=0)
        dist = np.abs(rec["H"][t_first, cols] - p["v_th"])
        if np.any(dist > BAND):
            i = int(np.argmax(dist > BAND))
            return dict(item=b, error=f"item {b}: spike mismatch outside the band at t={t_first[i]}, "
                                      f"neuron {cols[i]}: |H - v_th| = {dist[i]:.3e}")
        force[t_first, cols] = S_g[t_first, cols].astype(np.int64)
        exempt += len(cols)
    else:
        return dict(item=b, error=f"item {b}: forced-spike protocol did not converge")
    g = oracle.backward(rec, gS, sg_kind=p["sg"], sg_scale=p["sg_scale"], detach_reset=p["detach"])
    # a plain float32 evaluation of the same equations on this item's inputs and
    # spike train: what float32 arithmetic itself needs here (tests/parity.py)
    r32 = fp32_eval.evaluate(X, rec["S"], gS, alpha=p["alpha"], beta=p["beta"], v_th=p["v_th"], kappa=p["kappa"],
                             xi=p["xi"], zeta=p["zeta"], mask=p["mask"], C=p["C"], S=p["S"], psi=p["psi"],
                             stateful=p["stateful"], residual=p["residual"], k=p["k"], sg=p["sg"],
                             sg_scale=p["sg_scale"], detach=p["detach"])
    out = dict(item=b, error=None, exempt=exempt)
    # elementwise errors of this item's outputs (scale: |o| + rms over the item),
    # the kernel's and the float32 evaluation's; judged over all items together
    # (judge_elementwise), since a bound is set by the whole tensor's worst element
    for name, got, ref, f32, rtol in (("v_soma", H_g, rec["H"], r32["H"], RTOL_F32),
                                      ("grad_x", gX_g, g["gX"], r32["gX"], job["rtol_io"])):
        out["gpu_" + name] = fp32_eval.elementwise_ratio(got, ref)
        out["fp32_" + name] = fp32_eval.elementwise_ratio(f32, ref)
        den = np.linalg.norm(ref)
        nrel = float(np.linalg.norm(got - ref) / den) if den > 0 else 0.0
        if nrel > rtol:
            out["error"] = f"item {b}: {name} norm-wise error {nrel:.3e}"
            return out
    for k in ("kappa", "xi", "zeta", "alpha", "beta"):
        out["g_" + k] = g["g_" + k]
        out["abs_" + k] = g["abs_" + k]
        out["f32_" + k] = r32["g_" + k]      # this item's float32 sums
    return out


def judge_elementwise(res: list, rtol_io: float) -> list:
    """The elementwise bounds over all checked items: the kernel's worst element
    of each tensor against tolerance(rtol, the float32 evaluation's worst element
    of the same tensor).  Returns the failures (empty when every bound holds)."""
    errors = []
    for name, rtol in (("v_soma", RTOL_F32), ("grad_x", rtol_io)):
        gpu = max(r["gpu_" + name] for r in res)
        e32 = max(r["fp32_" + name] for r in res)
        tol = tolerance(rtol, e32)
        if gpu > tol:
            worst = max(res, key=lambda r: r["gpu_" + name])["item"]
            errors.append(f"{name}: worst error/scale {gpu:.3e} (item {worst}) > {tol:.3g} "
                          f"(float32 evaluation: {e32:.3e})")
    return errors
