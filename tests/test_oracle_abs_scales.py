"""Pins of the oracle's term scales A = sum |terms| (``abs_kappa``, ``abs_xi``,
``abs_zeta``, ``abs_alpha``, ``abs_beta``), the scale against which the parity
tests judge each summed parameter gradient's rounding error.

A parameter shared by many uses (kappa by every step, batch item and position of
its channel; alpha by every step and compartment; beta by every step and
neuron) has a gradient that is the sum of one term per use.  Giving each use its
own leaf in float64 autograd of the forward equations (Methods, "Dendritic
spiking neuron"; the surrogate of Eq. methods-sg) yields those terms one by one,
independently of the oracle's backward; their absolute values summed per
channel are A.  Two facts of A itself are checked as well: A >= |g| entry by
entry (triangle inequality), and A = |g| when every term has one sign.
"""

import math

import numpy as np
import pytest

import oracle
from oracle import PSI_IDENTITY, PSI_MEXHAT, SG_ATAN, SG_SIGMOID


def _case(rng, *, T=5, batch=2, C=3, S=2, B=3, k=1, psi_kind=PSI_MEXHAT, stateful=True, mask=True,
          residual=False):
    N, P = batch * C * S, B * k
    return dict(X=rng.normal(0.0, 1.2, size=(T, N, P)), kappa=rng.uniform(0.3, 1.3, size=(C, B)),
                xi=rng.normal(0.0, 0.5, size=(C, P)), zeta=rng.uniform(0.5, 2.0, size=(C, B)),
                mask=(rng.random((C, B)) < 0.6).astype(np.uint8) if mask else None,
                gS=rng.normal(size=(T, N)), gV=rng.normal(size=(T, N)), C=C, S=S, k=k, psi_kind=psi_kind,
                stateful=stateful, residual=residual, alpha=0.6, beta=0.7, v_th=1.0)


def _oracle(case, sg_kind, sg_scale, detach):
    rec = oracle.forward(case["X"], alpha=case["alpha"], beta=case["beta"], v_th=case["v_th"],
                         kappa=case["kappa"], xi=case["xi"], zeta=case["zeta"], mask=case["mask"],
                         C=case["C"], S=case["S"], psi_kind=case["psi_kind"], stateful=case["stateful"],
                         residual=case["residual"], comps_per_branch=case["k"])
    return oracle.backward(rec, case["gS"], case["gV"], sg_kind=sg_kind, sg_scale=sg_scale,
                           detach_reset=detach)


def per_use_terms(case, sg_kind, sg_scale, detach):
    """Float64 autograd of the forward with one leaf per use of each parameter:
    kappa, zeta [T, N, B], xi and alpha [T, N, P], beta [T, N].  Returns the
    gradient of every leaf, i.e. every term of every parameter gradient."""
    import torch

    f64 = torch.float64
    X = torch.tensor(case["X"], dtype=f64)
    T, N, P = X.shape
    k = case["k"]
    B = P // k
    C, S = case["C"], case["S"]
    cidx = torch.as_tensor((np.arange(N) // S) % C)
    m = torch.tensor(np.ones((C, B)) if case["mask"] is None else (case["mask"] != 0) * 1.0, dtype=f64)
    leaf = lambda a: a.clone().detach().requires_grad_(True)
    kap = leaf(torch.tensor(case["kappa"], dtype=f64)[cidx].expand(T, N, B))
    xi = leaf(torch.tensor(case["xi"], dtype=f64)[cidx].expand(T, N, P))
    zet = leaf(torch.tensor(case["zeta"], dtype=f64)[cidx].expand(T, N, B))
    alp = leaf(torch.full((T, N, P), case["alpha"], dtype=f64))
    bet = leaf(torch.full((T, N), case["beta"], dtype=f64))

    class Spike(torch.autograd.Function):
        @staticmethod
        def forward(ctx, x):
            ctx.save_for_backward(x)
            return (x >= 0).to(x.dtype)

        @staticmethod
        def backward(ctx, g):
            (x,) = ctx.saved_tensors
            if sg_kind == SG_ATAN:
                return g / (1.0 + (math.pi * x) ** 2)
            sig = torch.sigmoid(sg_scale * x)
            return g * sg_scale * sig * (1.0 - sig)

    vd = torch.zeros(N, P, dtype=f64)
    h = torch.zeros(N, dtype=f64)
    s = torch.zeros(N, dtype=f64)
    loss = torch.zeros((), dtype=f64)
    gS, gV = torch.tensor(case["gS"]), torch.tensor(case["gV"])
    for t in range(T):
        vd = alp[t] * vd + X[t] if case["stateful"] else X[t]
        dv = vd - xi[t]
        nrm = torch.abs(dv) if k == 1 else torch.linalg.vector_norm(dv.reshape(N, B, k), dim=2)
        u = nrm / zet[t]
        y = (1 - u ** 2) * torch.exp(-u ** 2 / 2) if case["psi_kind"] == PSI_MEXHAT else u
        z = (kap[t] * m[cidx] * y).sum(dim=1)
        if case["residual"]:
            z = z + X[t].mean(dim=1)
        h = bet[t] * (1 - (s.detach() if detach else s)) * h + z
        s = Spike.apply(h - case["v_th"])
        loss = loss + (gS[t] * s).sum() + (gV[t] * h).sum()
    loss.backward()
    g = lambda a: np.zeros(tuple(a.shape)) if a.grad is None else a.grad.numpy()
    return dict(kappa=g(kap), xi=g(xi), zeta=g(zet), alpha=g(alp), beta=g(bet))


def _per_channel(a, case):
    """[T, N, W] -> [C, W]: sum over time, batch items and positions."""
    T, N, W = a.shape
    C, S = case["C"], case["S"]
    return a.reshape(T, N // (C * S), C, S, W).sum(axis=(0, 1, 3))


@pytest.mark.parametrize("psi_kind", [PSI_MEXHAT, PSI_IDENTITY])
@pytest.mark.parametrize("sg_kind", [SG_ATAN, SG_SIGMOID])
@pytest.mark.parametrize("detach", [False, True])
@pytest.mark.parametrize("stateful,residual,k", [(True, False, 1), (False, True, 1), (True, True, 2),
                                                 (False, False, 3)])
def test_abs_scales_are_sums_of_per_use_term_magnitudes(psi_kind, sg_kind, detach, stateful, residual, k):
    rng = np.random.default_rng(31)
    case = _case(rng, k=k, psi_kind=psi_kind, stateful=stateful, residual=residual)
    g = _oracle(case, sg_kind, 3.0, detach)
    terms = per_use_terms(case, sg_kind, 3.0, detach)
    for name in ("kappa", "xi", "zeta"):
        A = _per_channel(np.abs(terms[name]), case)
        assert np.allclose(g["abs_" + name], A, rtol=1e-11, atol=1e-14), name
        # the terms also sum to the gradient itself
        assert np.allclose(g["g_" + name], _per_channel(terms[name], case), rtol=1e-10, atol=1e-13), name
    A_alpha = float(np.abs(terms["alpha"]).sum()) if stateful else 0.0
    assert math.isclose(g["abs_alpha"], A_alpha, rel_tol=1e-11, abs_tol=1e-14)
    assert math.isclose(g["abs_beta"], float(np.abs(terms["beta"]).sum()), rel_tol=1e-11, abs_tol=1e-14)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_abs_scales_bound_the_gradients(seed):
    rng = np.random.default_rng(seed)
    case = _case(rng, T=6, B=4, k=1 + seed % 2, residual=seed == 3)
    g = _oracle(case, SG_SIGMOID, 4.0, False)
    for name in ("kappa", "xi", "zeta"):
        assert np.all(g["abs_" + name] >= np.abs(g["g_" + name])), name
    assert g["abs_alpha"] >= abs(g["g_alpha"]) and g["abs_beta"] >= abs(g["g_beta"])
    # with mixed signs the bound is strict somewhere (A is not |g| by construction)
    assert np.any(g["abs_kappa"] > np.abs(g["g_kappa"]) * (1 + 1e-9))


def test_abs_scales_equal_the_gradients_when_every_term_has_one_sign():
    """Identity psi, xi < 0 < X (so d = Vd - xi > 0), gS >= 0, gV > 0 and the reset
    detached (so dS = gS): every dH > 0, and the terms of g_kappa (m dH Y, Y = u > 0),
    g_alpha (lam Vd), g_beta (dH H) are positive, those of g_xi (-r) and g_zeta
    (-g_u u / zeta) negative.  A threshold above most potentials keeps the reset factor
    (1 - S) of g_beta's terms nonzero.  Then A = |g| (the same numbers summed, up to
    rounding)."""
    rng = np.random.default_rng(5)
    T, batch, C, S, B = 6, 2, 3, 2, 4
    N = batch * C * S
    case = dict(X=rng.uniform(0.1, 1.0, size=(T, N, B)), kappa=rng.uniform(0.3, 1.3, size=(C, B)),
                xi=-rng.uniform(0.1, 0.5, size=(C, B)), zeta=rng.uniform(0.5, 2.0, size=(C, B)), mask=None,
                gS=rng.uniform(0.0, 1.0, size=(T, N)), gV=rng.uniform(0.1, 1.0, size=(T, N)), C=C, S=S, k=1,
                psi_kind=PSI_IDENTITY, stateful=True, residual=False, alpha=0.6, beta=0.7, v_th=8.0)
    g = _oracle(case, SG_ATAN, 4.0, True)
    assert np.all(g["g_kappa"] > 0) and np.all(g["g_xi"] < 0) and np.all(g["g_zeta"] < 0)
    for name in ("kappa", "xi", "zeta"):
        assert np.allclose(g["abs_" + name], np.abs(g["g_" + name]), rtol=1e-14, atol=0), name
    assert g["g_alpha"] > 0 and math.isclose(g["abs_alpha"], g["g_alpha"], rel_tol=1e-14)
    assert g["g_beta"] > 0 and math.isclose(g["abs_beta"], g["g_beta"], rel_tol=1e-14)
