"""Pins of the float64 oracle against facts that do not come from the oracle itself.

Each test fixes the oracle to something independent of its code: the exact
worked example in tests/golden (derived by hand from the paper's equations),
closed forms of the recurrences, textbook special cases (LIF), a separately
written scalar stepper, float64 autograd of the forward equations (for the
backward), and central finite differences of a smooth forward (also for the
backward).  A dropped term, a wrong sign, a transposed index or a wrong
parameter gather in ``oracle.forward`` / ``oracle.backward`` fails at least one.
"""

import math
import os

import numpy as np
import pytest

import oracle
from oracle import PSI_IDENTITY, PSI_MEXHAT, SG_ATAN, SG_SIGMOID

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# helpers written independently of the oracle
# ---------------------------------------------------------------------------
def load_worked_example():
    rows = {}
    with open(os.path.join(GOLDEN, "worked_example_forward.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, t, *vals = line.split()
            rows.setdefault(name, {})[int(t)] = [float(v) for v in vals]
    T = max(rows["X"])
    get = lambda k: np.array([rows[k][t] for t in range(1, T + 1)])
    return dict(X=get("X")[:, None, :], Vd=get("Vd"), Z=get("Z")[:, 0],
                H=get("H")[:, 0], S=get("S")[:, 0])


WORKED = dict(alpha=0.5, beta=0.5, v_th=1.0, kappa=np.array([[0.5, 0.25]]),
              xi=None, zeta=None, mask=None, C=1, S=1, psi_kind=PSI_IDENTITY)


def rand_case(rng, T=5, batch=2, C=3, S=2, B=3, psi_kind=PSI_MEXHAT, stateful=True,
              mask=False, scale=1.0, residual=False, k=1):
    """k compartments per branch: X is [T, N, B k], xi is [C, B k]."""
    N = batch * C * S
    X = rng.normal(0.0, scale, size=(T, N, B * k))
    kappa = rng.uniform(0.0, 1.0, size=(C, B)) + 0.3
    xi = rng.normal(0.0, 0.5, size=(C, B * k))
    zeta = rng.uniform(0.5, 2.0, size=(C, B))
    m = (rng.random((C, B)) < 0.6).astype(np.uint8) if mask else None
    gS = rng.normal(size=(T, N))
    gV = rng.normal(size=(T, N))
    return dict(X=X, kappa=kappa, xi=xi, zeta=zeta, mask=m, gS=gS, gV=gV, C=C, S=S,
                psi_kind=psi_kind, stateful=stateful, alpha=0.6, beta=0.7, v_th=1.0, residual=residual,
                k=k)


def run_oracle(case, force=None):
    return oracle.forward(case["X"], alpha=case["alpha"], beta=case["beta"], v_th=case["v_th"],
                          kappa=case["kappa"], xi=case["xi"], zeta=case["zeta"],
                          mask=case["mask"], C=case["C"], S=case["S"],
                          psi_kind=case["psi_kind"], stateful=case["stateful"],
                          residual=case.get("residual", False), comps_per_branch=case.get("k", 1),
                          force=force)


# ---------------------------------------------------------------------------
# Worked example (exact)
# ---------------------------------------------------------------------------
def test_worked_example_forward_exact():
    w = load_worked_example()
    rec = oracle.forward(w["X"], **WORKED)
    assert np.array_equal(rec["Vd"][1:, 0, :], w["Vd"])
    assert np.array_equal(rec["Z"][:, 0], w["Z"])
    assert np.array_equal(rec["H"][:, 0], w["H"])
    assert np.array_equal(rec["S"][:, 0], w["S"])


def test_worked_example_backward_by_hand():
    """Somatic adjoint of the worked example, atan surrogate, full reset gradient,
    gS = 1, gV = 0, worked out by hand from the reset-charge and fire equations:
    H - v_th = (0, -1/2, 1/2), so sg = (1, q, q) with q = 1/(1 + pi^2/4);
    dH3 = q;  dH2 = q (1 - beta H2 dH3) + beta dH3;  dH1 = 1 - beta H1 dH2 (S1 = 1 kills
    the leak term).  Branch 1 has Vd = 0 at t = 2, 3, so its gX there is 0 (sgn(0) = 0)."""
    w = load_worked_example()
    rec = oracle.forward(w["X"], **WORKED)
    g = oracle.backward(rec, np.ones((3, 1)), sg_kind=SG_ATAN)
    q = 1.0 / (1.0 + math.pi ** 2 / 4.0)
    dH3 = q
    dH2 = q * (1.0 - 0.5 * 0.5 * dH3) + 0.5 * dH3
    dH1 = 1.0 - 0.5 * 1.0 * dH2
    assert np.allclose(g["dH"][:, 0], [dH1, dH2, dH3], rtol=1e-14, atol=0)
    # gX: lam[t] = kappa dH sgn(Vd) + alpha lam[t+1], per branch.
    lam3 = np.array([0.5 * dH3, 0.0])
    lam2 = np.array([0.5 * dH2, 0.0]) + 0.5 * lam3
    lam1 = np.array([0.5 * dH1, 0.25 * dH1]) + 0.5 * lam2
    assert np.allclose(g["gX"][:, 0, :], [lam1, lam2, lam3], rtol=1e-14, atol=1e-300)
    assert g["gX"][1, 0, 1] == 0.0 and g["gX"][2, 0, 1] == 0.0
    # g_alpha = sum_t sum_b lam_b[t] Vd_b[t-1]
    ga = lam2 @ np.array([1.0, 2.0]) + lam3 @ np.array([1.0, 0.0])
    assert math.isclose(g["g_alpha"], ga, rel_tol=1e-14)
    # g_kappa = sum_t dH[t] Y[t]
    gk = dH1 * np.array([1, 2]) + dH2 * np.array([1, 0]) + dH3 * np.array([2.5, 0])
    assert np.allclose(g["g_kappa"][0], gk, rtol=1e-14)
    # g_beta = sum_t dH[t] (1 - S[t-1]) H[t-1]: only t = 3 counts (S[1] = 1 resets step 2)
    assert math.isclose(g["g_beta"], dH3 * 0.5, rel_tol=1e-14)


# ---------------------------------------------------------------------------
# Activation and surrogate: textbook values and derivatives
# ---------------------------------------------------------------------------
def test_mexican_hat_textbook_values():
    u = np.array([0.0, 1.0, math.sqrt(3.0)])
    y = oracle.psi(u, PSI_MEXHAT)
    assert y[0] == 1.0
    assert abs(y[1]) < 1e-16
    assert math.isclose(y[2], -2.0 * math.exp(-1.5), rel_tol=1e-15)  # the minimum
    dy = oracle.dpsi(u, PSI_MEXHAT)
    assert dy[0] == 0.0 and abs(dy[2]) < 1e-15
    # It is the negated second derivative of the Gaussian exp(-u^2/2).
    uu = np.linspace(-4, 4, 161)
    h = 1e-4
    g = lambda x: np.exp(-0.5 * x * x)
    second = (g(uu + h) - 2 * g(uu) + g(uu - h)) / h ** 2
    assert np.allclose(oracle.psi(np.abs(uu), PSI_MEXHAT), -second, atol=1e-7)
    assert np.array_equal(oracle.psi(uu, PSI_IDENTITY), uu)


@pytest.mark.parametrize("kind", [PSI_MEXHAT, PSI_IDENTITY])
def test_dpsi_is_derivative_of_psi(kind):
    u = np.linspace(0.01, 5.0, 300)
    h = 1e-6
    fd = (oracle.psi(u + h, kind) - oracle.psi(u - h, kind)) / (2 * h)
    assert np.allclose(oracle.dpsi(u, kind), fd, rtol=1e-7, atol=1e-9)


@pytest.mark.parametrize("kind,scale", [(SG_ATAN, 1.0), (SG_SIGMOID, 4.0), (SG_SIGMOID, 2.5)])
def test_surrogate_is_derivative_of_primitive(kind, scale):
    from scipy import integrate, special

    x = np.linspace(-3, 3, 241)
    if kind == SG_ATAN:
        F = lambda v: np.arctan(np.pi * v) / np.pi + 0.5
    else:
        F = lambda v: special.expit(scale * v)
    h = 1e-6
    fd = (F(x + h) - F(x - h)) / (2 * h)
    assert np.allclose(oracle.surrogate_grad(x, kind, scale), fd, rtol=1e-7, atol=1e-10)
    # A surrogate of Theta' integrates to the unit step height.
    tot, _ = integrate.quad(lambda v: float(oracle.surrogate_grad(np.array([v]), kind, scale)[0]),
                            -np.inf, np.inf, limit=200)
    assert math.isclose(tot, 1.0, rel_tol=1e-7)
    # Peak values: 1 for atan, a/4 for the sigmoid.
    peak = oracle.surrogate_grad(np.array([0.0]), kind, scale)[0]
    assert math.isclose(peak, 1.0 if kind == SG_ATAN else scale / 4.0, rel_tol=1e-15)
    # Far tails stay finite and tiny.
    tails = oracle.surrogate_grad(np.array([-800.0, 800.0]), kind, scale)
    assert np.all(np.isfinite(tails)) and np.all(tails < 1e-5)


# ---------------------------------------------------------------------------
# Closed forms of the recurrences
# ---------------------------------------------------------------------------
def test_dendrite_impulse_response_and_closed_form():
    T, alpha = 9, 0.8
    X = np.zeros((T, 1, 1))
    X[0, 0, 0] = 1.0
    rec = oracle.forward(X, alpha=alpha, beta=0.5, v_th=1e9, kappa=np.ones((1, 1)), C=1,
                         psi_kind=PSI_IDENTITY)
    assert np.allclose(rec["Vd"][1:, 0, 0], alpha ** np.arange(T), rtol=1e-15)
    rng = np.random.default_rng(3)
    X = rng.normal(size=(T, 4, 3))
    rec = oracle.forward(X, alpha=alpha, beta=0.5, v_th=1.0, kappa=np.ones((4, 3)), C=4,
                         psi_kind=PSI_IDENTITY)
    for t in range(T):
        closed = sum(alpha ** (t - s) * X[s] for s in range(t + 1))
        assert np.allclose(rec["Vd"][t + 1], closed, rtol=1e-13, atol=1e-14)


def test_alpha_zero_equals_stateless_bitwise():
    rng = np.random.default_rng(4)
    case = rand_case(rng)
    case["alpha"] = 0.0
    a = run_oracle(case)
    case["stateful"] = False
    b = run_oracle(case)
    for k in ("Vd", "H", "S", "Y"):
        assert np.array_equal(a[k], b[k])


@pytest.mark.parametrize("psi_kind", [PSI_MEXHAT, PSI_IDENTITY])
@pytest.mark.parametrize("sg_kind", [SG_ATAN, SG_SIGMOID])
def test_single_step_closed_form(psi_kind, sg_kind):
    rng = np.random.default_rng(5)
    case = rand_case(rng, T=1, psi_kind=psi_kind, mask=True)
    rec = run_oracle(case)
    g = oracle.backward(rec, case["gS"], case["gV"], sg_kind=sg_kind)
    C, S, B = case["C"], case["S"], case["X"].shape[2]
    N = case["X"].shape[1]
    for n in range(N):
        c = (n // S) % C
        z = 0.0
        gx = np.zeros(B)
        for b in range(B):
            if case["mask"][c, b] == 0:
                continue
            dd = case["X"][0, n, b] - case["xi"][c, b]
            uu = abs(dd) / case["zeta"][c, b]
            if psi_kind == PSI_MEXHAT:
                y, dy = (1 - uu * uu) * math.exp(-uu * uu / 2), uu * (uu * uu - 3) * math.exp(-uu * uu / 2)
            else:
                y, dy = uu, 1.0
            z += case["kappa"][c, b] * y
            gx[b] = case["kappa"][c, b] * dy * np.sign(dd) / case["zeta"][c, b]
        assert math.isclose(rec["H"][0, n], z, rel_tol=1e-14, abs_tol=1e-15)
        assert rec["S"][0, n] == float(z >= case["v_th"])
        if sg_kind == SG_ATAN:
            sg = 1.0 / (1.0 + (math.pi * (z - case["v_th"])) ** 2)
        else:
            sig = 1.0 / (1.0 + math.exp(-4.0 * (z - case["v_th"])))
            sg = 4.0 * sig * (1.0 - sig)
        dH = case["gV"][0, n] + sg * case["gS"][0, n]
        assert np.allclose(g["gX"][0, n], gx * dH, rtol=1e-12, atol=1e-14)


def test_constant_drive_mexican_hat_zero_input():
    """Zero input with psi = MH is not silent: psi(|xi|/zeta) gives a constant drive
    z0 per step.  Below threshold, H[t] = z0 (1 - beta^t)/(1 - beta) until it first
    reaches v_th; the step after a spike restarts from H = z0 (multiplicative reset).
    At or above threshold the neuron fires every step with H = z0."""
    beta, T = 0.5, 12
    # Channel 0: drive 0.6 (< v_th): H = 0.6, 0.9, 1.05 -> spike, then restart.
    # Channel 1: drive 1.0 exactly (tie fires every step).
    kappa = np.array([[0.6], [1.0]])
    X = np.zeros((T, 2, 1))
    rec = oracle.forward(X, alpha=0.5, beta=beta, v_th=1.0, kappa=kappa, C=2,
                         psi_kind=PSI_MEXHAT)
    z0 = 0.6
    h, expect_h, expect_s = 0.0, [], []
    k = 0
    for t in range(T):
        k += 1
        hk = z0 * (1 - beta ** k) / (1 - beta)
        expect_h.append(hk)
        s = hk >= 1.0
        expect_s.append(float(s))
        if s:
            k = 0
    assert np.allclose(rec["H"][:, 0], expect_h, rtol=1e-14)
    assert np.array_equal(rec["S"][:, 0], expect_s)
    assert np.all(rec["H"][:, 1] == 1.0) and np.all(rec["S"][:, 1] == 1.0)


def textbook_lif(x, beta, v_th):
    """Leaky integrate-and-fire with multiplicative hard reset to 0 (point neuron)."""
    v, s = 0.0, 0.0
    out_v, out_s = [], []
    for xt in x:
        v = beta * (1.0 - s) * v + xt
        s = 1.0 if v >= v_th else 0.0
        out_v.append(v)
        out_s.append(s)
    return np.array(out_v), np.array(out_s)


def test_reduces_to_lif():
    """B = 1, psi = identity, kappa = 1, xi = 0, zeta = 1: for X >= 0 and alpha = 0 the
    layer is a LIF neuron bit for bit; for signed X it is LIF(|EMA_alpha(X)|)."""
    rng = np.random.default_rng(6)
    T, N = 16, 7
    X = np.abs(rng.normal(0.0, 0.8, size=(T, N, 1)))
    rec = oracle.forward(X, alpha=0.0, beta=0.9, v_th=1.0, kappa=np.ones((N, 1)), C=N,
                         psi_kind=PSI_IDENTITY)
    for n in range(N):
        v, s = textbook_lif(X[:, n, 0], 0.9, 1.0)
        assert np.array_equal(rec["H"][:, n], v)
        assert np.array_equal(rec["S"][:, n], s)
    Xs = rng.normal(0.0, 0.8, size=(T, N, 1))
    rec = oracle.forward(Xs, alpha=0.7, beta=0.9, v_th=1.0, kappa=np.ones((N, 1)), C=N,
                         psi_kind=PSI_IDENTITY)
    for n in range(N):
        ema = np.zeros(T)
        acc = 0.0
        for t in range(T):
            acc = 0.7 * acc + Xs[t, n, 0]
            ema[t] = acc
        v, s = textbook_lif(np.abs(ema), 0.9, 1.0)
        assert np.allclose(rec["H"][:, n], v, rtol=1e-13, atol=1e-15)
        assert np.array_equal(rec["S"][:, n], s)


def test_zero_input_identity_is_silent():
    X = np.zeros((6, 8, 4))
    rec = oracle.forward(X, alpha=0.5, beta=0.5, v_th=1.0, kappa=np.ones((4, 4)), C=4,
                         psi_kind=PSI_IDENTITY)
    assert np.all(rec["S"] == 0) and np.all(rec["H"] == 0)
    g = oracle.backward(rec, np.ones((6, 8)), np.ones((6, 8)), sg_kind=SG_ATAN)
    assert np.all(g["gX"] == 0)          # sgn(0) = 0 subgradient of the L2 norm


# ---------------------------------------------------------------------------
# Independent scalar stepper (forward)
# ---------------------------------------------------------------------------
def scalar_stepper(case):
    X = case["X"]
    T, N, P = X.shape
    k = case.get("k", 1)
    B = P // k
    C, S = case["C"], case["S"]
    H = np.zeros((T, N))
    Sp = np.zeros((T, N))
    for n in range(N):
        c = (n // S) % C
        vd = [0.0] * P
        h = s = 0.0
        for t in range(T):
            z = 0.0
            for b in range(B):
                ss = 0.0
                for i in range(b * k, (b + 1) * k):   # the compartments on branch b
                    vd[i] = case["alpha"] * vd[i] + X[t, n, i] if case["stateful"] else X[t, n, i]
                    xi = 0.0 if case["xi"] is None else case["xi"][c, i]
                    ss += (vd[i] - xi) ** 2
                ze = 1.0 if case["zeta"] is None else case["zeta"][c, b]
                uu = math.sqrt(ss) / ze
                y = (1.0 - uu * uu) * math.exp(-0.5 * uu * uu) if case["psi_kind"] == PSI_MEXHAT else uu
                on = case["mask"] is None or case["mask"][c, b] != 0
                z += case["kappa"][c, b] * y if on else 0.0
            h = case["beta"] * (1.0 - s) * h + z
            s = 1.0 if h >= case["v_th"] else 0.0
            H[t, n], Sp[t, n] = h, s
    return H, Sp


@pytest.mark.parametrize("psi_kind", [PSI_MEXHAT, PSI_IDENTITY])
@pytest.mark.parametrize("stateful", [True, False])
@pytest.mark.parametrize("mask", [False, True])
@pytest.mark.parametrize("k", [1, 3])
def test_forward_matches_scalar_stepper(psi_kind, stateful, mask, k):
    rng = np.random.default_rng(7)
    case = rand_case(rng, T=6, batch=2, C=3, S=2, B=4, psi_kind=psi_kind, stateful=stateful,
                     mask=mask, k=k)
    rec = run_oracle(case)
    H, Sp = scalar_stepper(case)
    assert np.allclose(rec["H"], H, rtol=1e-12, atol=1e-13)
    assert np.array_equal(rec["S"], Sp)


# ---------------------------------------------------------------------------
# Backward against float64 autograd of the forward equations
# ---------------------------------------------------------------------------
def autograd_grads(case, sg_kind, sg_scale, detach_reset):
    import torch

    torch_dtype = torch.float64
    X = torch.tensor(case["X"], dtype=torch_dtype, requires_grad=True)
    T, N, P = X.shape
    k = case.get("k", 1)
    B = P // k
    C, S = case["C"], case["S"]
    batch = N // (C * S)
    kappa = torch.tensor(case["kappa"], dtype=torch_dtype, requires_grad=True)
    xi = torch.tensor(case["xi"] if case["xi"] is not None else np.zeros((C, P)),
                      dtype=torch_dtype, requires_grad=True)
    zeta = torch.tensor(case["zeta"] if case["zeta"] is not None else np.ones((C, B)),
                        dtype=torch_dtype, requires_grad=True)
    alpha = torch.tensor(case["alpha"], dtype=torch_dtype, requires_grad=True)
    beta = torch.tensor(case["beta"], dtype=torch_dtype, requires_grad=True)
    m = torch.tensor(np.ones((C, B)) if case["mask"] is None else (case["mask"] != 0) * 1.0,
                     dtype=torch_dtype)

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

    def per_neuron(p):
        w = p.shape[1]
        return p[None, :, None, :].expand(batch, C, S, w).reshape(N, w)

    vd = torch.zeros(N, P, dtype=torch_dtype)
    h = torch.zeros(N, dtype=torch_dtype)
    s = torch.zeros(N, dtype=torch_dtype)
    loss = torch.zeros((), dtype=torch_dtype)
    gS = torch.tensor(case["gS"])
    gV = torch.tensor(case["gV"])
    for t in range(T):
        vd = alpha * vd + X[t] if case["stateful"] else X[t]
        dv = vd - per_neuron(xi)
        # branch b holds compartments b k .. b k + k - 1; torch's vector norm
        # (subgradient 0 at the origin) for k > 1
        nrm = torch.abs(dv) if k == 1 else torch.linalg.vector_norm(dv.reshape(N, B, k), dim=2)
        uu = nrm / per_neuron(zeta)
        y = (1 - uu ** 2) * torch.exp(-uu ** 2 / 2) if case["psi_kind"] == PSI_MEXHAT else uu
        z = (per_neuron(kappa * m) * y).sum(dim=1)
        if case.get("residual", False):
            z = z + X[t].mean(dim=1)
        reset = s.detach() if detach_reset else s
        h = beta * (1 - reset) * h + z
        s = Spike.apply(h - case["v_th"])
        loss = loss + (gS[t] * s).sum() + (gV[t] * h).sum()
    loss.backward()
    ga = 0.0 if alpha.grad is None else float(alpha.grad)
    gb = 0.0 if beta.grad is None else float(beta.grad)
    return dict(gX=X.grad.numpy(), g_kappa=kappa.grad.numpy(), g_xi=xi.grad.numpy(),
                g_zeta=zeta.grad.numpy(), g_alpha=ga, g_beta=gb)


@pytest.mark.parametrize("sg_kind", [SG_ATAN, SG_SIGMOID])
@pytest.mark.parametrize("detach_reset", [False, True])
def test_worked_example_backward_vs_autograd(sg_kind, detach_reset):
    w = load_worked_example()
    case = dict(X=w["X"], gS=np.ones((3, 1)), gV=np.zeros((3, 1)), stateful=True, **WORKED)
    rec = oracle.forward(w["X"], **WORKED)
    g = oracle.backward(rec, case["gS"], case["gV"], sg_kind=sg_kind, detach_reset=detach_reset)
    a = autograd_grads(case, sg_kind, 4.0, detach_reset)
    for k in ("gX", "g_kappa", "g_xi", "g_zeta"):
        assert np.allclose(g[k], a[k], rtol=1e-12, atol=1e-15), k
    assert math.isclose(g["g_alpha"], a["g_alpha"], rel_tol=1e-12)


@pytest.mark.parametrize("psi_kind", [PSI_MEXHAT, PSI_IDENTITY])
@pytest.mark.parametrize("sg_kind", [SG_ATAN, SG_SIGMOID])
@pytest.mark.parametrize("detach_reset", [False, True])
@pytest.mark.parametrize("stateful,mask,residual,k", [(True, False, False, 1), (True, True, False, 1),
                                                     (False, True, False, 1), (True, True, True, 1),
                                                     (False, False, True, 1), (True, True, False, 2),
                                                     (False, False, True, 4), (True, False, True, 3)])
def test_backward_matches_autograd(psi_kind, sg_kind, detach_reset, stateful, mask, residual, k):
    rng = np.random.default_rng(8)
    case = rand_case(rng, T=6, batch=2, C=3, S=2, B=3, psi_kind=psi_kind, stateful=stateful,
                     mask=mask, scale=1.2, residual=residual, k=k)
    rec = run_oracle(case)
    g = oracle.backward(rec, case["gS"], case["gV"], sg_kind=sg_kind, sg_scale=3.0,
                        detach_reset=detach_reset)
    a = autograd_grads(case, sg_kind, 3.0, detach_reset)
    for k in ("gX", "g_kappa", "g_xi", "g_zeta"):
        assert np.allclose(g[k], a[k], rtol=1e-11, atol=1e-13), k
    assert math.isclose(g["g_alpha"], a["g_alpha"], rel_tol=1e-11, abs_tol=1e-13)
    assert math.isclose(g["g_beta"], a["g_beta"], rel_tol=1e-11, abs_tol=1e-13)
    if mask:
        off = case["mask"] == 0
        for key in ("g_kappa", "g_zeta"):
            assert np.all(g[key][off] == 0.0)
        assert np.all(g["g_xi"][np.repeat(off, case["k"], axis=1)] == 0.0)


# ---------------------------------------------------------------------------
# Backward against central finite differences of a smooth forward
# ---------------------------------------------------------------------------
def smooth_loss(case, base, sg_kind, sg_scale, detach_reset, X=None, kappa=None, xi=None,
                zeta=None, alpha=None, beta=None):
    """Loss sum(gS S~) + sum(gV H) of a forward whose spike is
    S~[t] = S_base[t] + F(H[t] - v_th) - F(H_base[t] - v_th), F the surrogate's
    primitive.  At the base point S~ equals the recorded spikes, so the
    trajectory is the recorded one, and dS~/dH is the surrogate: the gradient of
    this loss is what BPTT with the surrogate must return."""
    from scipy import special

    X = case["X"] if X is None else X
    kappa = case["kappa"] if kappa is None else kappa
    xi = case["xi"] if xi is None else xi
    zeta = case["zeta"] if zeta is None else zeta
    alpha = case["alpha"] if alpha is None else alpha
    beta = case["beta"] if beta is None else beta
    T, N, P = X.shape
    k = case.get("k", 1)
    B = P // k
    C, S = case["C"], case["S"]
    m = np.ones((C, B)) if case["mask"] is None else (case["mask"] != 0) * 1.0
    if sg_kind == SG_ATAN:
        F = lambda v: np.arctan(np.pi * v) / np.pi + 0.5
    else:
        F = lambda v: special.expit(sg_scale * v)
    cidx = (np.arange(N) // S) % C
    vd = np.zeros((N, P))
    h = np.zeros(N)
    s_t = np.zeros(N)
    s_b = np.zeros(N)
    loss = 0.0
    for t in range(T):
        vd = alpha * vd + X[t] if case["stateful"] else X[t]
        dv = vd - xi[cidx]
        nrm = np.abs(dv) if k == 1 else np.sqrt(np.sum(dv.reshape(N, B, k) ** 2, axis=2))
        uu = nrm / zeta[cidx]
        y = (1 - uu * uu) * np.exp(-0.5 * uu * uu) if case["psi_kind"] == PSI_MEXHAT else uu
        z = ((kappa * m)[cidx] * y).sum(axis=1)
        if case.get("residual", False):
            z = z + X[t].sum(axis=1) / P
        h = beta * (1 - (s_b if detach_reset else s_t)) * h + z
        s_t = base["S"][t] + F(h - case["v_th"]) - F(base["H"][t] - case["v_th"])
        s_b = base["S"][t]
        loss += np.sum(case["gS"][t] * s_t) + np.sum(case["gV"][t] * h)
    return loss


@pytest.mark.parametrize("psi_kind", [PSI_MEXHAT, PSI_IDENTITY])
@pytest.mark.parametrize("sg_kind", [SG_ATAN, SG_SIGMOID])
@pytest.mark.parametrize("detach_reset", [False, True])
@pytest.mark.parametrize("residual,k", [(False, 1), (True, 1), (False, 2), (True, 3)])
def test_backward_matches_finite_differences(psi_kind, sg_kind, detach_reset, residual, k):
    rng = np.random.default_rng(9)
    case = rand_case(rng, T=4, batch=1, C=2, S=2, B=3, psi_kind=psi_kind, mask=True, scale=1.2,
                     residual=residual, k=k)
    rec = run_oracle(case)
    g = oracle.backward(rec, case["gS"], case["gV"], sg_kind=sg_kind, sg_scale=4.0,
                        detach_reset=detach_reset)
    base = dict(S=rec["S"], H=rec["H"])
    L = lambda **kw: smooth_loss(case, base, sg_kind, 4.0, detach_reset, **kw)
    assert math.isclose(L(), np.sum(case["gS"] * rec["S"]) + np.sum(case["gV"] * rec["H"]),
                        rel_tol=1e-13)
    eps = 1e-6

    def fd(name, arr):
        out = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            p, q = arr.copy(), arr.copy()
            p[idx] += eps
            q[idx] -= eps
            out[idx] = (L(**{name: p}) - L(**{name: q})) / (2 * eps)
        return out

    for name, key in (("X", "gX"), ("kappa", "g_kappa"), ("xi", "g_xi"), ("zeta", "g_zeta")):
        num = fd(name, case[name])
        scale = np.max(np.abs(num)) + 1e-30
        assert np.allclose(g[key], num, rtol=1e-6, atol=1e-7 * scale), name
    num_a = (L(alpha=case["alpha"] + eps) - L(alpha=case["alpha"] - eps)) / (2 * eps)
    assert math.isclose(g["g_alpha"], num_a, rel_tol=1e-6, abs_tol=1e-8)
    num_b = (L(beta=case["beta"] + eps) - L(beta=case["beta"] - eps)) / (2 * eps)
    assert math.isclose(g["g_beta"], num_b, rel_tol=1e-6, abs_tol=1e-8)


# ---------------------------------------------------------------------------
# Invariants
# ---------------------------------------------------------------------------
def test_mask_invariants():
    rng = np.random.default_rng(10)
    case = rand_case(rng, mask=True)
    rec = run_oracle(case)
    g = oracle.backward(rec, case["gS"], case["gV"])
    # (kappa, m) equals (kappa (.) m, no mask) in the forward.
    c2 = dict(case, kappa=case["kappa"] * case["mask"], mask=None)
    rec2 = run_oracle(c2)
    assert np.array_equal(rec["H"], rec2["H"]) and np.array_equal(rec["S"], rec2["S"])
    # An all-ones mask equals no mask.
    c3 = dict(case, mask=np.ones_like(case["mask"]))
    c4 = dict(case, mask=None)
    assert np.array_equal(run_oracle(c3)["H"], run_oracle(c4)["H"])
    # A gated-off branch gets exactly zero gradient everywhere.
    off = case["mask"] == 0
    C, S = case["C"], case["S"]
    cidx = (np.arange(case["X"].shape[1]) // S) % C
    assert np.all(g["gX"][:, off[cidx]] == 0.0)
    for k in ("g_kappa", "g_xi", "g_zeta"):
        assert np.all(g[k][off] == 0.0)
    # Changing X (even to NaN/inf) on gated-off branches changes nothing.
    X2 = case["X"].copy()
    X2[:, off[cidx]] = np.where(rng.random(X2[:, off[cidx]].shape) < 0.5, np.nan, 1e300)
    rec5 = run_oracle(dict(case, X=X2))
    assert np.array_equal(rec["H"], rec5["H"]) and np.array_equal(rec["S"], rec5["S"])


def test_causality():
    rng = np.random.default_rng(11)
    case = rand_case(rng, T=8)
    rec = run_oracle(case)
    X2 = case["X"].copy()
    X2[5:] += rng.normal(size=X2[5:].shape)
    rec2 = run_oracle(dict(case, X=X2))
    assert np.array_equal(rec["H"][:5], rec2["H"][:5])
    assert np.array_equal(rec["S"][:5], rec2["S"][:5])
    assert not np.array_equal(rec["H"][5:], rec2["H"][5:])


def test_backward_is_linear_in_output_gradients():
    rng = np.random.default_rng(12)
    case = rand_case(rng, mask=True)
    rec = run_oracle(case)
    gS2, gV2 = rng.normal(size=case["gS"].shape), rng.normal(size=case["gV"].shape)
    a = oracle.backward(rec, case["gS"], case["gV"])
    b = oracle.backward(rec, gS2, gV2)
    ab = oracle.backward(rec, 2.0 * case["gS"] - 3.0 * gS2, 2.0 * case["gV"] - 3.0 * gV2)
    for k in ("gX", "g_kappa", "g_xi", "g_zeta", "g_alpha"):
        assert np.allclose(ab[k], 2.0 * np.asarray(a[k]) - 3.0 * np.asarray(b[k]),
                           rtol=1e-10, atol=1e-12), k


def test_batch_chunking_invariance():
    rng = np.random.default_rng(13)
    case = rand_case(rng, batch=4, mask=True)
    rec = run_oracle(case)
    g = oracle.backward(rec, case["gS"], case["gV"])
    N = case["X"].shape[1]
    half = N // 2
    acc = dict(g_kappa=0.0, g_xi=0.0, g_zeta=0.0, g_alpha=0.0)
    for sl in (slice(0, half), slice(half, N)):
        c = dict(case, X=case["X"][:, sl], gS=case["gS"][:, sl], gV=case["gV"][:, sl])
        r = run_oracle(c)
        assert np.array_equal(r["S"], rec["S"][:, sl])
        gg = oracle.backward(r, c["gS"], c["gV"])
        assert np.allclose(gg["gX"], g["gX"][:, sl], rtol=1e-14, atol=0)
        for k in acc:
            acc[k] = acc[k] + gg[k]
    for k in acc:
        assert np.allclose(acc[k], g[k], rtol=1e-12, atol=1e-14), k


def test_neuron_permutation_within_channel():
    """Neurons of one channel share parameters, so permuting spatial positions
    permutes every output the same way and leaves the parameter gradients alone."""
    rng = np.random.default_rng(14)
    case = rand_case(rng, batch=2, C=2, S=5)
    rec = run_oracle(case)
    g = oracle.backward(rec, case["gS"], case["gV"])
    perm = np.arange(case["X"].shape[1]).reshape(2, 2, 5)[:, :, rng.permutation(5)].reshape(-1)
    c = dict(case, X=case["X"][:, perm], gS=case["gS"][:, perm], gV=case["gV"][:, perm])
    r = run_oracle(c)
    gg = oracle.backward(r, c["gS"], c["gV"])
    assert np.array_equal(r["H"], rec["H"][:, perm])
    assert np.allclose(gg["gX"], g["gX"][:, perm], rtol=1e-15, atol=0)
    for k in ("g_kappa", "g_xi", "g_zeta"):
        assert np.allclose(gg[k], g[k], rtol=1e-12)


def test_forced_spikes_override_decision():
    rng = np.random.default_rng(15)
    case = rand_case(rng, T=5)
    rec = run_oracle(case)
    force = -np.ones(rec["S"].shape, dtype=np.int64)
    force[2, 0] = 1 - int(rec["S"][2, 0])
    r2 = run_oracle(case, force=force)
    assert r2["S"][2, 0] == force[2, 0]
    assert np.array_equal(r2["S"][:2], rec["S"][:2])
    assert np.array_equal(r2["H"][:3], rec["H"][:3])
    others = np.ones(rec["S"].shape[1], dtype=bool)
    others[0] = False
    assert np.array_equal(r2["S"][:, others], rec["S"][:, others])


# ---------------------------------------------------------------------------
# Residual dendrite (Eq. methods-residual)
# ---------------------------------------------------------------------------
def test_residual_with_zero_strengths_is_lif_of_the_mean_input():
    """kappa = 0: the soma sees only (1/P) sum_i X_i, so the layer is a LIF neuron
    driven by the mean input (bit for bit against the textbook LIF on that mean)."""
    rng = np.random.default_rng(20)
    T, N, B = 12, 5, 4
    X = rng.normal(0.4, 1.0, size=(T, N, B))
    rec = oracle.forward(X, alpha=0.6, beta=0.8, v_th=1.0, kappa=np.zeros((N, B)), C=N,
                         psi_kind=PSI_MEXHAT, residual=True)
    for n in range(N):
        v, s = textbook_lif(X[:, n, :].mean(axis=1), 0.8, 1.0)
        assert np.array_equal(rec["H"][:, n], v)
        assert np.array_equal(rec["S"][:, n], s)


@pytest.mark.parametrize("psi_kind", [PSI_MEXHAT, PSI_IDENTITY])
def test_residual_single_step_closed_form(psi_kind):
    rng = np.random.default_rng(21)
    case = rand_case(rng, T=1, psi_kind=psi_kind, mask=True, residual=True)
    case["gV"] = np.zeros_like(case["gV"])
    rec = run_oracle(case)
    base = dict(case, residual=False)
    rec0 = run_oracle(base)
    B = case["X"].shape[2]
    assert np.allclose(rec["H"][0], rec0["H"][0] + case["X"][0].mean(axis=1), rtol=1e-14, atol=1e-15)
    g = oracle.backward(rec, case["gS"], sg_kind=SG_ATAN)
    g0 = oracle.backward(rec0, case["gS"], sg_kind=SG_ATAN)
    sg = 1.0 / (1.0 + (math.pi * (rec["H"][0] - 1.0)) ** 2)
    sg0 = 1.0 / (1.0 + (math.pi * (rec0["H"][0] - 1.0)) ** 2)
    dH = sg * case["gS"][0]
    # the dendritic part scales with dH; the residual part adds dH / P to every compartment
    expect = g0["gX"][0] * (dH / np.where(sg0 * case["gS"][0] == 0, 1, sg0 * case["gS"][0]))[:, None] + dH[:, None] / B
    assert np.allclose(g["gX"][0], expect, rtol=1e-11, atol=1e-13)


def test_plif_beta_gradient_of_a_free_leak():
    """No input after the first step, no spikes: H[t] = beta^(t-1) z for t >= 1, so with
    gV = 1 at the last step only and the reset path detached (no surrogate term),
    dL/dbeta = (T-1) beta^(T-2) z (textbook derivative)."""
    T, beta, z = 6, 0.7, 0.6
    X = np.zeros((T, 1, 1))
    X[0, 0, 0] = z
    rec = oracle.forward(X, alpha=0.0, beta=beta, v_th=10.0, kappa=np.ones((1, 1)), C=1,
                         psi_kind=PSI_IDENTITY, stateful=False)
    gV = np.zeros((T, 1))
    gV[-1, 0] = 1.0
    g = oracle.backward(rec, np.zeros((T, 1)), gV, sg_kind=SG_ATAN, detach_reset=True)
    assert math.isclose(rec["H"][-1, 0], beta ** (T - 1) * z, rel_tol=1e-14)
    assert math.isclose(g["g_beta"], (T - 1) * beta ** (T - 2) * z, rel_tol=1e-13)


# ---------------------------------------------------------------------------
# Several compartments per branch (Eq. methods-branch-aggregation, k = P/B > 1)
# ---------------------------------------------------------------------------
TWO_COMP = dict(alpha=0.5, beta=0.5, v_th=1.0, kappa=np.array([[0.5, 0.25]]),
                xi=np.array([[0.0, 0.0, 2.0, 0.0]]), zeta=np.array([[10.0, 4.0]]), mask=None, C=1, S=1,
                psi_kind=PSI_IDENTITY, comps_per_branch=2)
TWO_COMP_X = np.array([[3.0, 4.0, 0.0, 0.0], [4.5, 6.0, 5.0, 4.0]])[:, None, :]


def test_two_compartment_worked_example_by_hand():
    """B = 2 branches of k = 2 compartments (compartments 0, 1 on branch 0 and 2, 3 on
    branch 1), Identity, worked out by hand; every value is a dyadic rational.
      t = 1: Vd = (3, 4, 0, 0), d = Vd - xi = (3, 4, -2, 0), norms (5, 2), u = (1/2, 1/2),
             Z = 0.5/2 + 0.25/2 = 0.375 = H1, no spike.
      t = 2: Vd = (6, 8, 5, 4), d = (6, 8, 3, 4), norms (10, 5), u = (1, 5/4),
             Z = 0.5 + 0.3125, H2 = 0.375/2 + 0.8125 = 1: a tie, which fires.
    Backward with gS = 1, gV = 0, atan surrogate, full reset gradient:
      dH2 = sg(0) = 1;  dS1 = 1 - beta H1 dH2 = 0.8125;  dH1 = q dS1 + beta dH2,
      q = sg(H1 - 1) = 1 / (1 + pi^2 (5/8)^2);
      r_i = kappa_b dH d_i / (zeta_b ||d_b||),  lam = r + alpha lam[t+1]."""
    rec = oracle.forward(TWO_COMP_X, **TWO_COMP)
    assert np.array_equal(rec["H"][:, 0], [0.375, 1.0])
    assert np.array_equal(rec["S"][:, 0], [0.0, 1.0])
    assert np.array_equal(rec["u"][:, 0, :], [[0.5, 0.5], [1.0, 1.25]])
    g = oracle.backward(rec, np.ones((2, 1)), sg_kind=SG_ATAN)
    q = 1.0 / (1.0 + math.pi ** 2 * 0.390625)
    dH2 = 1.0
    dH1 = q * 0.8125 + 0.5 * dH2
    assert np.allclose(g["dH"][:, 0], [dH1, dH2], rtol=1e-14, atol=0)
    r2 = np.array([0.5 * 6 / 100, 0.5 * 8 / 100, 0.25 * 3 / 20, 0.25 * 4 / 20])
    r1 = dH1 * np.array([0.5 * 3 / 50, 0.5 * 4 / 50, 0.25 * -2 / 8, 0.0])
    lam2 = r2
    lam1 = r1 + 0.5 * lam2
    assert np.allclose(g["gX"][:, 0, :], [lam1, lam2], rtol=1e-14, atol=1e-300)
    assert np.allclose(g["g_xi"][0], -(r1 + r2), rtol=1e-14)
    assert np.allclose(g["g_kappa"][0], [dH1 * 0.5 + 1.0, dH1 * 0.5 + 1.25], rtol=1e-14)
    assert np.allclose(g["g_zeta"][0], [-(0.5 * dH1 * 0.5 / 10 + 0.5 * 1.0 / 10),
                                        -(0.25 * dH1 * 0.5 / 4 + 0.25 * 1.25 / 4)], rtol=1e-14)
    assert math.isclose(g["g_alpha"], lam2 @ np.array([3.0, 4.0, 0.0, 0.0]), rel_tol=1e-14)
    assert math.isclose(g["g_beta"], dH2 * 0.375, rel_tol=1e-14)


def test_replicated_compartments_equal_one_with_scaled_dilation():
    """k identical compartments (same input, same xi) have norm sqrt(k) |d|, so the layer
    equals the one-compartment layer with zeta / sqrt(k); the input gradient splits evenly
    over the k copies, xi's likewise, and zeta's scales by 1/sqrt(k)."""
    rng = np.random.default_rng(30)
    k = 4
    base = rand_case(rng, T=6, B=3, mask=True, psi_kind=PSI_MEXHAT, k=1)
    rep_case = dict(base, X=np.repeat(base["X"], k, axis=2), xi=np.repeat(base["xi"], k, axis=1), k=k)
    one = dict(base, zeta=base["zeta"] / math.sqrt(k))
    a, b = run_oracle(rep_case), run_oracle(one)
    assert np.allclose(a["H"], b["H"], rtol=1e-12, atol=1e-13)
    assert np.array_equal(a["S"], b["S"])
    ga = oracle.backward(a, base["gS"], base["gV"], sg_kind=SG_SIGMOID)
    gb = oracle.backward(b, base["gS"], base["gV"], sg_kind=SG_SIGMOID)
    T, N = base["gS"].shape
    assert np.allclose(ga["gX"].reshape(T, N, 3, k), gb["gX"][..., None] / k, rtol=1e-10, atol=1e-13)
    assert np.allclose(ga["g_xi"].reshape(base["C"], 3, k), gb["g_xi"][..., None] / k, rtol=1e-10, atol=1e-13)
    assert np.allclose(ga["g_zeta"], gb["g_zeta"] / math.sqrt(k), rtol=1e-10, atol=1e-13)
    assert np.allclose(ga["g_kappa"], gb["g_kappa"], rtol=1e-10, atol=1e-13)
    assert math.isclose(ga["g_alpha"], gb["g_alpha"], rel_tol=1e-10)


def test_compartment_order_within_a_branch_does_not_matter():
    """The norm is symmetric in a branch's compartments: permuting them (with their xi)
    permutes gX and g_xi and leaves everything else alone; moving a compartment to
    another branch changes the result."""
    rng = np.random.default_rng(31)
    k, B = 3, 2
    case = rand_case(rng, T=5, B=B, k=k, mask=False)
    perm = np.concatenate([b * k + rng.permutation(k) for b in range(B)])
    c2 = dict(case, X=case["X"][:, :, perm], xi=case["xi"][:, perm])
    a, b = run_oracle(case), run_oracle(c2)
    assert np.allclose(a["H"], b["H"], rtol=1e-13) and np.array_equal(a["S"], b["S"])
    ga, gb = oracle.backward(a, case["gS"], case["gV"]), oracle.backward(b, case["gS"], case["gV"])
    assert np.allclose(gb["gX"], ga["gX"][:, :, perm], rtol=1e-12, atol=1e-14)
    assert np.allclose(gb["g_xi"], ga["g_xi"][:, perm], rtol=1e-12, atol=1e-14)
    swap = np.arange(B * k)
    swap[[0, k]] = swap[[k, 0]]   # compartment 0 to branch 1 and back
    c3 = dict(case, X=case["X"][:, :, swap], xi=case["xi"][:, swap])
    assert not np.allclose(run_oracle(c3)["H"], a["H"], rtol=1e-6)


@pytest.mark.parametrize("T,batch,C,S", [(0, 2, 3, 4), (5, 0, 3, 4), (5, 2, 0, 4), (5, 2, 3, 0), (0, 0, 0, 0)])
def test_empty_layer_has_empty_outputs_and_zero_gradients(T, batch, C, S):
    """A layer with no neuron-step: every output has no elements and every
    parameter gradient is a sum with no terms, +0; the same layer with one more
    step or sample is not empty (the shapes follow the layer, not a special case)."""
    B, k = 3, 2
    N, P = batch * C * S, B * k
    rng = np.random.default_rng(2)
    kw = dict(alpha=0.5, beta=0.5, v_th=1.0, kappa=rng.random((C, B)), xi=rng.random((C, P)),
              zeta=rng.random((C, B)) + 0.5, mask=(rng.random((C, B)) < 0.5).astype(np.uint8), C=C, S=S,
              comps_per_branch=k, residual=True)
    rec = oracle.forward(np.zeros((T, N, P)), **kw)
    assert rec["S"].shape == (T, N) and rec["H"].shape == (T, N)
    g = oracle.backward(rec, np.zeros((T, N)))
    assert g["gX"].shape == (T, N, P)
    for name, shape in (("g_kappa", (C, B)), ("g_xi", (C, P)), ("g_zeta", (C, B))):
        assert g[name].shape == shape
        assert not g[name].any() and not np.signbit(g[name]).any()
    assert g["g_alpha"] == 0.0 and g["g_beta"] == 0.0
    assert not math.copysign(1.0, g["g_alpha"]) < 0 and not math.copysign(1.0, g["g_beta"]) < 0
    if C * S > 0 and batch > 0:
        rec1 = oracle.forward(np.ones((T + 1, N, P)), **kw)
        g1 = oracle.backward(rec1, np.ones((T + 1, N)))
        assert np.abs(g1["g_kappa"]).sum() > 0
    with pytest.raises(ValueError):
        oracle.forward(np.zeros((T, 1, P)), **dict(kw, C=0)) if C == 0 else oracle.forward(np.zeros((T, N + 1, P)), **kw)
