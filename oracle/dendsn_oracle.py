"""Float64 CPU oracle of the DendSN layer: forward scan and surrogate-gradient BPTT.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call this
module; only the test-suite, the smoke check and the CPU-baseline leg of the
benchmark do.  It shares no code, constants or helpers with the HIP library.

Every array is float64.  Shapes follow the layer form of the paper (Methods,
"Dendritic spiking neural networks"): the synaptic input of one layer is
``X[t, n, i]`` with T time steps, N = batch * C * S neurons ordered
``(batch, channel, spatial)`` and P = B k compartments, k per branch (constraint
(1): every branch holds P/B compartments).  Compartment i lies on branch
b = i // k, i.e. the wiring matrix Gamma groups consecutive compartments
(Gamma[b, i] = 1 iff b k <= i < (b + 1) k); with k = 1 compartment b is branch b.
Neurons of one channel share the parameters (constraint (3)): the translation
xi per compartment ``[C, P]``, the dilation zeta, the strength kappa and the
branch-gating mask per branch ``[C, B]``; alpha is shared by the whole layer.

Forward recurrences, in the paper's order (Methods, "Dendritic spiking neuron"):

  Eq. (methods-compartment)         Vd_i[t] = alpha * Vd_i[t-1] + X_i[t],  Vd[0] = 0
                                    (Stateless Dendrite variant: Vd_i[t] = X_i[t])
  Eq. (methods-branch-aggregation)  d_i[t]  = Vd_i[t] - xi_i
                                    u_b[t]  = sqrt(sum_{i in C_b} d_i[t]^2) / zeta_b
                                    Y_b[t]  = psi(u_b[t])
  Eq. (methods-mexican-hat)         psi(x)  = (1 - x^2) exp(-x^2 / 2)   ("MH"), or psi(x) = x ("Identity")
  Eq. (methods-soma-input)          Z[t]    = sum_b kappa*_b Y_b[t]
  Eq. (methods-residual)            Z[t]   += (1/P) sum_i X_i[t]   (ResStateful / ResStateless variants)
  Eq. (methods-dbg-mask)            kappa*  = kappa (.) m   (dendritic branch gating; m = 1 without a mask)
  Eq. (methods-lif-reset-charge)    H[t]    = beta (1 - S[t-1]) H[t-1] + Z[t],  H[0] = 0, S[0] = 0
  Eq. (methods-lif-fire)            S[t]    = Theta(H[t] - v_th),  Theta(x) = 1 iff x >= 0

H is the somatic potential V^s of the paper (the charged value before the reset
that is applied at the next step).

Backward: the paper trains the layer with BPTT, replacing Theta' by the
derivative of a smooth surrogate (Methods, Eq. (methods-sg), the arctangent
surrogate); a sigmoid surrogate sigma(a x) is offered as well (the paper's spike
probability of Eq. (methods-l5pc-spike-prob) uses a = 4).  The adjoints below
are the chain rule applied to the forward recurrences above, in reverse time:

  dS[t]   = gS[t] - beta H[t] dH[t+1]                 (second term dropped when the reset is detached)
  dH[t]   = gV[t] + sg(H[t] - v_th) dS[t] + beta (1 - S[t]) dH[t+1]
  g_beta += dH[t] (1 - S[t-1]) H[t-1]                 (PLIF soma: beta learnable)
  g_u_b   = kappa*_b dH[t] psi'(u_b[t])
  r_i[t]  = g_u_b d_i[t] / (zeta_b ||d_{C_b}[t]||)    (d/dVd_i of u_b; the L2 norm's subgradient
                                                       at 0 is taken as 0, which for k = 1 is
                                                       r = g_u sgn(d) / zeta with sgn(0) = 0)
  lam_i[t]= r_i[t] + alpha lam_i[t+1]                 (Stateless: lam = r)
  gX      = lam (+ dH / P with the residual term);
  g_kappa_b += m dH Y_b;  g_xi_i += -r_i;  g_zeta_b += -g_u_b u_b / zeta_b;
  g_alpha   += sum_i lam_i[t] Vd_i[t-1]

The backward consumes the recorded spikes S rather than re-deciding Theta, so
that the oracle's gradient is exactly the gradient of the forward whose spikes
it reports.

Parity pins for every function here live in tests/test_oracle_pins.py.
"""

from __future__ import annotations

import numpy as np

PSI_IDENTITY = "identity"
PSI_MEXHAT = "mexhat"
SG_ATAN = "atan"
SG_SIGMOID = "sigmoid"


# --------------------------------------------------------------------------
# Dendritic activation, Eq. (methods-mexican-hat) and the Identity variant
# (Methods, "DendSN variants", activation-free branch).
# --------------------------------------------------------------------------
def psi(u: np.ndarray, kind: str) -> np.ndarray:
    """psi(u): Mexican hat (1 - u^2) exp(-u^2/2) or the identity."""
    if kind == PSI_MEXHAT:
        return (1.0 - u * u) * np.exp(-0.5 * u * u)
    if kind == PSI_IDENTITY:
        return u.copy()
    raise ValueError(f"unknown psi {kind!r}")


def dpsi(u: np.ndarray, kind: str) -> np.ndarray:
    """psi'(u).  Mexican hat: d/du[(1-u^2) e^{-u^2/2}] = u (u^2 - 3) e^{-u^2/2}."""
    if kind == PSI_MEXHAT:
        return u * (u * u - 3.0) * np.exp(-0.5 * u * u)
    if kind == PSI_IDENTITY:
        return np.ones_like(u)
    raise ValueError(f"unknown psi {kind!r}")


# --------------------------------------------------------------------------
# Surrogate derivative of Theta, Eq. (methods-sg) and the sigmoid form.
# --------------------------------------------------------------------------
def _sigmoid(z: np.ndarray) -> np.ndarray:
    """Logistic function in the form that never overflows exp."""
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def surrogate_grad(x: np.ndarray, kind: str, scale: float = 4.0) -> np.ndarray:
    """Theta'(x) replaced by the surrogate's derivative.

    atan:    d/dx [arctan(pi x)/pi + 1/2] = 1 / (1 + pi^2 x^2)   (Eq. methods-sg)
    sigmoid: d/dx sigma(a x) = a sigma(a x) (1 - sigma(a x)),  a = scale
    """
    x = np.asarray(x, dtype=np.float64)
    if kind == SG_ATAN:
        return 1.0 / (1.0 + (np.pi * x) ** 2)
    if kind == SG_SIGMOID:
        s = _sigmoid(scale * x)
        return scale * s * (1.0 - s)
    raise ValueError(f"unknown surrogate {kind!r}")


# --------------------------------------------------------------------------
# Parameter layout helpers (Methods, "Dendritic spiking neural networks",
# constraint (3): per-channel parameters shared over spatial positions).
# --------------------------------------------------------------------------
def _per_neuron(p: np.ndarray, batch: int, C: int, S: int) -> np.ndarray:
    """Expand a [C, W] per-channel table to [N, W] with N ordered (batch, C, S)."""
    W = p.shape[1]
    return np.broadcast_to(p[None, :, None, :], (batch, C, S, W)).reshape(batch * C * S, W)


def _channel_sum(a: np.ndarray, batch: int, C: int, S: int) -> np.ndarray:
    """Sum a [T, N, W] array over time, batch and spatial positions -> [C, W]."""
    T, N, W = a.shape
    return a.reshape(T, batch, C, S, W).sum(axis=(0, 1, 3))


def _check_shapes(X, kappa, C, S, k):
    if X.ndim != 3:
        raise ValueError("X must be [T, N, P]")
    T, N, P = X.shape
    if C * S == 0:
        # A layer without neurons: every per-neuron array is empty and every
        # sum over neurons has no terms, whatever the batch size.
        if N != 0:
            raise ValueError("N must be batch * C * S")
        if k < 1 or P % k != 0:
            raise ValueError("P must be a multiple of the compartments per branch k")
        if kappa.shape != (C, P // k):
            raise ValueError("kappa must be [C, B]")
        return T, N, P, P // k, 0
    if N % (C * S) != 0:
        raise ValueError("N must be batch * C * S")
    if k < 1 or P % k != 0:
        raise ValueError("P must be a multiple of the compartments per branch k")
    B = P // k
    if kappa.shape != (C, B):
        raise ValueError("kappa must be [C, B]")
    return T, N, P, B, N // (C * S)


# --------------------------------------------------------------------------
# Forward scan.
# --------------------------------------------------------------------------
def forward(
    X: np.ndarray,
    *,
    alpha: float,
    beta: float,
    v_th: float,
    kappa: np.ndarray,
    xi: np.ndarray | None = None,
    zeta: np.ndarray | None = None,
    mask: np.ndarray | None = None,
    C: int,
    S: int = 1,
    psi_kind: str = PSI_MEXHAT,
    stateful: bool = True,
    residual: bool = False,
    comps_per_branch: int = 1,
    force: np.ndarray | None = None,
) -> dict:
    """Run the DendSN layer forward over all T steps.

    X: [T, N, P] with P = B k, k = comps_per_branch; kappa, zeta: [C, B];
    xi: [C, P] (xi None -> 0, zeta None -> 1); mask: [C, B] of {0, 1} or None
    (all ones).
    force: optional [T, N] int array; entries 0 or 1 override the spike decision
    at that step (used to impose a decision taken elsewhere), -1 leaves it free.

    Returns a record with Vd [T+1, N, P] (Vd[0] = 0), d [T, N, P], the branch
    norms, u and Y [T, N, B], Z, H, S [T, N] and the inputs ``backward`` needs.
    """
    X = np.asarray(X, dtype=np.float64)
    kappa = np.asarray(kappa, dtype=np.float64)
    k = int(comps_per_branch)
    T, N, P, B, batch = _check_shapes(X, kappa, C, S, k)
    xi = np.zeros((C, P)) if xi is None else np.asarray(xi, dtype=np.float64)
    if xi.shape != (C, P):
        raise ValueError("xi must be [C, P]: one translation per compartment")
    zeta = np.ones((C, B)) if zeta is None else np.asarray(zeta, dtype=np.float64)
    m = np.ones((C, B)) if mask is None else (np.asarray(mask) != 0).astype(np.float64)
    if np.any(zeta <= 0):
        raise ValueError("zeta must be positive (dilation factor)")
    if stateful and not (0.0 <= alpha < 1.0):
        raise ValueError("alpha must lie in [0, 1)")
    if not (0.0 <= beta < 1.0):
        raise ValueError("beta must lie in [0, 1)")

    xi_n = _per_neuron(xi, batch, C, S)
    zeta_n = _per_neuron(zeta, batch, C, S)
    kstar_n = _per_neuron(kappa * m, batch, C, S)
    m_n = _per_neuron(m, batch, C, S)

    Vd = np.zeros((T + 1, N, P))
    d = np.zeros((T, N, P))
    nrm = np.zeros((T, N, B))
    u = np.zeros((T, N, B))
    Y = np.zeros((T, N, B))
    Z = np.zeros((T, N))
    H = np.zeros((T, N))
    Sp = np.zeros((T, N))
    h_prev = np.zeros(N)
    s_prev = np.zeros(N)
    for t in range(T):
        # Eq. (methods-compartment), or the Stateless Dendrite variant.
        Vd[t + 1] = alpha * Vd[t] + X[t] if stateful else X[t]
        # Eq. (methods-branch-aggregation): the L2 norm over the branch's k
        # compartments (consecutive compartments share a branch), dilated by zeta_b.
        d[t] = Vd[t + 1] - xi_n
        nrm[t] = np.sqrt((d[t] * d[t]).reshape(N, B, k).sum(axis=2))
        u[t] = nrm[t] / zeta_n
        Y[t] = psi(u[t], psi_kind)
        # Eq. (methods-soma-input) with the gated strengths of Eq. (methods-dbg-mask).
        # A gated-off branch contributes nothing, whatever its Y.
        Z[t] = np.where(m_n != 0, kstar_n * Y[t], 0.0).sum(axis=1)
        if residual:
            # Eq. (methods-residual): the mean synaptic input of the P compartments
            # (gating scales branch strengths only, so every compartment takes part).
            Z[t] = Z[t] + X[t].sum(axis=1) / P
        # Eq. (methods-lif-reset-charge) and Eq. (methods-lif-fire).
        H[t] = beta * (1.0 - s_prev) * h_prev + Z[t]
        s = (H[t] - v_th >= 0.0).astype(np.float64)
        if force is not None:
            f = force[t]
            s = np.where(f >= 0, f.astype(np.float64), s)
        Sp[t] = s
        h_prev, s_prev = H[t], s

    return dict(
        X=X, Vd=Vd, d=d, nrm=nrm, u=u, Y=Y, Z=Z, H=H, S=Sp, k=k,
        alpha=float(alpha), beta=float(beta), v_th=float(v_th),
        kappa=kappa, xi=xi, zeta=zeta, m=m, C=C, S_sp=S, batch=batch,
        psi_kind=psi_kind, stateful=bool(stateful), residual=bool(residual),
    )


# --------------------------------------------------------------------------
# Backward scan (BPTT with a surrogate for Theta').
# --------------------------------------------------------------------------
def backward(
    rec: dict,
    gS: np.ndarray,
    gV: np.ndarray | None = None,
    *,
    sg_kind: str = SG_SIGMOID,
    sg_scale: float = 4.0,
    detach_reset: bool = False,
) -> dict:
    """Gradients of sum(gS * S) + sum(gV * H) w.r.t. X, kappa, xi, zeta, alpha.

    Also returns, for each parameter gradient, the sum of the absolute values of
    the terms that make it up (``abs_*``): the scale against which a summed
    gradient's rounding error is judged.
    """
    T, N, B = rec["Y"].shape
    k = rec["k"]
    P = B * k
    C, S, batch = rec["C"], rec["S_sp"], rec["batch"]
    alpha, beta, v_th = rec["alpha"], rec["beta"], rec["v_th"]
    stateful = rec["stateful"]
    gS = np.asarray(gS, dtype=np.float64)
    gV = np.zeros((T, N)) if gV is None else np.asarray(gV, dtype=np.float64)

    m_n = _per_neuron(rec["m"], batch, C, S)
    kstar_n = _per_neuron(rec["kappa"] * rec["m"], batch, C, S)
    zeta_n = _per_neuron(rec["zeta"], batch, C, S)
    H, Sp, u, d, Y, Vd = rec["H"], rec["S"], rec["u"], rec["d"], rec["Y"], rec["Vd"]
    nrm = rec["nrm"]

    dH = np.zeros((T, N))
    gX = np.zeros((T, N, P))
    t_beta = np.zeros((T, N))
    t_kappa = np.zeros((T, N, B))
    t_xi = np.zeros((T, N, P))
    t_zeta = np.zeros((T, N, B))
    t_alpha = np.zeros((T, N, P))
    dH_next = np.zeros(N)
    lam_next = np.zeros((N, P))
    sg_all = surrogate_grad(H - v_th, sg_kind, sg_scale)
    for t in range(T - 1, -1, -1):
        # Somatic adjoint: S[t] feeds H[t+1] through the reset factor (1 - S[t]),
        # H[t] feeds H[t+1] through beta (1 - S[t]) and S[t] through Theta.
        dS = gS[t] if detach_reset else gS[t] - beta * H[t] * dH_next
        dH[t] = gV[t] + sg_all[t] * dS + beta * (1.0 - Sp[t]) * dH_next
        # Z[t] enters H[t] with unit weight, so dZ[t] = dH[t].
        g_u = kstar_n * dH[t][:, None] * dpsi(u[t], rec["psi_kind"])
        # du_b/dVd_i = (d_i / ||d_b||) / zeta_b for i on branch b (for k = 1 the unit
        # direction d / |d| is sgn(d) exactly); 0 where the norm vanishes and on
        # gated-off branches (nothing of theirs reaches the soma).
        live = np.repeat((m_n != 0) & (nrm[t] > 0.0), k, axis=1)                    # [N, P]
        unit = np.where(live, d[t] / np.where(live, np.repeat(nrm[t], k, axis=1), 1.0), 0.0)
        r = np.where(live, np.repeat(g_u, k, axis=1) * unit / np.repeat(zeta_n, k, axis=1), 0.0)
        lam = r + alpha * lam_next if stateful else r
        gX[t] = lam + dH[t][:, None] / P if rec["residual"] else lam
        # H[t] = beta (1 - S[t-1]) H[t-1] + Z[t]: the PLIF soma's beta gradient
        if t > 0:
            t_beta[t] = dH[t] * (1.0 - Sp[t - 1]) * H[t - 1]
        t_kappa[t] = np.where(m_n != 0, dH[t][:, None] * Y[t], 0.0)
        t_xi[t] = -r
        t_zeta[t] = np.where(m_n != 0, -g_u * u[t] / zeta_n, 0.0)
        if stateful:
            t_alpha[t] = lam * Vd[t]          # Vd[t] is V^d at the previous step
        dH_next, lam_next = dH[t], lam

    return dict(
        gX=gX,
        dH=dH,
        g_kappa=_channel_sum(t_kappa, batch, C, S),
        g_xi=_channel_sum(t_xi, batch, C, S),
        g_zeta=_channel_sum(t_zeta, batch, C, S),
        g_alpha=float(t_alpha.sum()),
        g_beta=float(t_beta.sum()),
        abs_beta=float(np.abs(t_beta).sum()),
        abs_kappa=_channel_sum(np.abs(t_kappa), batch, C, S),
        abs_xi=_channel_sum(np.abs(t_xi), batch, C, S),
        abs_zeta=_channel_sum(np.abs(t_zeta), batch, C, S),
        abs_alpha=float(np.abs(t_alpha).sum()),
    )
