"""A plain float32 evaluation of the DendSN layer equations: accuracy evidence.

TEST INFRASTRUCTURE ONLY.  This is neither the oracle (float64, tests only) nor
the HIP library: it evaluates the same recurrences (Methods, "Dendritic spiking
neuron": Eqs. methods-compartment, methods-branch-aggregation,
methods-mexican-hat, methods-soma-input, methods-residual,
methods-lif-reset-charge, methods-lif-fire; the surrogate of Eq. methods-sg) and
their adjoints in numpy float32, every intermediate rounded to float32, on a
given spike train.  Its distance from the float64 oracle on an input is what any
float32 evaluation of the method must be allowed there: the parity tolerances
for float32 outputs are derived from it (tests/parity.py), so no bound is looser
than what float32 arithmetic itself needs on that input.

The spike train is imposed (the oracle's, which the parity protocol has already
aligned with the kernel's), so the comparison measures the rounding of the
continuous quantities, not a different branch of the threshold decision.
"""

from __future__ import annotations

import numpy as np

F = np.float32


def _expand(p, batch, C, S):
    """[C, W] per-channel table -> [N, W], N ordered (batch, C, S)."""
    W = p.shape[1]
    return np.ascontiguousarray(np.broadcast_to(p[None, :, None, :], (batch, C, S, W)).reshape(batch * C * S, W))


def _chan(a, batch, C, S):
    """[N, W] -> [C, W]: sum over batch items and positions, in float32."""
    N, W = a.shape
    return a.reshape(batch, C, S, W).sum(axis=(0, 2), dtype=F)


def evaluate(X, spikes, gS, gV=None, *, alpha, beta, v_th, kappa, xi=None, zeta=None, mask=None, C, S=1,
             psi="mexhat", stateful=True, residual=False, k=1, sg="sigmoid", sg_scale=4.0, detach=False):
    """Forward (H) and backward (grad_x, parameter gradients) in float32 on the
    imposed spike train ``spikes`` [T, N].  X: [T, N, P]; gS, gV: [T, N]."""
    X = np.asarray(X, F)
    T, N, P = X.shape
    B = P // k
    batch = N // (C * S)
    sp = np.asarray(spikes, F)
    gS = np.asarray(gS, F)
    gV = np.zeros((T, N), F) if gV is None else np.asarray(gV, F)
    a, b, vth = F(alpha if stateful else 0.0), F(beta), F(v_th)
    kap = np.asarray(kappa, F)
    m = np.ones((C, B), F) if mask is None else (np.asarray(mask) != 0).astype(F)
    ks = _expand(kap * m, batch, C, S)                                        # [N, B]
    on = _expand(m, batch, C, S) != 0
    xin = _expand(np.zeros((C, P), F) if xi is None else np.asarray(xi, F), batch, C, S)
    rz = _expand(F(1) / (np.ones((C, B), F) if zeta is None else np.asarray(zeta, F)), batch, C, S)
    rp = F(1.0 / P)

    # forward: dendrite, aggregation, activation, branch sum, soma
    vd = np.zeros((N, P), F)
    Vd = np.zeros((T + 1, N, P), F)
    d = np.zeros((T, N, P), F)
    nrm = np.zeros((T, N, B), F)
    e = np.zeros((T, N, B), F)
    y = np.zeros((T, N, B), F)
    H = np.zeros((T, N), F)
    h = np.zeros(N, F)
    s_prev = np.zeros(N, F)
    for t in range(T):
        vd = a * vd + X[t] if stateful else X[t].copy()
        vd[np.repeat(~on, k, axis=1)] = 0                     # a gated-off branch integrates nothing
        Vd[t + 1] = vd
        d[t] = vd - xin
        nrm[t] = np.sqrt((d[t] * d[t]).reshape(N, B, k).sum(axis=2, dtype=F))
        u = nrm[t] * rz
        if psi == "mexhat":
            e[t] = np.exp(F(-0.5) * u * u)
            y[t] = (F(1) - u * u) * e[t]
        else:
            y[t] = u
        z = (ks * y[t]).sum(axis=1, dtype=F)
        if residual:
            z = z + X[t].sum(axis=1, dtype=F) * rp
        h = b * (F(1) - s_prev) * h + z
        H[t] = h
        s_prev = sp[t]

    # backward, last step first
    gX = np.zeros((T, N, P), F)
    acc_k = np.zeros((N, B), F)
    acc_xi = np.zeros((N, P), F)
    acc_z = np.zeros((N, B), F)
    acc_a = np.zeros((N, P), F)
    acc_b = np.zeros(N, F)
    dh_next = np.zeros(N, F)
    lam = np.zeros((N, P), F)
    for t in range(T - 1, -1, -1):
        x = H[t] - vth
        if sg == "atan":
            px = F(np.pi) * x
            sgv = F(1) / (F(1) + px * px)
        else:  # a sigma(a x) (1 - sigma(a x)) = a e / (1 + e)^2 with e = exp(-|a x|)
            ex = np.exp(-np.abs(F(sg_scale) * x))
            sgv = F(sg_scale) * ex / ((F(1) + ex) * (F(1) + ex))
        dS = gS[t] if detach else gS[t] - b * H[t] * dh_next
        dh = gV[t] + sgv * dS + b * (F(1) - sp[t]) * dh_next
        u = nrm[t] * rz
        dpsi = u * (u * u - F(3)) * e[t] if psi == "mexhat" else np.ones_like(u)
        g_u = ks * dh[:, None] * dpsi                                          # [N, B]
        live = on & (nrm[t] > 0)
        w = np.where(live, g_u * rz / np.where(live, nrm[t], F(1)), F(0))      # factor of d_i
        r = np.repeat(w, k, axis=1) * d[t]
        lam = r + a * lam if stateful else r
        gX[t] = lam + dh[:, None] * rp if residual else lam
        acc_k += np.where(on, dh[:, None] * y[t], F(0))
        acc_xi -= r
        acc_z += np.where(on, -g_u * u * rz, F(0))
        if stateful:
            acc_a += lam * Vd[t]
        if t > 0:
            acc_b += dh * (F(1) - sp[t - 1]) * H[t - 1]
        dh_next = dh
    return dict(H=H, gX=gX, g_kappa=_chan(acc_k, batch, C, S), g_xi=_chan(acc_xi, batch, C, S),
                g_zeta=_chan(acc_z, batch, C, S), g_alpha=float(acc_a.sum(dtype=F)) if stateful else 0.0,
                g_beta=float(acc_b.sum(dtype=F)))


def elementwise_ratio(got, ref):
    """max |got - ref| / (|ref| + rms(ref)): the elementwise error measure of the
    parity tests."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    scale = np.abs(ref) + np.sqrt(np.mean(ref * ref))
    return float(np.max(np.abs(got - ref) / np.maximum(scale, 1e-300)))


def summed_ratio(got, ref, absum):
    """max |got - ref| / (A + rms(A)) for summed gradients with term scale A."""
    got, ref, absum = (np.asarray(v, np.float64) for v in (got, ref, absum))
    floor = np.sqrt(np.mean(absum * absum)) if absum.ndim else 0.0
    return float(np.max(np.abs(got - ref) / np.maximum(absum + floor, 1e-30)))
