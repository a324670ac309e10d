"""The oracle's pins have teeth: each plausible mistake planted in a copy of the
oracle (on the CPU, never in the real module) makes at least one pin fail."""

import types

import pytest

import oracle.dendsn_oracle as real
import tests.test_oracle_pins as pins

MUTANTS = {
    "reset gradient term dropped": ("gS[t] - beta * H[t] * dH_next", "gS[t] + 0.0 * H[t] * dH_next"),
    "sign of g_xi": ("t_xi[t] = -r", "t_xi[t] = r"),
    "leak of the dendritic adjoint dropped": ("lam = r + alpha * lam_next if stateful", "lam = r + 0.0 * lam_next if stateful"),
    "g_alpha uses Vd[t] instead of Vd[t-1]": ("t_alpha[t] = lam * Vd[t]", "t_alpha[t] = lam * Vd[t + 1]"),
    "psi' sign": ("return u * (u * u - 3.0) * np.exp", "return u * (3.0 - u * u) * np.exp"),
    "tie does not fire": ("(H[t] - v_th >= 0.0)", "(H[t] - v_th > 0.0)"),
    "beta dropped from the leak": ("H[t] = beta * (1.0 - s_prev) * h_prev", "H[t] = (1.0 - s_prev) * h_prev"),
    "reset dropped": ("H[t] = beta * (1.0 - s_prev) * h_prev", "H[t] = beta * h_prev"),
    "atan surrogate missing pi": ("1.0 / (1.0 + (np.pi * x) ** 2)", "1.0 / (1.0 + (x) ** 2)"),
    "zeta multiplies instead of divides": ("u[t] = nrm[t] / zeta_n", "u[t] = nrm[t] * zeta_n"),
    "channel gather transposed (S, C order)": (
        "np.broadcast_to(p[None, :, None, :], (batch, C, S, W))",
        "np.broadcast_to(p.T.reshape(-1)[:C * W].reshape(C, W)[None, :, None, :], (batch, C, S, W))"),
    "mask ignored in the backward": [
        ("live = np.repeat((m_n != 0) & (nrm[t] > 0.0), k, axis=1)", "live = np.repeat(nrm[t] > 0.0, k, axis=1)"),
        ('kstar_n = _per_neuron(rec["kappa"] * rec["m"], batch, C, S)',
         'kstar_n = _per_neuron(rec["kappa"], batch, C, S)')],
    "branch norm without the square root": ("nrm[t] = np.sqrt((d[t] * d[t]).reshape(N, B, k).sum(axis=2))",
                                            "nrm[t] = (d[t] * d[t]).reshape(N, B, k).sum(axis=2)"),
    "compartments grouped with stride B": ("nrm[t] = np.sqrt((d[t] * d[t]).reshape(N, B, k).sum(axis=2))",
                                           "nrm[t] = np.sqrt((d[t] * d[t]).reshape(N, k, B).sum(axis=1))"),
    "branch gradient spread with stride B": ("r = np.where(live, np.repeat(g_u, k, axis=1)",
                                             "r = np.where(live, np.tile(g_u, (1, k))"),
    "norm gradient divides by the squared norm": (
        "unit = np.where(live, d[t] / np.where(live, np.repeat(nrm[t], k, axis=1), 1.0), 0.0)",
        "unit = np.where(live, d[t] / np.where(live, np.repeat(nrm[t] ** 2, k, axis=1), 1.0), 0.0)"),
    "g_zeta missing 1/zeta": ("-g_u * u[t] / zeta_n", "-g_u * u[t]"),
    "sigmoid surrogate scale dropped": ("return scale * s * (1.0 - s)", "return s * (1.0 - s)"),
    "residual gradient dropped": ('gX[t] = lam + dH[t][:, None] / P if rec["residual"] else lam',
                                  'gX[t] = lam'),
    "residual uses the sum, not the mean": ("Z[t] = Z[t] + X[t].sum(axis=1) / P", "Z[t] = Z[t] + X[t].sum(axis=1)"),
    "residual divides by the branch count": ("Z[t] = Z[t] + X[t].sum(axis=1) / P", "Z[t] = Z[t] + X[t].sum(axis=1) / B"),
    "g_beta uses H[t] instead of H[t-1]": ("t_beta[t] = dH[t] * (1.0 - Sp[t - 1]) * H[t - 1]",
                                           "t_beta[t] = dH[t] * (1.0 - Sp[t - 1]) * H[t]"),
    "g_beta ignores the reset": ("t_beta[t] = dH[t] * (1.0 - Sp[t - 1]) * H[t - 1]",
                                 "t_beta[t] = dH[t] * H[t - 1]"),
    "stateless still leaks": ("Vd[t + 1] = alpha * Vd[t] + X[t] if stateful else X[t]",
                              "Vd[t + 1] = alpha * Vd[t] + X[t]"),
}

# Pins that run in well under a second each, with fixed parameters.
PIN_CALLS = [
    lambda: pins.test_worked_example_forward_exact(),
    lambda: pins.test_worked_example_backward_by_hand(),
    lambda: pins.test_worked_example_backward_vs_autograd("sigmoid", False),
    lambda: pins.test_single_step_closed_form("mexhat", "atan"),
    lambda: pins.test_constant_drive_mexican_hat_zero_input(),
    lambda: pins.test_forward_matches_scalar_stepper("mexhat", True, True, 1),
    lambda: pins.test_forward_matches_scalar_stepper("identity", False, False, 1),
    lambda: pins.test_backward_matches_autograd("mexhat", "sigmoid", False, True, True, False, 1),
    lambda: pins.test_backward_matches_autograd("identity", "atan", False, False, True, False, 1),
    lambda: pins.test_mask_invariants(),
    lambda: pins.test_backward_matches_autograd("mexhat", "sigmoid", False, True, True, True, 1),
    lambda: pins.test_residual_with_zero_strengths_is_lif_of_the_mean_input(),
    lambda: pins.test_plif_beta_gradient_of_a_free_leak(),
    lambda: pins.test_two_compartment_worked_example_by_hand(),
    lambda: pins.test_forward_matches_scalar_stepper("mexhat", True, True, 3),
    lambda: pins.test_backward_matches_autograd("mexhat", "sigmoid", False, True, True, False, 2),
    lambda: pins.test_backward_matches_autograd("identity", "atan", False, True, False, True, 3),
]


def _mutant_module(edits):
    src = open(real.__file__).read()
    for src_from, src_to in edits:
        assert src.count(src_from) >= 1, f"mutation anchor not found: {src_from!r}"
        src = src.replace(src_from, src_to)
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src, "oracle_mutant", "exec"), mod.__dict__)
    return mod


def test_unmutated_oracle_passes_every_pin_call():
    for call in PIN_CALLS:
        call()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    edits = MUTANTS[name]
    mod = _mutant_module(edits if isinstance(edits, list) else [edits])
    monkeypatch.setattr(pins, "oracle", mod)
    caught = []
    for i, call in enumerate(PIN_CALLS):
        try:
            call()
        except (AssertionError, ValueError, FloatingPointError):
            caught.append(i)
    assert caught, f"no pin detects the planted mistake: {name}"
