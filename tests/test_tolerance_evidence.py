"""Evidence behind the parity tolerances (tests/parity.py): what a plain float32
evaluation of the equations (tests/fp32_eval.py) reaches against the float64
oracle, on the layers the GPU parity tests use.

- The float32 evaluation computes the same function as the oracle: on short
  layers it agrees to float32 rounding (a dropped term or a wrong sign in it
  would show as an O(1) error).
- On four-step layers with alpha = beta = 1/2 float32 meets rtol = 1e-5, so
  their bound is rtol (or, for the cifar-shaped grad_x where float32 reaches
  5.3e-6, barely above it).
- On the long-horizon layer (T = 64, alpha = 0.8, beta = 0.9) float32 cannot
  reach rtol on grad_x: the measured error is about 2.7e-5, so the bound there
  is twice that (about 5.4e-5), where a formula over the chains' memories had
  allowed 1.25e-4.
- The full-size harness (tests/fullsize.py) passes a float32-accurate result
  and rejects one with a planted error.
"""

import numpy as np
import pytest

import paper_2412_06355_amd as dendsn
from tests import fp32_eval
from tests.parity import (FP32_MARGIN, RTOL_F32, fp32_errors, make_case, oracle_grads, run_oracle,
                          tolerance)


def _cfg(**kw):
    base = dict(T=4, batch=2, C=256, S=1, B=4, beta=0.5, v_th=1.0, psi="mexhat", sg="sigmoid", sg_scale=4.0)
    base.update(kw)
    return dendsn.DendSNConfig(**base)


def _errors(cfg, **kw):
    case = make_case(cfg, **kw)
    rec = run_oracle(case)
    og = oracle_grads(case, rec)
    return fp32_errors(case, rec, og)


@pytest.mark.parametrize("variant", ["mexhat-sigmoid", "identity-atan", "mask-residual", "kc2-stateless",
                                     "kc4-detach", "plif"])
def test_fp32_evaluation_computes_the_oracles_function(variant):
    c = _cfg(T=6, batch=2, C=24, S=3, B=4, beta=0.7,
             psi="identity" if "identity" in variant else "mexhat",
             sg="atan" if "atan" in variant else "sigmoid",
             residual="residual" in variant, stateful="stateless" not in variant,
             detach_reset="detach" in variant,
             comps_per_branch=2 if "kc2" in variant else (4 if "kc4" in variant else 1))
    e = _errors(c, seed=3, x_std=1.2, alpha=0.6, mask_rho=0.6 if "mask" in variant else None,
                with_gv=True, beta_dev=0.8 if variant == "plif" else None)
    for k, v in e.items():
        assert v < RTOL_F32, (k, v)


@pytest.mark.parametrize("shape", [dict(T=4, batch=2, C=256, S=1, B=4),
                                   dict(T=4, batch=1, C=128, S=1024, B=8)])
def test_fp32_meets_rtol_on_four_step_layers(shape):
    e = _errors(_cfg(**shape), seed=7, x_std=0.5, random_affine=False)
    for k, v in e.items():
        assert v < RTOL_F32, (k, v)
        assert tolerance(RTOL_F32, v) <= FP32_MARGIN * RTOL_F32


def test_long_horizon_needs_more_than_rtol_in_fp32():
    """The reduced long-horizon layer of the GPU parity tests (batch 2 of 32)."""
    c = _cfg(T=64, batch=2, C=4096, S=1, B=16, beta=0.9, ckpt_every=8)
    e = _errors(c, seed=7, x_mean=0.1, alpha=0.8, random_affine=False)
    # grad_x: the adjoint of two leaky chains over 64 steps, through a steep surrogate
    assert 1.5e-5 < e["grad_x"] < 5e-5, e["grad_x"]
    tol = tolerance(RTOL_F32, e["grad_x"])
    assert tol == FP32_MARGIN * e["grad_x"] and tol < 1e-4
    # the potential itself and the summed gradients stay inside rtol
    for k in ("v_soma", "g_kappa", "g_xi", "g_zeta", "g_alpha", "g_beta"):
        assert tolerance(RTOL_F32, e[k]) == RTOL_F32, (k, e[k])


def _write(path, a):
    mm = np.memmap(path, dtype=np.float32, mode="w+", shape=a.shape)
    mm[...] = a
    mm.flush()
    return (str(path), list(a.shape))


@pytest.mark.parametrize("plant", [False, True])
def test_full_size_harness_accepts_fp32_and_rejects_a_planted_error(tmp_path, plant):
    """check_item on one batch item whose 'kernel' outputs come from the float32
    evaluation: it must pass; with one grad_x element off by 3x its bound, fail."""
    from tests.fullsize import check_item, judge_elementwise

    c = _cfg(T=16, batch=2, C=64, S=1, B=8, beta=0.9, ckpt_every=4)
    case = make_case(c, seed=5, x_mean=0.1, alpha=0.8, random_affine=False)
    rec = run_oracle(case)
    og = oracle_grads(case, rec)
    r = fp32_eval.evaluate(case.X, rec["S"], case.gS, alpha=case.alpha, beta=c.beta, v_th=c.v_th,
                           kappa=case.kappa, C=c.C, S=c.S, psi=c.psi, stateful=c.stateful, k=1, sg=c.sg,
                           sg_scale=c.sg_scale)
    gX = r["gX"].copy()
    if plant:
        M = c.C * c.S
        o = og["gX"][:, M:2 * M]          # batch item 1, the one checked below
        scale = np.abs(o) + np.sqrt(np.mean(o * o))
        t, n, b = np.unravel_index(np.argmax(np.abs(o)), o.shape)
        bound = tolerance(RTOL_F32, fp32_eval.elementwise_ratio(r["gX"][:, M:2 * M], o)) * scale[t, n, b]
        gX[t, M + n, b] = o[t, n, b] + 3 * bound
    files = dict(X=_write(tmp_path / "X", case.X), gS=_write(tmp_path / "gS", case.gS),
                 S=_write(tmp_path / "S", rec["S"].astype(np.float32)), H=_write(tmp_path / "H", r["H"]),
                 gX=_write(tmp_path / "gX", gX))
    params = dict(alpha=case.alpha, beta=c.beta, v_th=c.v_th, kappa=case.kappa, xi=None, zeta=None, mask=None,
                  C=c.C, S=c.S, psi=c.psi, stateful=c.stateful, residual=False, k=1, sg=c.sg,
                  sg_scale=c.sg_scale, detach=False)
    res = check_item(dict(item=1, M=c.C * c.S, T=c.T, params=params, rtol_io=RTOL_F32, **files))
    assert res["error"] is None, res["error"]
    errors = judge_elementwise([res], RTOL_F32)
    if plant:
        assert errors and "grad_x" in errors[0]
    else:
        assert not errors, errors
