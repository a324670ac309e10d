"""Empty layers (no neuron-step: T, batch, C or S of 0) through the C ABI on the
GPU.  The forward accepts them and writes nothing; both backward entry points
write +0 to every parameter gradient requested (sums with no terms), as the
oracle does for the same layer; the Python conveniences return empty outputs."""

import numpy as np
import pytest

import paper_2412_06355_amd as dendsn
from oracle import dendsn_oracle as oracle
from tests.parity import announce

pytestmark = pytest.mark.gpu

EMPTY = [
    dict(T=0, batch=2, C=16, S=4, B=4),
    dict(T=8, batch=0, C=16, S=4, B=4, ckpt_every=4),
    dict(T=4, batch=2, C=0, S=4, B=8),
    dict(T=4, batch=2, C=16, S=0, B=8, io="bf16"),
    dict(T=4, batch=3, C=8, S=0, B=5, comps_per_branch=2, stateful=False),
    dict(T=0, batch=0, C=0, S=0, B=4, residual=True),
    dict(T=64, batch=0, C=4096, S=1, B=16, ckpt_every=8),
    dict(T=4, batch=2, C=32, S=0, B=8, layout="channel_major"),
]


def _cfg(kw):
    base = dict(beta=0.5, v_th=1.0, psi="mexhat", sg="sigmoid", sg_scale=4.0)
    base.update(kw)
    return dendsn.DendSNConfig(**base)


def _inputs(cfg, device):
    import torch

    io = torch.bfloat16 if cfg.io == "bf16" else torch.float32
    g = torch.Generator(device="cpu").manual_seed(5)
    shape = (cfg.T, cfg.batch, cfg.C, cfg.P, cfg.S) if cfg.layout == "channel_major" else (cfg.T, cfg.N, cfg.P)
    rnd = lambda *s: torch.rand(*s, generator=g).to(device)
    return dict(
        x=torch.empty(shape, dtype=io, device=device),
        alpha=torch.tensor([0.5], dtype=torch.float32, device=device),
        kappa=rnd(cfg.C, cfg.B),
        xi=rnd(cfg.C, cfg.P) - 0.5,
        zeta=rnd(cfg.C, cfg.B) + 0.5,
        mask=(rnd(cfg.C, cfg.B) < 0.5).to(torch.uint8),
        gS=torch.empty((cfg.T, cfg.N), dtype=io, device=device),
    )


def _poisoned_grads(cfg, device):
    import torch

    nan = lambda *s: torch.full(s, float("nan"), dtype=torch.float32, device=device)
    return dict(grad_alpha=nan(1), grad_beta=nan(1), grad_kappa=nan(cfg.C, cfg.B), grad_xi=nan(cfg.C, cfg.P),
                grad_zeta=nan(cfg.C, cfg.B))


def _assert_positive_zero(name, t):
    import torch

    bits = t.contiguous().view(torch.int32)
    assert bool((bits == 0).all()), (name, t)


@pytest.mark.parametrize("kw", EMPTY, ids=lambda kw: ",".join(f"{k}={v}" for k, v in kw.items()))
def test_empty_layer(gpu_device, kw):
    import torch

    cfg = _cfg(kw)
    announce(f"empty layer: {cfg}")
    assert dendsn.dendsn_ckpt_bytes(cfg) == 0
    d = _inputs(cfg, gpu_device)
    spikes, v_soma, ckpt = dendsn.forward(cfg, d["x"], d["alpha"], d["kappa"], d["xi"], d["zeta"], d["mask"],
                                          want_v_soma=True)
    assert spikes.shape == (cfg.T, cfg.N) and v_soma.shape == (cfg.T, cfg.N) and ckpt is None

    # the oracle on the same (empty) layer: every gradient an empty sum
    rec = oracle.forward(np.zeros((cfg.T, cfg.N, cfg.P)), alpha=0.5, beta=cfg.beta, v_th=cfg.v_th,
                         kappa=d["kappa"].cpu().numpy(), xi=d["xi"].cpu().numpy(), zeta=d["zeta"].cpu().numpy(),
                         mask=d["mask"].cpu().numpy(), C=cfg.C, S=cfg.S, psi_kind=cfg.psi, stateful=cfg.stateful,
                         residual=cfg.residual, comps_per_branch=cfg.comps_per_branch)
    ref = oracle.backward(rec, np.zeros((cfg.T, cfg.N)), sg_kind=cfg.sg, sg_scale=cfg.sg_scale)

    gx = torch.empty_like(d["x"])
    ws = torch.empty(((dendsn.dendsn_bwd_workspace_bytes(cfg) + 3) // 4,), dtype=torch.float32, device=gpu_device)
    for entry in ("workspace", "noalloc"):
        out = _poisoned_grads(cfg, gpu_device)
        args = (cfg, d["x"], d["alpha"], None, d["kappa"], d["xi"], d["zeta"], d["mask"], None, d["gS"], None, gx,
                out["grad_alpha"], out["grad_beta"], out["grad_kappa"], out["grad_xi"], out["grad_zeta"])
        if entry == "workspace":
            dendsn.dendsn_backward(*args, ws)
        else:
            dendsn.dendsn_backward_noalloc(*args)
        torch.cuda.synchronize(gpu_device)
        for k, v in out.items():
            _assert_positive_zero(f"{entry}/{k}", v)
        np.testing.assert_array_equal(out["grad_kappa"].cpu().numpy(), ref["g_kappa"])
        np.testing.assert_array_equal(out["grad_xi"].cpu().numpy(), ref["g_xi"])
        np.testing.assert_array_equal(out["grad_zeta"].cpu().numpy(), ref["g_zeta"])
        assert out["grad_alpha"].item() == ref["g_alpha"] and out["grad_beta"].item() == ref["g_beta"]

    g = dendsn.backward(cfg, d["x"], d["alpha"], d["kappa"], d["xi"], d["zeta"], d["mask"], ckpt, d["gS"])
    torch.cuda.synchronize(gpu_device)
    assert g["grad_x"].shape == d["x"].shape
    for k in ("grad_alpha", "grad_beta", "grad_kappa", "grad_xi", "grad_zeta"):
        _assert_positive_zero(k, g[k])
