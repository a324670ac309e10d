"""The largest sample slice the library takes: lane byte offsets inside one
sample's [C, S, P] slice are 32-bit, so the layer below sits just under that
limit (255 channels of 2^20 positions, 4 fp32 branches: 4,278,190,080 bytes per
sample), with two samples and an interior checkpoint (X, grad_x and the
checkpoint each span more than 4 GiB).  Sampled neurons — the first and last of
each sample, the last channel's final tile and a random spread — are checked
against the float64 oracle one by one (spikes under the forced-spike protocol,
v_soma and grad_x elementwise); neurons are independent, so each is an oracle
layer of its own with its channel's parameters.  Needs ~60 GB of device memory."""

import numpy as np
import pytest

import oracle
import paper_2412_06355_amd as dendsn
from tests.parity import BAND, RTOL_F32, announce

pytestmark = pytest.mark.gpu


def test_largest_sample_slice(gpu_device):
    import torch

    T, batch, C, S, B = 2, 2, 255, 1 << 20, 4
    cfg = dendsn.DendSNConfig(T=T, batch=batch, C=C, S=S, B=B, ckpt_every=1, beta=0.5, v_th=1.0,
                              psi="mexhat", sg="sigmoid", sg_scale=4.0)
    M, N = C * S, batch * C * S
    assert M * B * 4 < 2**32 <= (M + S) * B * 4  # one more channel would exceed the limit
    announce(f"largest sample slice: T={T} batch={batch} C={C} S={S} B={B} fp32, N={N}")
    g = torch.Generator(device=gpu_device)
    g.manual_seed(11)
    X = torch.empty((T, N, B), dtype=torch.float32, device=gpu_device).normal_(0.0, 1.0, generator=g)
    gS = torch.empty((T, N), dtype=torch.float32, device=gpu_device).normal_(0.0, 1.0, generator=g)
    kappa = torch.empty((C, B), dtype=torch.float32, device=gpu_device).uniform_(0.0, 1.0, generator=g)
    alpha = torch.tensor([0.5], dtype=torch.float32, device=gpu_device)
    spikes, v_soma, ckpt = dendsn.forward(cfg, X, alpha, kappa, want_v_soma=True)
    assert ckpt is not None and ckpt.numel() * 4 > 2**32
    grads = dendsn.backward(cfg, X, alpha, kappa, None, None, None, ckpt, gS)
    torch.cuda.synchronize(gpu_device)

    rng = np.random.default_rng(5)
    idx = np.unique(np.concatenate([
        [0, M - 1, M, N - 1],
        np.arange(N - 512, N),                     # the last channel's final tile of the last sample
        np.arange(M - 512, M),                     # ... and of the first sample
        rng.integers(0, N, 1500),
    ]))
    it = torch.from_numpy(idx).to(gpu_device)
    f = lambda t: t.index_select(1, it).double().cpu().numpy()
    Xs, gSs, Sg, Hg, gXg = f(X), f(gS), f(spikes), f(v_soma), f(grads["grad_x"])
    kap = kappa.double().cpu().numpy()[(idx % M) // S]          # each sampled neuron's channel
    del X, gS, spikes, v_soma, ckpt, grads
    torch.cuda.empty_cache()

    # every sampled neuron as a channel of its own (C = n, S = 1)
    n = len(idx)
    kw = dict(alpha=0.5, beta=0.5, v_th=1.0, kappa=kap, C=n, S=1, psi_kind="mexhat", stateful=True)
    force = -np.ones((T, n), dtype=np.int64)
    exempt = 0
    for _ in range(T + 1):
        rec = oracle.forward(Xs, force=force if exempt else None, **kw)
        diff = rec["S"] != Sg
        if not diff.any():
            break
        cols = np.nonzero(diff.any(axis=0))[0]
        t_first = diff[:, cols].argmax(axis=0)
        dist = np.abs(rec["H"][t_first, cols] - 1.0)
        assert np.all(dist <= BAND), f"spike mismatch outside the band: {float(dist.max()):.3e}"
        force[t_first, cols] = Sg[t_first, cols].astype(np.int64)
        exempt += len(cols)
    else:
        pytest.fail("forced-spike protocol did not converge")
    og = oracle.backward(rec, gSs, sg_kind="sigmoid", sg_scale=4.0)
    for name, got, ref in (("v_soma", Hg, rec["H"]), ("grad_x", gXg, og["gX"])):
        scale = np.abs(ref) + np.sqrt(np.mean(ref * ref))
        err = float(np.max(np.abs(got - ref) / scale))
        assert err <= RTOL_F32, (name, err)
    announce(f"largest sample slice: {n} sampled neurons match the oracle ({exempt} near-threshold exemptions)")
