"""Seeded synthetic workloads for the DendSN layer scan.

This module only draws random inputs and names shapes; it holds none of the
neuron model's arithmetic, so both the float64 oracle (in tests) and the HIP
library's callers can take their inputs from it without sharing any of the
method's code.

The paper's datasets are not used: each workload stands in for a layer shape
the paper trains (spiking convolutions on 32x32 CIFAR-like inputs, an
ImageNet-sized stem, a long-horizon fully connected layer, the task-incremental
fully connected layer with dendritic branch gating), with inputs drawn i.i.d.
from the stated normal distribution.

Layout: X and its gradient are [T, N, P] with the P = B k compartments
innermost (k per branch, a branch's compartments adjacent) and neurons ordered
(batch, channel, spatial), N = batch * C * S.  Spikes and their gradient are
[T, N].  Per-channel parameters are [C, B] (kappa, zeta, gating mask) and
[C, P] (xi).
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    T: int
    batch: int
    C: int
    S: int
    B: int
    io: str = "f32"              # "f32" or "bf16" storage of X, spikes, gX, gS
    x_mean: float = 0.0
    x_std: float = 1.0
    alpha: float = 0.5           # dendritic decay (learnable, shared by the layer)
    beta: float = 0.5            # somatic decay
    v_th: float = 1.0
    psi: str = "mexhat"
    sg: str = "sigmoid"
    sg_scale: float = 4.0
    ckpt_every: int = 0          # 0: no interior checkpoint (K >= T)
    tasks: int = 0               # >0: one branch-gating mask per task, q = 1..tasks
    mask_rho: float = 0.5
    stateful: bool = True
    detach_reset: bool = False
    comps_per_branch: int = 1    # k = P / B
    residual: bool = False       # residual dendrite (ResStateful / ResStateless)
    layout: str = "npb"          # X / grad_x layout: [T, N, P] or "channel_major" [T, batch, C, P, S]

    @property
    def N(self) -> int:
        return self.batch * self.C * self.S

    @property
    def P(self) -> int:
        return self.B * self.comps_per_branch

    @property
    def nbs(self) -> int:
        """Neuron-branch-steps of one forward (or one backward) pass."""
        return self.T * self.N * self.B

    @property
    def K(self) -> int:
        return self.ckpt_every if self.ckpt_every > 0 else self.T

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # T=4, batch 2, 256 neurons per sample, 4 branches; the oracle finishes instantly.
    "tiny": Workload("tiny", T=4, batch=2, C=256, S=1, B=4),
    # Spiking conv activation on 32x32 maps: batch 128, 128 channels, 8 branches.
    "cifar": Workload("cifar", T=4, batch=128, C=128, S=32 * 32, B=8, x_std=0.5),
    # ImageNet-stem-sized activation, 112x112 maps, bf16 storage with fp32 state.
    "imagenet_stem": Workload("imagenet_stem", T=4, batch=32, C=64, S=112 * 112, B=4, io="bf16"),
    # Long-horizon fully connected layer with a state checkpoint every 8 steps.
    "long_horizon": Workload("long_horizon", T=64, batch=32, C=4096, S=1, B=16, x_mean=0.1,
                             alpha=0.8, beta=0.9, ckpt_every=8),
    # Task-incremental fully connected layer with a per-task branch-gating mask.
    "dbg": Workload("dbg", T=4, batch=64, C=8192, S=1, B=32, tasks=10, mask_rho=0.5),
    "cifar_b16": Workload("cifar_b16", T=4, batch=64, C=128, S=32 * 32, B=16, x_std=0.5),
    # The CIFAR-shaped layer with bf16 storage.
    "cifar_bf16": Workload("cifar_bf16", T=4, batch=128, C=128, S=32 * 32, B=8, x_std=0.5, io="bf16"),
    # The paper's common dendrite (P = 4 compartments on B = 2 branches) on the
    # CIFAR-shaped conv activation.
    "cifar_p4b2": Workload("cifar_p4b2", T=4, batch=128, C=128, S=32 * 32, B=2, comps_per_branch=2, x_std=0.5),
    "cifar_p4b2_bf16": Workload("cifar_p4b2_bf16", T=4, batch=128, C=128, S=32 * 32, B=2, comps_per_branch=2,
                                x_std=0.5, io="bf16"),
    # The same layer consuming the producing conv layer's output as it is laid
    # out, [T, batch, C P, H, W] (groups of P consecutive feature maps).
    "cifar_p4b2_cm": Workload("cifar_p4b2_cm", T=4, batch=128, C=128, S=32 * 32, B=2, comps_per_branch=2, x_std=0.5,
                              layout="channel_major"),
    "cifar_cm": Workload("cifar_cm", T=4, batch=128, C=128, S=32 * 32, B=8, x_std=0.5, layout="channel_major"),
    # ResStateless dendrite (Tiny-ImageNet-style deep network: 64x64 maps),
    # identity activation, P = 4 on B = 2.
    "tiny_imagenet_res": Workload("tiny_imagenet_res", T=4, batch=64, C=64, S=64 * 64, B=2, comps_per_branch=2,
                                  psi="identity", stateful=False, residual=True),
    # Stateless dendrite on a neuromorphic (CIFAR10-DVS-style) conv layer, T = 10,
    # P = 10 compartments on B = 5 branches (one lane holds a whole neuron).
    # A state checkpoint every 4 steps keeps the backward's re-advance short.
    "dvs_p10b5": Workload("dvs_p10b5", T=10, batch=16, C=128, S=32 * 32, B=5, comps_per_branch=2,
                          stateful=False, ckpt_every=4),
    # The same layer with the stateful dendrite (leak alpha = 0.5): the paper's
    # cost ordering of the dendrite variants on one shape.
    "dvs_p10b5_stateful": Workload("dvs_p10b5_stateful", T=10, batch=16, C=128, S=32 * 32, B=5,
                                   comps_per_branch=2, ckpt_every=4),
}


def branch_mask(C: int, B: int, task: int, rho: float = 0.5) -> np.ndarray:
    """Per-task gating mask [C, B] of {0, 1}: i.i.d. Bernoulli(rho), fixed by the
    task index (the same task always draws the same mask)."""
    return (np.random.default_rng(task).random((C, B)) < rho).astype(np.uint8)


def params(wl: Workload, seed: int = 0, random_affine: bool = False):
    """Branch strengths kappa ~ U(0, 1) per channel; xi = 0, zeta = 1 unless
    ``random_affine`` (then xi ~ N(0, 0.5), zeta ~ U(0.5, 2))."""
    rng = np.random.default_rng([seed, 1])
    kappa = rng.uniform(0.0, 1.0, size=(wl.C, wl.B)).astype(np.float32)
    if random_affine:
        xi = rng.normal(0.0, 0.5, size=(wl.C, wl.P)).astype(np.float32)
        zeta = rng.uniform(0.5, 2.0, size=(wl.C, wl.B)).astype(np.float32)
    else:
        xi = np.zeros((wl.C, wl.P), np.float32)
        zeta = np.ones((wl.C, wl.B), np.float32)
    return dict(kappa=kappa, xi=xi, zeta=zeta)


def _torch_dtype(io: str):
    import torch

    return {"f32": torch.float32, "bf16": torch.bfloat16}[io]


def activations(wl: Workload, device="cpu", seed: int = 0, batch: int | None = None):
    """X [T, N, P] ~ N(x_mean, x_std) (i.i.d., so the same draw serves the
    channel-major layout) and the spike gradient gS [T, N] ~ N(0, 1),
    drawn in float32 by torch's generator on ``device`` and then stored in the
    workload's I/O dtype (bf16 by round-to-nearest-even)."""
    import torch

    b = wl.batch if batch is None else batch
    N = b * wl.C * wl.S
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    dt = _torch_dtype(wl.io)
    X = torch.empty((wl.T, N, wl.P), dtype=torch.float32, device=device)
    X.normal_(wl.x_mean, wl.x_std, generator=g)
    gS = torch.empty((wl.T, N), dtype=torch.float32, device=device)
    gS.normal_(0.0, 1.0, generator=g)
    if dt != torch.float32:
        X = X.to(dt)
        gS = gS.to(dt)
    return X, gS
