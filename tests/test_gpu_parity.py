"""GPU parity: the HIP library (through the C ABI) against the float64 oracle,
element by element, on seeded inputs (see tests/parity.py for the protocol).

Sizes are ones the oracle finishes in seconds, chosen to span several tiles,
every tiling mode (spatial tiles, fully connected tiles, multi-channel tiles),
every lane mapping, ragged tails in space, batch and time, and chunked /
checkpointed backward segments.
"""

import zlib

import numpy as np
import pytest

import paper_2412_06355_amd as dendsn
from tests.parity import announce, compare, make_case, run_gpu, to_device

pytestmark = pytest.mark.gpu


def cfg(**kw):
    base = dict(T=4, batch=2, C=256, S=1, B=4, beta=0.5, v_th=1.0, psi="mexhat", sg="sigmoid", sg_scale=4.0)
    base.update(kw)
    return dendsn.DendSNConfig(**base)


# --- the tiny layer: T=4, batch 2, 256 neurons, 4 branches, X ~ N(0,1) seed 0 ---
@pytest.mark.parametrize("psi", ["mexhat", "identity"])
@pytest.mark.parametrize("sg", ["sigmoid", "atan"])
@pytest.mark.parametrize("detach", [False, True])
def test_tiny_layer(gpu_device, psi, sg, detach):
    c = cfg(psi=psi, sg=sg, detach_reset=detach)
    case = make_case(c, seed=0, random_affine=False, name=f"tiny/{psi}/{sg}/detach={detach}")
    rep = compare(case, run_gpu(case, gpu_device))
    print(rep)


def test_tiny_layer_with_grad_v_soma(gpu_device):
    case = make_case(cfg(), seed=1, with_gv=True, name="tiny/gV")
    compare(case, run_gpu(case, gpu_device))


# --- shapes covering tiling modes, lane mappings and ragged tails ---
SHAPES = [
    # T, batch, C, S, B, io, K
    (1, 3, 5, 1, 1, "f32", 1),
    (2, 2, 3, 7, 2, "f32", 2),
    (3, 1, 4, 300, 3, "f32", 3),
    (5, 3, 6, 5, 5, "bf16", 2),
    (7, 2, 9, 64, 6, "f32", 3),
    (9, 2, 3, 130, 7, "f32", 4),
    (6, 5, 11, 1, 10, "f32", 6),
    (5, 2, 7, 3, 12, "bf16", 5),
    (4, 3, 70, 1, 16, "f32", 4),
    (4, 2, 40, 1, 32, "f32", 4),
    (4, 2, 20, 1, 64, "f32", 2),
    (3, 2, 8, 1, 128, "bf16", 3),
    (4, 3, 5, 513, 8, "bf16", 4),
    (4, 2, 3, 257, 4, "bf16", 4),
    (11, 2, 3, 33, 4, "f32", 5),
    (17, 2, 9, 1, 16, "f32", 17),
    (20, 2, 5, 1, 4, "f32", 20),
    (16, 3, 3, 2, 8, "f32", 16),
    (13, 2, 6, 1, 8, "bf16", 13),
    (10, 2, 4, 100, 2, "f32", 10),
    (6, 2, 20, 1, 16, "bf16", 3),     # bf16 backward splits a neuron differently from the forward
    # fp32 16 branches: the forward holds 8 per lane over two lanes (32-byte rows,
    # staged), the backward 4 over four; conv tiles with four positions per lane
    (4, 2, 3, 700, 16, "f32", 4),     # forward fast path, a ragged last tile
    (5, 2, 3, 600, 16, "f32", 3),     # general forward path with checkpoints
    (8, 2, 2, 1100, 16, "f32", 4),    # padded-free T = 8 with an interior checkpoint
    (4, 2, 9, 40, 32, "bf16", 4),
    (5, 2, 3, 1, 64, "bf16", 2),
    # fully connected, 8 or more lanes per neuron: the backward's two batch ways
    # with an odd batch and a last tile of one channel
    (5, 3, 33, 1, 32, "f32", 2),
    (4, 3, 17, 1, 32, "bf16", 4),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "T{}b{}C{}S{}B{}{}K{}".format(*s))
@pytest.mark.parametrize("variant", ["mh-sig-mask", "id-atan-stateless", "mh-atan-detach",
                                     "res-mh-sig-mask-plif", "res-id-atan-stateless"])
def test_shapes(gpu_device, shape, variant):
    T, batch, C, S, B, io, K = shape
    psi = "identity" if "-id-" in f"-{variant}-" else "mexhat"
    sg = "sigmoid" if "sig" in variant else "atan"
    c = cfg(T=T, batch=batch, C=C, S=S, B=B, io=io, ckpt_every=K, psi=psi, sg=sg,
            stateful="stateless" not in variant, detach_reset="detach" in variant, beta=0.7,
            residual=variant.startswith("res"))
    seed = zlib.crc32(repr((shape, variant)).encode()) % 1000
    case = make_case(c, seed=seed, x_std=1.2, alpha=0.6,
                     mask_rho=0.5 if "mask" in variant else None, name=f"{shape}/{variant}",
                     beta_dev=0.8 if "plif" in variant else None)
    compare(case, run_gpu(case, gpu_device))


# --- four-step spatial backward with two positions per lane (whole tiles) ---
NW2_SHAPES = [
    # T, batch, C, S, B, k, io
    (4, 3, 5, 256, 8, 1, "f32"),
    (4, 2, 3, 1024, 4, 1, "bf16"),
    (4, 5, 2, 512, 16, 1, "f32"),
    (4, 2, 4, 512, 2, 2, "f32"),
    (4, 3, 2, 1024, 8, 1, "bf16"),
    (4, 2, 3, 256, 32, 1, "f32"),
    (4, 3, 2, 1024, 8, 1, "f32"),      # four positions per lane
    (4, 2, 2, 512, 4, 4, "f32"),
]


@pytest.mark.parametrize("shape", NW2_SHAPES, ids=lambda s: "T{}b{}C{}S{}B{}k{}{}".format(*s))
@pytest.mark.parametrize("variant", ["mh-sig-mask", "res-id-atan-stateless-plif"])
def test_two_positions_per_lane(gpu_device, shape, variant):
    T, batch, C, S, B, k, io = shape
    c = cfg(T=T, batch=batch, C=C, S=S, B=B, comps_per_branch=k, io=io,
            psi="identity" if "-id-" in f"-{variant}-" else "mexhat", sg="sigmoid" if "sig" in variant else "atan",
            stateful="stateless" not in variant, residual=variant.startswith("res"), beta=0.7)
    seed = zlib.crc32(repr((shape, variant, "nw2")).encode()) % 1000
    case = make_case(c, seed=seed, x_std=1.2, alpha=0.6, mask_rho=0.5 if "mask" in variant else None,
                     name=f"nw2/{shape}/{variant}", beta_dev=0.8 if "plif" in variant else None, with_gv=True)
    compare(case, run_gpu(case, gpu_device))


# --- the forward with several positions per lane and batch item, any length ---
FWD_NW_SHAPES = [
    # T, batch, C, S, B, k, io, K, layout, batch_groups
    (7, 3, 2, 1024, 8, 1, "f32", 3, "npb", 0),       # 4 positions over 2 lanes, padded chunk, checkpoints
    (5, 5, 2, 512, 4, 1, "f32", 2, "npb", 0),        # 2 positions, one lane; ragged batch groups
    (6, 2, 3, 1024, 16, 1, "bf16", 4, "npb", 0),     # bf16 over 2 lanes
    (9, 3, 2, 512, 2, 2, "f32", 4, "channel_major", 0),
    (4, 6, 1, 2048, 8, 1, "f32", 4, "npb", 2),       # 3 batch items x 4 positions per lane
    (3, 2, 2, 768, 8, 1, "f32", 2, "npb", 0),        # S = 768: 2 positions
]


@pytest.mark.parametrize("shape", FWD_NW_SHAPES, ids=lambda s: "T{}b{}C{}S{}B{}k{}{}K{}{}g{}".format(*s))
@pytest.mark.parametrize("variant", ["mh-sig-mask", "res-id-atan-stateless-plif"])
def test_forward_positions_per_lane(gpu_device, shape, variant):
    T, batch, C, S, B, k, io, K, layout, groups = shape
    c = cfg(T=T, batch=batch, C=C, S=S, B=B, comps_per_branch=k, io=io, ckpt_every=K, layout=layout,
            batch_groups=groups, psi="identity" if "-id-" in f"-{variant}-" else "mexhat",
            sg="sigmoid" if "sig" in variant else "atan", stateful="stateless" not in variant,
            residual=variant.startswith("res"), beta=0.7)
    seed = zlib.crc32(repr((shape, variant, "fwd-nw")).encode()) % 1000
    case = make_case(c, seed=seed, x_std=1.2, alpha=0.6, mask_rho=0.5 if "mask" in variant else None,
                     name=f"fwd-nw/{shape}/{variant}", beta_dev=0.8 if "plif" in variant else None, with_gv=True)
    compare(case, run_gpu(case, gpu_device))


# --- fully connected layers large enough for XCD runs of 32 blocks ---
@pytest.mark.parametrize("shape", [(8, 32, 2048, 16, "f32", 4), (4, 64, 1024, 32, "f32", 4),
                                   (6, 32, 8192, 8, "bf16", 3)],
                         ids=lambda s: "T{}b{}C{}B{}{}K{}".format(*s))
def test_fully_connected_xcd_runs(gpu_device, shape):
    T, batch, C, B, io, K = shape
    c = cfg(T=T, batch=batch, C=C, S=1, B=B, io=io, ckpt_every=K, beta=0.7)
    seed = zlib.crc32(repr((shape, "fc-xcd")).encode()) % 1000
    case = make_case(c, seed=seed, x_std=1.2, alpha=0.6, mask_rho=0.5, name=f"fc-xcd/{shape}", with_gv=True)
    compare(case, run_gpu(case, gpu_device))


# --- several compartments per branch (L2 norm over a branch's compartments) ---
KC_SHAPES = [
    # T, batch, C, S, B, k, io, K
    (4, 2, 5, 300, 2, 2, "f32", 4),      # fast fp32, one lane per neuron, conv tiles
    (6, 3, 70, 1, 8, 2, "f32", 3),       # fast fp32, 4 lanes per neuron, FC tiles
    (5, 2, 9, 7, 1, 4, "f32", 5),        # fast fp32, k = 4
    (7, 2, 6, 33, 4, 4, "f32", 2),       # fast fp32, k = 4, 4 lanes
    (4, 3, 4, 257, 4, 2, "bf16", 4),     # fast bf16
    (9, 2, 5, 1, 16, 2, "bf16", 4),      # fast bf16, 4 lanes
    (4, 2, 7, 65, 2, 4, "bf16", 4),      # fast bf16, k = 4
    (4, 2, 6, 40, 5, 2, "f32", 4),       # generic: P = 10, B = 5
    (10, 2, 3, 5, 3, 2, "f32", 4),       # generic, checkpoints
    (4, 2, 5, 1, 7, 2, "f32", 4),        # generic, 14 compartments in a lane
    (5, 2, 4, 9, 3, 4, "f32", 5),        # generic, k = 4
    (4, 2, 6, 130, 2, 2, "bf16", 4),     # generic bf16
    (6, 3, 4, 3, 1, 4, "bf16", 6),       # generic bf16, k = 4
    (3, 2, 5, 17, 1, 2, "f32", 3),       # generic, one branch
    # wide lane rows staged through LDS (full, aligned waves) beside unstaged ones
    (4, 2, 3, 300, 5, 2, "f32", 4),      # generic P = 10, conv tiles: a ragged last tile
    (4, 2, 4, 96, 5, 2, "bf16", 4),      # generic bf16 P = 10 (20-byte lane rows), one chunk
    (10, 2, 4, 96, 5, 2, "bf16", 4),     # the same over three checkpoint segments
    (10, 2, 2, 512, 5, 2, "f32", 4),     # P = 10 over 512-position maps: forward one position per lane
]


@pytest.mark.parametrize("shape", KC_SHAPES, ids=lambda s: "T{}b{}C{}S{}B{}k{}{}K{}".format(*s))
@pytest.mark.parametrize("variant", ["mh-sig-mask", "id-atan-stateless-res", "mh-atan-detach-plif-res"])
def test_compartments_per_branch(gpu_device, shape, variant):
    T, batch, C, S, B, k, io, K = shape
    psi = "identity" if "-id-" in f"-{variant}-" else "mexhat"
    c = cfg(T=T, batch=batch, C=C, S=S, B=B, comps_per_branch=k, io=io, ckpt_every=K, psi=psi,
            sg="sigmoid" if "sig" in variant else "atan", stateful="stateless" not in variant,
            detach_reset="detach" in variant, residual="res" in variant, beta=0.7)
    seed = zlib.crc32(repr((shape, variant)).encode()) % 1000
    case = make_case(c, seed=seed, x_std=1.2, alpha=0.6, mask_rho=0.5 if "mask" in variant else None,
                     name=f"kc/{shape}/{variant}", beta_dev=0.8 if "plif" in variant else None)
    compare(case, run_gpu(case, gpu_device))


# Stateful dendrite, fp32 lane rows wider than 16 bytes, one chunk per segment
# (K <= 4) and T != 4: the segment pipeline whose rows and checkpointed state
# arrive in LDS by DMA (full, aligned waves) beside partially active waves that
# keep lane loads.
WIDE_STATEFUL = [
    # T, batch, C, S, B, k, K
    (10, 2, 4, 96, 5, 2, 4),     # P = 10, segments 4, 4, 2; whole channels per tile, last wave partial
    (7, 3, 2, 300, 5, 2, 4),     # conv tiles with a ragged last tile; segments 4, 3
    (6, 2, 3, 128, 3, 2, 2),     # 24-byte lane rows, segments of 2
    (9, 2, 2, 256, 7, 2, 3),     # 56-byte lane rows (a partial last round of pieces), segments of 3
    (3, 2, 4, 64, 5, 2, 3),      # T < 4: one segment of 3 steps
    (6, 2, 2, 256, 3, 4, 4),     # k = 4, 48-byte rows (whole rounds of pieces only); segments 4, 2
    (4, 2, 4, 96, 5, 2, 4),      # T = K = 4: every neuron one segment
    (4, 3, 3, 300, 7, 2, 4),     # T = 4, 56-byte rows, conv tiles with a ragged last tile
    (10, 2, 2, 512, 5, 2, 4),    # 512-position maps: whole tiles, the forward one position per lane
]


@pytest.mark.parametrize("shape", WIDE_STATEFUL, ids=lambda s: "T{}b{}C{}S{}B{}k{}K{}".format(*s))
@pytest.mark.parametrize("variant", ["mh-sig", "mh-sig-mask-gv", "id-atan-detach-plif-res"])
def test_stateful_wide_rows_segment_pipeline(gpu_device, shape, variant):
    T, batch, C, S, B, k, K = shape
    c = cfg(T=T, batch=batch, C=C, S=S, B=B, comps_per_branch=k, ckpt_every=K,
            psi="identity" if variant.startswith("id") else "mexhat", sg="sigmoid" if "sig" in variant else "atan",
            detach_reset="detach" in variant, residual="res" in variant, beta=0.7)
    seed = zlib.crc32(repr((shape, variant)).encode()) % 1000
    case = make_case(c, seed=seed, x_std=1.2, alpha=0.7, mask_rho=0.5 if "mask" in variant else None,
                     with_gv="gv" in variant, name=f"wide-sf/{shape}/{variant}",
                     beta_dev=0.8 if "plif" in variant else None)
    compare(case, run_gpu(case, gpu_device))


@pytest.mark.parametrize("B,k,io", [(5, 2, "f32"), (7, 2, "f32"), (5, 2, "bf16")])
def test_wide_rows_checkpoint_interval_is_bit_invariant(gpu_device, B, k, io):
    """K = 2 and 4 take the stateful segment pipeline (fp32), K = 12 the
    neuron-by-neuron path: spikes and every gradient agree bit for bit."""
    import torch

    base = cfg(T=12, batch=2, C=4, S=64, B=B, comps_per_branch=k, io=io, beta=0.8, ckpt_every=4)
    case = make_case(base, seed=41 + B, x_mean=0.1, alpha=0.7, mask_rho=0.6, name=f"wide-ckpt/{B}/{io}")
    d = to_device(case, gpu_device)
    outs = []
    for K in (4, 12, 2):
        case.cfg = base.with_(ckpt_every=K)
        outs.append(run_gpu(case, gpu_device, dev=d)["raw"])
    for o in outs[1:]:
        assert torch.equal(o["spikes"], outs[0]["spikes"])
        for name in ("grad_x", "grad_alpha", "grad_beta", "grad_kappa", "grad_xi", "grad_zeta"):
            assert torch.equal(_bits(o["grads"][name]), _bits(outs[0]["grads"][name])), name
    compare(case, run_gpu(case, gpu_device, dev=d))


def test_compartments_checkpoint_interval_is_bit_invariant(gpu_device):
    import torch

    base = cfg(T=24, batch=2, C=40, S=1, B=8, comps_per_branch=2, beta=0.9, ckpt_every=8)
    case = make_case(base, seed=23, x_mean=0.1, alpha=0.8, mask_rho=0.7, name="kc-ckpt")
    d = to_device(case, gpu_device)
    outs = []
    for K in (8, 24, 5):
        case.cfg = base.with_(ckpt_every=K)
        outs.append(run_gpu(case, gpu_device, dev=d)["raw"])
    for o in outs[1:]:
        assert torch.equal(o["spikes"], outs[0]["spikes"])
        assert torch.equal(_bits(o["grads"]["grad_x"]), _bits(outs[0]["grads"]["grad_x"]))
    compare(case, run_gpu(case, gpu_device, dev=d))


def test_replicated_compartments_match_one_compartment(gpu_device):
    """k equal compartments (same input and xi) act as one with zeta / sqrt(k): spikes
    agree and each copy gets 1/k of the one-compartment input gradient."""
    k = 4
    one = cfg(T=4, batch=2, C=16, S=64, B=2, psi="identity")
    c1 = make_case(one, seed=24, random_affine=True, name="kc-rep/one")
    ck = make_case(one.with_(comps_per_branch=k), seed=24, name="kc-rep/k")
    ck.X = np.repeat(c1.X, k, axis=2)
    ck.xi = np.repeat(c1.xi, k, axis=1)
    ck.zeta = c1.zeta.copy()
    ck.kappa, ck.gS = c1.kappa, c1.gS
    c1.zeta = (c1.zeta / 2.0).astype(np.float32)   # sqrt(4) = 2, exact
    g1, gk = run_gpu(c1, gpu_device), run_gpu(ck, gpu_device)
    compare(c1, g1)
    compare(ck, gk)
    near = np.abs(g1["H"] - 1.0) < 1e-5
    assert np.all((g1["S"] == gk["S"]) | near)


# --- the paper's channel-major layer layout [T, batch, C, P, S] ---
CM_SHAPES = [
    # T, batch, C, S, B, k, io, K
    (4, 2, 3, 300, 4, 1, "f32", 4),      # spatial tiles (S >= 256), P = 4
    (5, 2, 7, 33, 8, 1, "f32", 2),       # whole channels per tile, P = 8
    (4, 3, 4, 257, 2, 2, "f32", 4),      # the paper's P = 4 on B = 2
    (6, 2, 5, 20, 1, 4, "bf16", 3),
    (4, 2, 3, 513, 4, 1, "bf16", 4),
    (7, 2, 6, 5, 3, 2, "f32", 7),        # P = 6
    (3, 2, 4, 64, 5, 1, "bf16", 3),
    (9, 1, 2, 300, 2, 4, "f32", 4),      # P = 8, checkpoints
    (4, 2, 3, 260, 16, 1, "f32", 4),     # 4 lanes per neuron
    (5, 2, 4, 70, 6, 1, "bf16", 5),      # 2 lanes of 3 branches
    (4, 2, 3, 300, 8, 2, "f32", 2),      # P = 16 over 4 lanes
    (6, 2, 5, 31, 4, 4, "bf16", 4),      # P = 16, k = 4, 4 lanes
    (4, 2, 2, 400, 7, 1, "f32", 4),      # odd branch count, one lane
    (4, 3, 3, 512, 2, 2, "f32", 4),      # two positions per lane in the backward
    (4, 2, 2, 1024, 4, 1, "f32", 4),
]


@pytest.mark.parametrize("shape", CM_SHAPES, ids=lambda s: "T{}b{}C{}S{}B{}k{}{}K{}".format(*s))
@pytest.mark.parametrize("variant", ["mh-sig-mask", "id-atan-stateless-res-plif"])
def test_channel_major_layout(gpu_device, shape, variant):
    T, batch, C, S, B, k, io, K = shape
    c = cfg(T=T, batch=batch, C=C, S=S, B=B, comps_per_branch=k, io=io, ckpt_every=K, layout="channel_major",
            psi="identity" if "-id-" in f"-{variant}-" else "mexhat", sg="sigmoid" if "sig" in variant else "atan",
            stateful="stateless" not in variant, residual="res" in variant, beta=0.7)
    seed = zlib.crc32(repr((shape, variant, "cm")).encode()) % 1000
    case = make_case(c, seed=seed, x_std=1.2, alpha=0.6, mask_rho=0.5 if "mask" in variant else None,
                     name=f"cm/{shape}/{variant}", beta_dev=0.8 if "plif" in variant else None)
    compare(case, run_gpu(case, gpu_device))


@pytest.mark.parametrize("B,k,io", [(4, 1, "f32"), (8, 1, "f32"), (2, 2, "f32"), (4, 1, "bf16"), (16, 1, "f32"),
                                    (8, 2, "bf16")])
def test_channel_major_equals_compartments_innermost(gpu_device, B, k, io):
    """Same neurons, same per-lane arithmetic order: the two layouts give
    bit-identical spikes, potentials and input gradients (after the permutation)."""
    import torch

    base = cfg(T=5, batch=2, C=6, S=300, B=B, comps_per_branch=k, io=io, ckpt_every=3)
    case = make_case(base, seed=33, mask_rho=0.6, name=f"cm-vs-npb/B{B}k{k}{io}")
    a = run_gpu(case, gpu_device)
    case.cfg = base.with_(layout="channel_major")
    b = run_gpu(case, gpu_device)
    assert torch.equal(a["raw"]["spikes"], b["raw"]["spikes"])
    assert torch.equal(a["raw"]["v_soma"], b["raw"]["v_soma"])
    assert np.array_equal(a["gX"], b["gX"])
    compare(case, b)


# --- residual dendrite (ResStateful / ResStateless) and the PLIF soma ---
@pytest.mark.parametrize("stateful", [True, False])
@pytest.mark.parametrize("plif", [False, True])
@pytest.mark.parametrize("detach", [False, True])
def test_tiny_residual_and_plif(gpu_device, stateful, plif, detach):
    c = cfg(stateful=stateful, residual=True, detach_reset=detach)
    case = make_case(c, seed=3, with_gv=True, name=f"tiny/res/stateful={stateful}/plif={plif}/detach={detach}",
                     beta_dev=0.65 if plif else None)
    rep = compare(case, run_gpu(case, gpu_device))
    print(rep)


def test_device_beta_overrides_cfg_beta(gpu_device):
    """A device beta is the decay the scan uses: bit-identical to the same value in cfg."""
    import torch

    base = cfg(T=9, batch=3, C=40, S=17, B=8, ckpt_every=4)
    case = make_case(base.with_(beta=0.1), seed=21, mask_rho=0.6, name="device-beta", beta_dev=0.85)
    d = to_device(case, gpu_device)
    a = run_gpu(case, gpu_device, dev=d)
    compare(case, a)
    case.cfg, case.beta_dev = base.with_(beta=0.85), None
    d["beta"] = None
    b = run_gpu(case, gpu_device, dev=d)
    assert torch.equal(a["raw"]["spikes"], b["raw"]["spikes"])
    for k in a["raw"]["grads"]:
        assert torch.equal(_bits(a["raw"]["grads"][k]), _bits(b["raw"]["grads"][k])), k


def test_dbg_per_task_dense_strengths(gpu_device):
    """DBG_e: each task keeps its own dense branch strengths kappa_q next to its
    mask m_q; a call for task q passes kappa_q and m_q."""
    c = cfg(T=4, batch=3, C=96, S=1, B=16, residual=False)
    for q in range(3):
        case = make_case(c, seed=40 + q, mask_rho=0.5, name=f"dbg-e/task{q}")
        compare(case, run_gpu(case, gpu_device))


# --- the benchmark layer shapes with the batch cut down (every other size kept) ---
REDUCED = {
    "cifar": dict(T=4, batch=2, C=128, S=1024, B=8, x_std=0.5),
    "imagenet_stem": dict(T=4, batch=1, C=64, S=12544, B=4, io="bf16"),
    "long_horizon": dict(T=64, batch=2, C=4096, S=1, B=16, x_mean=0.1, alpha=0.8, beta=0.9, ckpt_every=8),
    "dbg": dict(T=4, batch=2, C=8192, S=1, B=32, mask_rho=0.5),
    "long_horizon_res_plif": dict(T=64, batch=2, C=4096, S=1, B=16, x_mean=0.1, alpha=0.8, beta=0.9,
                                  ckpt_every=8, residual=True, beta_dev=0.9),
    "cifar_res": dict(T=4, batch=2, C=128, S=1024, B=8, x_std=0.5, residual=True),
    "cifar_p4b2": dict(T=4, batch=2, C=128, S=1024, B=2, comps_per_branch=2, x_std=0.5),
    "tiny_imagenet_res": dict(T=4, batch=1, C=64, S=4096, B=2, comps_per_branch=2, psi="identity",
                              stateful=False, residual=True),
    "dvs_p10b5": dict(T=10, batch=1, C=128, S=1024, B=5, comps_per_branch=2, stateful=False, ckpt_every=4),
}


@pytest.mark.parametrize("name", list(REDUCED))
def test_reduced_workloads(gpu_device, name):
    kw = dict(REDUCED[name])
    x_mean, x_std = kw.pop("x_mean", 0.0), kw.pop("x_std", 1.0)
    alpha, rho = kw.pop("alpha", 0.5), kw.pop("mask_rho", None)
    beta_dev = kw.pop("beta_dev", None)
    c = cfg(**kw)
    case = make_case(c, seed=7, x_mean=x_mean, x_std=x_std, alpha=alpha, random_affine=False,
                     mask_rho=rho, name=f"reduced/{name}", beta_dev=beta_dev)
    rep = compare(case, run_gpu(case, gpu_device))
    print(name, rep)


# --- invariants that must hold bit for bit on the GPU ---
def _bits(t):
    import torch

    return t.contiguous().view(torch.uint8)


def test_checkpoint_interval_is_bit_invariant(gpu_device):
    import torch

    base = cfg(T=64, batch=2, C=512, S=1, B=16, beta=0.9, ckpt_every=8)
    case = make_case(base, seed=11, x_mean=0.1, alpha=0.8, random_affine=True, mask_rho=0.7, name="ckpt8")
    d = to_device(case, gpu_device)
    outs = []
    for K in (8, 64, 5, 1):
        case.cfg = base.with_(ckpt_every=K)
        announce(f"ckpt interval K={K}")
        g = run_gpu(case, gpu_device, dev=d)["raw"]
        outs.append(g)
    ref = outs[0]
    for o in outs[1:]:
        assert torch.equal(o["spikes"], ref["spikes"])
        assert torch.equal(o["v_soma"], ref["v_soma"])
        assert torch.equal(_bits(o["grads"]["grad_x"]), _bits(ref["grads"]["grad_x"]))


@pytest.mark.parametrize("shape", ["generic-kc2-S40", "fast-kc1-fc", "bf16-kc2-S300"])
def test_stateless_checkpoint_interval_is_bit_invariant(gpu_device, shape):
    """The Stateless Dendrite checkpoints only the somatic potential; its backward
    restarts every segment from the input itself.  Every interval gives the
    same bits (and matches the oracle)."""
    import torch

    kw = {"generic-kc2-S40": dict(T=10, batch=2, C=24, S=40, B=5, comps_per_branch=2),
          "fast-kc1-fc": dict(T=13, batch=3, C=70, S=1, B=8),
          "bf16-kc2-S300": dict(T=9, batch=2, C=8, S=300, B=4, comps_per_branch=2, io="bf16")}[shape]
    base = cfg(stateful=False, beta=0.9, ckpt_every=4, **kw)
    case = make_case(base, seed=19, x_mean=0.1, mask_rho=0.7, with_gv=True, name=f"stateless-ckpt/{shape}")
    d = to_device(case, gpu_device)
    outs = []
    for K in (4, base.T, 3, 1):
        case.cfg = base.with_(ckpt_every=K)
        announce(f"stateless ckpt interval K={K}")
        outs.append(run_gpu(case, gpu_device, dev=d)["raw"])
    for o in outs[1:]:
        assert torch.equal(o["spikes"], outs[0]["spikes"])
        assert torch.equal(o["v_soma"], outs[0]["v_soma"])
        for k in o["grads"]:
            assert torch.equal(_bits(o["grads"][k]), _bits(outs[0]["grads"][k])), k
    compare(case, run_gpu(case, gpu_device, dev=d))


@pytest.mark.parametrize("shape", ["generic-kc2", "fast-kc1", "fast-kc2-bf16", "channel-major"])
def test_stateless_equals_stateful_with_zero_alpha(gpu_device, shape):
    """Methods, "DendSN variants": the Stateless Dendrite is the leaky one with
    alpha = 0.  The stateless kernels (which drop the leak altogether) and the
    stateful ones at alpha = 0 give equal spikes, potentials and gradients; only
    g_alpha differs (the stateless layer has no alpha)."""
    import torch

    kw = {"generic-kc2": dict(T=10, batch=2, C=24, S=40, B=5, comps_per_branch=2, ckpt_every=4),
          "fast-kc1": dict(T=4, batch=2, C=16, S=512, B=8),
          "fast-kc2-bf16": dict(T=6, batch=2, C=8, S=300, B=4, comps_per_branch=2, io="bf16", ckpt_every=3),
          "channel-major": dict(T=4, batch=2, C=16, S=100, B=2, comps_per_branch=2, layout="channel_major")}[shape]
    base = cfg(stateful=False, beta=0.8, **kw)
    case = make_case(base, seed=29, alpha=0.0, mask_rho=0.6, name=f"stateless-vs-alpha0/{shape}")
    d = to_device(case, gpu_device)
    a = run_gpu(case, gpu_device, dev=d)
    case.cfg = base.with_(stateful=True)
    b = run_gpu(case, gpu_device, dev=d)
    assert torch.equal(a["raw"]["spikes"], b["raw"]["spikes"])
    assert torch.equal(a["raw"]["v_soma"], b["raw"]["v_soma"])
    for k in ("grad_x", "grad_kappa", "grad_xi", "grad_zeta", "grad_beta"):
        assert torch.equal(a["raw"]["grads"][k], b["raw"]["grads"][k]), k
    assert a["g_alpha"] == 0.0


@pytest.mark.parametrize("B,io", [(8, "bf16"), (16, "bf16"), (64, "bf16"), (16, "f32")])
def test_recompute_from_checkpoints_is_bit_exact(gpu_device, B, io):
    """The backward recomputes the forward from state checkpoints; it must reproduce
    the forward's states bit for bit even where it splits a neuron over lanes
    differently (bf16), so every checkpoint interval gives the same bits."""
    import torch

    base = cfg(T=24, batch=2, C=40, S=1, B=B, io=io, beta=0.9, ckpt_every=6)
    case = make_case(base, seed=18, x_mean=0.1, alpha=0.8, mask_rho=0.7, name=f"ckpt-bits/B{B}{io}")
    d = to_device(case, gpu_device)
    outs = []
    for K in (6, 24, 1):
        case.cfg = base.with_(ckpt_every=K)
        outs.append(run_gpu(case, gpu_device, dev=d)["raw"])
    for o in outs[1:]:
        assert torch.equal(o["spikes"], outs[0]["spikes"])
        assert torch.equal(_bits(o["grads"]["grad_x"]), _bits(outs[0]["grads"]["grad_x"]))
    compare(case, run_gpu(case, gpu_device, dev=d))


def test_run_to_run_determinism(gpu_device):
    import torch

    case = make_case(cfg(T=6, batch=5, C=64, S=300, B=8), seed=12, mask_rho=0.5, name="determinism")
    d = to_device(case, gpu_device)
    a = run_gpu(case, gpu_device, dev=d)["raw"]
    b = run_gpu(case, gpu_device, dev=d)["raw"]
    assert torch.equal(a["spikes"], b["spikes"])
    for k in a["grads"]:
        assert torch.equal(_bits(a["grads"][k]), _bits(b["grads"][k])), k


def test_mask_of_ones_equals_no_mask(gpu_device):
    import torch

    case = make_case(cfg(T=5, batch=3, C=96, S=1, B=32), seed=13, name="mask-ones")
    d = to_device(case, gpu_device)
    a = run_gpu(case, gpu_device, dev=d)["raw"]
    d["mask"] = torch.ones((96, 32), dtype=torch.uint8, device=gpu_device)
    case.mask = np.ones((96, 32), np.uint8)
    b = run_gpu(case, gpu_device, dev=d)["raw"]
    assert torch.equal(a["spikes"], b["spikes"])
    for k in a["grads"]:
        assert torch.equal(_bits(a["grads"][k]), _bits(b["grads"][k])), k


@pytest.mark.parametrize("io,S", [("f32", 3), ("bf16", 3), ("bf16", 512)])
def test_masked_branches_get_exact_positive_zero(gpu_device, io, S):
    case = make_case(cfg(T=4, batch=2, C=64, S=S, B=8, io=io), seed=14, mask_rho=0.5, name=f"mask-zero/{io}/S{S}")
    # gated-off branches receive inf / nan inputs: nothing may leak out of them
    cidx = (np.arange(case.cfg.N) // case.cfg.S) % case.cfg.C
    off = (case.mask == 0)[cidx]
    case.X[:, off] = np.where(np.random.default_rng(0).random(case.X[:, off].shape) < 0.5, np.inf, np.nan)
    g = run_gpu(case, gpu_device)
    assert not np.any(np.signbit(g["gX"][:, off])) and np.all(g["gX"][:, off] == 0)
    for k in ("g_kappa", "g_xi", "g_zeta"):
        assert np.all(g[k][case.mask == 0] == 0) and not np.any(np.signbit(g[k][case.mask == 0]))
    assert np.all(np.isfinite(g["gX"])) and np.isfinite(g["g_alpha"])
    case.X[:, off] = 0.0
    compare(case, g)


def test_lif_reduction(gpu_device):
    """B = 1, identity, kappa = 1, xi = 0, zeta = 1, alpha = 0, X >= 0: a LIF neuron."""
    c = cfg(T=32, batch=4, C=300, S=1, B=1, psi="identity", beta=0.9, stateful=False)
    case = make_case(c, seed=15, random_affine=False, name="lif")
    case.X = np.abs(case.X)
    case.kappa = np.ones_like(case.kappa)
    g = run_gpu(case, gpu_device)
    x = case.X[:, :, 0].astype(np.float64)
    v = np.zeros(c.N)
    s = np.zeros(c.N)
    for t in range(c.T):
        v = 0.9 * (1 - s) * v + x[t]
        s = (v >= 1.0).astype(np.float64)
        near = np.abs(v - 1.0) <= 1e-6
        assert np.all((g["S"][t] == s) | near)
        s = np.where(near, g["S"][t], s)
        assert np.allclose(g["H"][t], v, rtol=1e-6, atol=1e-7)


def test_batch_grouping_changes_nothing_but_rounding(gpu_device):
    import torch

    base = cfg(T=4, batch=8, C=32, S=512, B=8)
    case = make_case(base, seed=16, name="groups")
    d = to_device(case, gpu_device)
    case.cfg = base.with_(batch_groups=1)
    a = run_gpu(case, gpu_device, dev=d)
    case.cfg = base.with_(batch_groups=8)
    b = run_gpu(case, gpu_device, dev=d)
    assert torch.equal(a["raw"]["spikes"], b["raw"]["spikes"])
    assert torch.equal(_bits(a["raw"]["grads"]["grad_x"]), _bits(b["raw"]["grads"]["grad_x"]))
    compare(case, a)
    compare(case, b)


def test_forward_without_checkpoints_for_inference(gpu_device):
    import torch

    c = cfg(T=12, batch=2, C=64, S=1, B=8, ckpt_every=4)
    case = make_case(c, seed=17, name="inference")
    d = to_device(case, gpu_device)
    s1, v1, ck = dendsn.forward(c, d["x"], d["alpha"], d["kappa"], d["xi"], d["zeta"], None, want_v_soma=True)
    s2, v2, ck2 = dendsn.forward(c, d["x"], d["alpha"], d["kappa"], d["xi"], d["zeta"], None, want_v_soma=True,
                                 save_ckpt=False)
    torch.cuda.synchronize()
    assert ck is not None and ck2 is None
    assert torch.equal(s1, s2) and torch.equal(v1, v2)


# --- degenerate cases of the method ---
def _degenerate(name, io):
    """A seeded case in one of the method's degenerate regimes."""
    stateless = name.startswith("x-equals-xi")
    kc = 2 if name.endswith("kc2") else 1
    c = cfg(T=5, batch=2, C=16, S=300, B=4, io=io, comps_per_branch=kc, ckpt_every=2,
            stateful=not stateless, residual=name == "all-gated-res",
            psi="identity" if name.endswith("id-kc2") else "mexhat",
            beta=0.0 if name == "beta-zero" else 0.5,
            v_th=0.0 if name == "always-fire" else 1.0)
    # saturated: X ~ N(1000, 10) keeps u >= 500, where exp(-u^2/2) underflows to 0 in fp32 and
    # fp64 alike (a zero-mean spread of 1000 would instead test fp32 cancellation in Vd)
    sat = name == "saturated"
    case = make_case(c, seed=zlib.crc32(f"{name}/{io}".encode()) % 1000, x_mean=1000.0 if sat else 0.0,
                     x_std=10.0 if sat else 1.2,
                     alpha=0.6, random_affine=True, mask_rho=0.5, name=f"degenerate/{name}/{io}")
    if name.startswith("all-gated"):
        case.mask = np.zeros_like(case.mask)             # every branch of every channel gated off
    else:
        case.mask = None
    if name in ("kappa-zero", "always-fire"):
        case.kappa = np.zeros_like(case.kappa)            # Z = 0: H stays 0 (always at threshold when v_th = 0)
    if stateless:
        # Vd = X = xi exactly: every branch at the norm's origin (zero subgradient)
        cidx = (np.arange(c.N) // c.S) % c.C
        case.X = np.broadcast_to(case.xi[cidx][None], case.X.shape).copy()
        if io == "bf16":
            import torch

            case.xi = torch.from_numpy(case.xi).to(torch.bfloat16).float().numpy()
            case.X = np.broadcast_to(case.xi[cidx][None], case.X.shape).copy()
    return case


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("name", ["all-gated", "all-gated-res", "kappa-zero", "always-fire", "beta-zero",
                                  "x-equals-xi", "x-equals-xi-id-kc2", "saturated"])
def test_degenerate_cases(gpu_device, name, io):
    case = _degenerate(name, io)
    gpu = run_gpu(case, gpu_device)
    rep = compare(case, gpu)
    if name in ("kappa-zero", "always-fire") or name == "all-gated":
        assert np.all(gpu["gX"] == 0.0)                   # nothing reaches X's gradient but through Z
    if name == "always-fire":
        assert np.all(gpu["S"] == 1.0)                    # H = 0 = v_th fires (Theta(0) = 1) at every step
    if name.startswith("x-equals-xi"):
        assert np.all(gpu["gX"] == 0.0)                   # the norm's subgradient at 0 is 0
    if name == "saturated":                               # psi = psi' = 0 on every branch: a silent layer
        assert np.all(gpu["S"] == 0.0) and np.all(gpu["H"] == 0.0) and np.all(gpu["gX"] == 0.0)
    print(name, io, rep)
