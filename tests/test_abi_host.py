"""Host-side checks of the C ABI: the library loads, exports every entry point
that include/dendsn.h declares, and rejects bad arguments before any launch.

Nothing here touches a GPU: every call either queries sizes or fails argument
validation, which the library performs on the host before any HIP call.
Pointers passed here are fake integers that the library never dereferences.
"""

import ctypes
import os
import re

import pytest

import paper_2412_06355_amd as dendsn
from paper_2412_06355_amd.binding import dendsn_cfg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dendsn.h")

OK, E_INVALID, E_UNSUPPORTED, E_WORKSPACE = 0, 1, 2, 3


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dendsn_[a-z_]+)\s*\(", text)))


def base_cfg(**kw):
    c = dict(T=4, batch=2, C=256, S=1, B=4, comps_per_branch=1, stateful=1, detach_reset=0,
             ckpt_every=4, io=0, psi=1, sg=1, sg_scale=4.0, beta=0.5, v_th=1.0, batch_groups=0, residual=0,
             layout=0)
    c.update(kw)
    return dendsn_cfg(**c)


L = None


@pytest.fixture(scope="module")
def lib():
    return dendsn.lib()


def fake(addr):
    return ctypes.c_void_p(addr)


GOOD = 0x10000  # 64 KiB-aligned fake device address


def fwd(lib, cfg, x=GOOD, alpha=GOOD + 0x100, kappa=GOOD + 0x200, xi=None, zeta=None, mask=None,
        spikes=GOOD + 0x300, v_soma=None, ckpt=None, beta=None):
    p = lambda v: None if v is None else fake(v)
    return lib.dendsn_forward(ctypes.byref(cfg), p(x), p(alpha), p(beta), p(kappa), p(xi), p(zeta), p(mask),
                              p(spikes), p(v_soma), p(ckpt), None)


def bwd(lib, cfg, ckpt=None, ws=GOOD + 0x1000, ws_bytes=1 << 40, x=GOOD, gx=GOOD + 0x400, gs=GOOD + 0x500,
        beta=None, grad_beta=None):
    p = lambda v: None if v is None else fake(v)
    return lib.dendsn_backward(ctypes.byref(cfg), p(x), p(GOOD + 0x100), p(beta), p(GOOD + 0x200), None, None,
                               None, p(ckpt), p(gs), None, p(gx), None, p(grad_beta), None, None, None, p(ws),
                               ctypes.c_size_t(ws_bytes), None)


def test_every_declared_function_is_exported(lib):
    declared = header_functions()
    assert set(declared) == set(dendsn.EXPORTS), declared
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code, name in [(0, "DENDSN_OK"), (1, "DENDSN_E_INVALID"), (2, "DENDSN_E_UNSUPPORTED"),
                       (3, "DENDSN_E_WORKSPACE"), (4, "DENDSN_E_HIP")]:
        assert dendsn.dendsn_status_str(code) == name


@pytest.mark.parametrize("T,K,batch,C,S,B,k", [(4, 4, 2, 256, 1, 4, 1), (64, 8, 32, 4096, 1, 16, 1),
                                               (10, 3, 3, 5, 7, 6, 1), (7, 100, 1, 1, 1, 1, 1),
                                               (9, 2, 2, 3, 5, 2, 2), (9, 4, 2, 3, 1, 5, 2), (6, 5, 1, 2, 3, 3, 4)])
def test_ckpt_bytes(lib, T, K, batch, C, S, B, k):
    cfg = dendsn.DendSNConfig(T=T, batch=batch, C=C, S=S, B=B, ckpt_every=K, comps_per_branch=k)
    nck = -(-T // K) - 1
    assert dendsn.dendsn_ckpt_bytes(cfg) == nck * batch * C * S * (B * k + 1) * 4
    # the Stateless Dendrite keeps only the somatic potential (its compartment
    # state is the step's input)
    assert dendsn.dendsn_ckpt_bytes(cfg.with_(stateful=False)) == nck * batch * C * S * 4


def test_workspace_bytes_positive_and_grows_with_groups(lib):
    cfg = dendsn.DendSNConfig(T=4, batch=128, C=128, S=1024, B=8)
    a = dendsn.dendsn_bwd_workspace_bytes(cfg.with_(batch_groups=1))
    b = dendsn.dendsn_bwd_workspace_bytes(cfg.with_(batch_groups=4))
    assert 0 < a < b


@pytest.mark.parametrize("kw,code", [
    (dict(T=-1), E_INVALID), (dict(batch=-1), E_INVALID), (dict(C=-1), E_INVALID), (dict(S=-1), E_INVALID),
    (dict(T=1 << 31), E_INVALID), (dict(C=1 << 50, S=0), E_INVALID), (dict(B=0, T=0), E_INVALID),
    (dict(B=0), E_INVALID), (dict(B=129), E_INVALID), (dict(comps_per_branch=0), E_INVALID),
    (dict(comps_per_branch=3), E_UNSUPPORTED), (dict(comps_per_branch=8), E_UNSUPPORTED),
    (dict(B=12, comps_per_branch=2), E_UNSUPPORTED), (dict(B=5, comps_per_branch=4), E_UNSUPPORTED),
    (dict(B=9), E_UNSUPPORTED), (dict(B=11), E_UNSUPPORTED),
    (dict(stateful=2), E_INVALID), (dict(detach_reset=-1), E_INVALID), (dict(ckpt_every=0), E_INVALID),
    (dict(io=2), E_INVALID), (dict(psi=5), E_INVALID), (dict(sg=3), E_INVALID),
    (dict(sg_scale=0.0), E_INVALID), (dict(sg_scale=float("nan")), E_INVALID),
    (dict(beta=float("inf")), E_INVALID), (dict(v_th=float("nan")), E_INVALID),
    (dict(batch_groups=-1), E_INVALID), (dict(batch=1 << 40, C=1 << 10), E_INVALID),
    (dict(residual=2), E_INVALID), (dict(residual=-1), E_INVALID),
    (dict(layout=2), E_INVALID), (dict(layout=-1), E_INVALID),
    (dict(layout=1, S=4, B=64), E_UNSUPPORTED), (dict(layout=1, S=4, B=16, comps_per_branch=2), E_UNSUPPORTED),
    (dict(layout=1, S=4, B=3, comps_per_branch=4), E_UNSUPPORTED), (dict(layout=1, S=4, B=9), E_UNSUPPORTED),
])
def test_bad_cfg_rejected_everywhere(lib, kw, code):
    cfg = base_cfg(**kw)
    out = ctypes.c_size_t(12345)
    assert lib.dendsn_ckpt_bytes(ctypes.byref(cfg), ctypes.byref(out)) == code
    assert out.value == 12345  # nothing written on failure
    assert lib.dendsn_bwd_workspace_bytes(ctypes.byref(cfg), ctypes.byref(out)) == code
    assert fwd(lib, cfg) == code
    assert dendsn.dendsn_last_error() != ""
    assert bwd(lib, cfg) == code


def test_null_cfg(lib):
    out = ctypes.c_size_t(0)
    assert lib.dendsn_ckpt_bytes(None, ctypes.byref(out)) == E_INVALID
    assert lib.dendsn_forward(None, *([None] * 11)) == E_INVALID
    assert lib.dendsn_backward(None, *([None] * 17), ctypes.c_size_t(0), None) == E_INVALID


def test_sigmoid_scale_ignored_for_atan(lib):
    out = ctypes.c_size_t(0)
    cfg = base_cfg(sg=0, sg_scale=0.0)
    assert lib.dendsn_ckpt_bytes(ctypes.byref(cfg), ctypes.byref(out)) == OK


def test_forward_argument_checks(lib):
    cfg = base_cfg()
    assert fwd(lib, cfg, x=None) == E_INVALID
    assert fwd(lib, cfg, kappa=None) == E_INVALID
    assert fwd(lib, cfg, spikes=None) == E_INVALID
    assert fwd(lib, cfg, alpha=None) == E_INVALID          # stateful needs alpha
    assert fwd(lib, cfg, x=GOOD + 4) == E_INVALID           # x must be 16-byte aligned
    assert fwd(lib, cfg, spikes=GOOD + 2) == E_INVALID      # fp32 spikes misaligned
    assert fwd(lib, cfg, beta=GOOD + 2) == E_INVALID        # device beta misaligned
    assert bwd(lib, cfg, beta=GOOD + 2) == E_INVALID
    assert bwd(lib, cfg, grad_beta=GOOD + 0x702) == E_INVALID
    assert fwd(lib, cfg, ckpt=GOOD + 8) == E_INVALID
    assert "align" in dendsn.dendsn_last_error()


@pytest.mark.parametrize("kw", [dict(T=0), dict(batch=0), dict(C=0), dict(S=0), dict(T=0, batch=0, C=0, S=0),
                                dict(T=0, ckpt_every=1), dict(batch=0, T=64, ckpt_every=8, B=16),
                                dict(S=0, C=8, B=8, layout=1), dict(C=0, io=1, B=8, comps_per_branch=2)])
def test_empty_layers_are_valid(lib, kw):
    """An empty layer (no neuron-step) is a valid call: no checkpoint bytes, a
    positive workspace, and a forward that accepts NULL for its arrays of no
    elements and launches nothing (so it returns OK without a GPU)."""
    cfg = base_cfg(**kw)
    out = ctypes.c_size_t(12345)
    assert lib.dendsn_ckpt_bytes(ctypes.byref(cfg), ctypes.byref(out)) == OK
    assert out.value == 0
    assert lib.dendsn_bwd_workspace_bytes(ctypes.byref(cfg), ctypes.byref(out)) == OK
    assert out.value > 0
    kappa = None if cfg.C == 0 else GOOD + 0x200
    assert fwd(lib, cfg, x=None, spikes=None, kappa=kappa) == OK
    assert fwd(lib, cfg, x=None, spikes=None, kappa=kappa, alpha=None) == E_INVALID  # stateful needs alpha
    assert fwd(lib, cfg, x=GOOD + 4, spikes=None, kappa=kappa) == E_INVALID            # alignment still checked
    if cfg.C > 0:
        assert fwd(lib, cfg, x=None, spikes=None, kappa=None) == E_INVALID
    # the backward's host checks run as for any layer (its launch needs a GPU)
    assert bwd(lib, cfg, x=None, gx=None, gs=None, ws=None) == E_WORKSPACE
    assert bwd(lib, cfg, x=None, gx=None, gs=None, ws_bytes=16) == E_WORKSPACE


def test_backward_argument_checks(lib):
    cfg = base_cfg(T=8, ckpt_every=4)                         # one interior checkpoint
    assert bwd(lib, cfg, ckpt=None) == E_INVALID
    assert "ckpt" in dendsn.dendsn_last_error()
    assert bwd(lib, cfg, ckpt=GOOD + 0x800, ws=None) == E_WORKSPACE
    assert bwd(lib, cfg, ckpt=GOOD + 0x800, ws_bytes=16) == E_WORKSPACE
    assert bwd(lib, cfg, ckpt=GOOD + 0x800, gx=None) == E_INVALID
    assert bwd(lib, cfg, ckpt=GOOD + 0x800, gs=None) == E_INVALID
    assert bwd(lib, cfg, ckpt=GOOD + 0x800, gx=GOOD + 0x404) == E_INVALID


def test_supported_branch_counts(lib):
    out = ctypes.c_size_t(0)
    for io in (0, 1):
        ok = []
        for B in range(1, 129):
            st = lib.dendsn_ckpt_bytes(ctypes.byref(base_cfg(B=B, io=io)), ctypes.byref(out))
            assert st in (OK, E_UNSUPPORTED)
            if st == OK:
                ok.append(B)
        # every count up to 8, the even ones up to 16, and the powers of two up to 64
        for B in list(range(1, 9)) + [10, 12, 14, 16, 32, 64]:
            assert B in ok, (io, B)


def test_python_binding_raises_on_error():
    cfg = dendsn.DendSNConfig(T=4, batch=2, C=4, S=1, B=4, comps_per_branch=3)
    with pytest.raises(dendsn.DendSNError) as e:
        dendsn.dendsn_ckpt_bytes(cfg)
    assert e.value.status == E_UNSUPPORTED


@pytest.mark.parametrize("io", [0, 1])
@pytest.mark.parametrize("B,k", [(1, 2), (2, 2), (3, 2), (4, 2), (5, 2), (6, 2), (7, 2), (8, 2), (16, 2), (32, 2),
                                 (1, 4), (2, 4), (3, 4), (4, 4), (8, 4), (16, 4)])
def test_supported_compartment_layouts(lib, io, B, k):
    """The host checks accept these branch counts with k compartments per branch
    (the GPU parity tests launch each of their kernels)."""
    cfg = base_cfg(B=B, comps_per_branch=k, io=io)
    out = ctypes.c_size_t(0)
    assert lib.dendsn_bwd_workspace_bytes(ctypes.byref(cfg), ctypes.byref(out)) == OK
    assert out.value > 0


def test_channel_major_layout_limits(lib):
    """Channel-major X with S > 1 supports the compiled lane splits (up to 16
    branches / 16 compartments); with S = 1 it is the [T, N, P] memory and every
    mapping applies."""
    out = ctypes.c_size_t(0)
    for B, k in [(1, 1), (5, 1), (6, 1), (7, 1), (8, 1), (16, 1), (4, 1), (4, 2), (8, 2),
                 (3, 2), (2, 4), (4, 4)]:
        assert lib.dendsn_ckpt_bytes(ctypes.byref(base_cfg(layout=1, S=9, B=B, comps_per_branch=k)),
                                     ctypes.byref(out)) == OK
    assert lib.dendsn_ckpt_bytes(ctypes.byref(base_cfg(layout=1, S=1, B=64)), ctypes.byref(out)) == OK


def test_binding_fails_loudly_without_the_library(monkeypatch, tmp_path):
    """No fallback: with the shared library absent every call raises."""
    from paper_2412_06355_amd import binding

    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "libdendsn.so"))
    with pytest.raises(RuntimeError, match="missing"):
        binding.dendsn_ckpt_bytes(dendsn.DendSNConfig(T=4, batch=2, C=4, S=1, B=4))


def test_product_code_never_touches_the_oracle():
    """The oracle is test infrastructure: the package and the C sources do not
    import, link or name it."""
    pkg = os.path.join(ROOT, "paper_2412_06355_amd")
    for base, _, files in os.walk(pkg):
        if "_build" in base:
            continue
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(base, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "dendsn_oracle" not in text, f


def test_sample_slice_limit(lib):
    # Lane offsets inside one sample's [C, S, P] slice are 32-bit byte offsets:
    # 255 channels of 2^20 positions x 4 fp32 branches (4,278,190,080 bytes) are
    # the largest slice tests run on the GPU; one more channel (exactly 4 GiB) is
    # refused before any launch, in both directions.
    cfg = base_cfg(T=2, batch=2, C=256, S=1 << 20, B=4, ckpt_every=1)
    assert fwd(lib, cfg, ckpt=GOOD + 0x800) == E_UNSUPPORTED
    assert "4 GiB" in dendsn.dendsn_last_error()
    assert bwd(lib, cfg, ckpt=GOOD + 0x800) == E_UNSUPPORTED
    out = ctypes.c_size_t(0)
    ok = base_cfg(T=2, batch=2, C=255, S=1 << 20, B=4, ckpt_every=1)
    assert lib.dendsn_ckpt_bytes(ctypes.byref(ok), ctypes.byref(out)) == 0
    assert out.value == 2 * 255 * (1 << 20) * 5 * 4   # one checkpoint: N (P + 1) floats, N = 2 C S


def test_python_backward_checks_the_checkpoint_buffer():
    """backward() refuses a checkpoint buffer that is missing, of another dtype or
    smaller than this layer's dendsn_ckpt_bytes, before anything is launched (the
    C ABI cannot see a buffer's size).  Host tensors: validation only."""
    import torch

    cfg = dendsn.DendSNConfig(T=8, batch=2, C=16, S=1, B=4, ckpt_every=4)
    need = dendsn.dendsn_ckpt_bytes(cfg)
    assert need > 0
    x = torch.zeros((cfg.T, cfg.N, cfg.P))
    alpha, kappa = torch.zeros(1), torch.zeros((cfg.C, cfg.B))
    gS = torch.zeros((cfg.T, cfg.N))
    call = lambda ck: dendsn.backward(cfg, x, alpha, kappa, None, None, None, ck, gS)
    with pytest.raises(ValueError, match="required"):
        call(None)
    with pytest.raises(ValueError, match="bytes"):
        call(torch.zeros(need // 4 - 1))                       # one float short
    with pytest.raises(ValueError, match="float32"):
        call(torch.zeros(need // 8, dtype=torch.float64))
    with pytest.raises(ValueError, match="float32"):
        call(torch.zeros(need // 2)[::2])                      # not contiguous
    # a longer-horizon cfg needs more checkpoint bytes than this one's buffer holds
    longer = cfg.with_(T=16)
    with pytest.raises(ValueError, match="bytes"):
        dendsn.backward(longer, torch.zeros((16, cfg.N, cfg.P)), alpha, kappa, None, None, None,
                        torch.zeros(need // 4), torch.zeros((16, cfg.N)))


def bwd_noalloc(lib, cfg, ckpt=None, x=GOOD, gx=GOOD + 0x400, gs=GOOD + 0x500):
    p = lambda v: None if v is None else fake(v)
    return lib.dendsn_backward_noalloc(ctypes.byref(cfg), p(x), p(GOOD + 0x100), None, p(GOOD + 0x200), None,
                                       None, None, p(ckpt), p(gs), None, p(gx), None, None, None, None, None,
                                       None)


def test_noalloc_backward_argument_checks(lib):
    """The allocation-free backward checks its arguments like dendsn_backward, and
    refuses a layer whose partials exceed its scratch array, all before any HIP
    call (no device is needed to reach these refusals)."""
    cfg = base_cfg(T=8, ckpt_every=4)
    assert bwd_noalloc(lib, cfg, ckpt=None) == E_INVALID
    assert bwd_noalloc(lib, cfg, ckpt=GOOD + 0x800, x=None) == E_INVALID
    assert bwd_noalloc(lib, cfg, ckpt=GOOD + 0x800, gx=GOOD + 0x404) == E_INVALID
    big = base_cfg(T=4, batch=128, C=65536, S=1, B=32)
    need = ctypes.c_size_t(0)
    assert lib.dendsn_bwd_workspace_bytes(ctypes.byref(big), ctypes.byref(need)) == OK
    assert need.value > dendsn.NOALLOC_SCRATCH_BYTES
    assert bwd_noalloc(lib, big) == E_WORKSPACE
    assert "scratch" in dendsn.dendsn_last_error()
    # the binding's size is the header's
    m = re.search(r"#define DENDSN_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == dendsn.NOALLOC_SCRATCH_BYTES
