"""ctypes binding of libdendsn.so (include/dendsn.h).

Argument marshalling only: torch tensors supply device memory and the current
HIP stream; every step of the scan runs in the library's HIP kernels.  The
functions named like the C entry points take the same arguments as the C ABI
(tensors in place of pointers); ``forward`` / ``backward`` are conveniences
that allocate the outputs.  There is no fallback: if the library is not built
or fails to load, every call raises.
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
from dataclasses import dataclass

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdendsn.so")

IO = {"f32": 0, "bf16": 1}
PSI = {"identity": 0, "mexhat": 1}
SG = {"atan": 0, "sigmoid": 1}
LAYOUT = {"npb": 0, "channel_major": 1}

NOALLOC_SCRATCH_BYTES = 32 << 20   # DENDSN_NOALLOC_SCRATCH_BYTES of include/dendsn.h

STATUS = {0: "DENDSN_OK", 1: "DENDSN_E_INVALID", 2: "DENDSN_E_UNSUPPORTED",
          3: "DENDSN_E_WORKSPACE", 4: "DENDSN_E_HIP"}


class DendSNError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"{STATUS.get(status, status)}: {detail}")


class dendsn_cfg(ctypes.Structure):
    _fields_ = [
        ("T", ctypes.c_int64),
        ("batch", ctypes.c_int64),
        ("C", ctypes.c_int64),
        ("S", ctypes.c_int64),
        ("B", ctypes.c_int32),
        ("comps_per_branch", ctypes.c_int32),
        ("stateful", ctypes.c_int32),
        ("detach_reset", ctypes.c_int32),
        ("ckpt_every", ctypes.c_int32),
        ("io", ctypes.c_int32),
        ("psi", ctypes.c_int32),
        ("sg", ctypes.c_int32),
        ("sg_scale", ctypes.c_float),
        ("beta", ctypes.c_float),
        ("v_th", ctypes.c_float),
        ("batch_groups", ctypes.c_int32),
        ("residual", ctypes.c_int32),
        ("layout", ctypes.c_int32),
    ]


@dataclass(frozen=True)
class DendSNConfig:
    """One DendSN layer: N = batch * C * S neurons with B branches of
    comps_per_branch compartments each (P in all), T steps."""

    T: int
    batch: int
    C: int
    S: int
    B: int
    stateful: bool = True
    detach_reset: bool = False
    ckpt_every: int = 0          # 0: no interior checkpoint
    io: str = "f32"
    psi: str = "mexhat"
    sg: str = "sigmoid"
    sg_scale: float = 4.0
    beta: float = 0.5
    v_th: float = 1.0
    batch_groups: int = 0
    comps_per_branch: int = 1
    residual: bool = False
    layout: str = "npb"          # X / grad_x: "npb" [T, N, P] or "channel_major" [T, batch, C, P, S]

    @property
    def N(self) -> int:
        return self.batch * self.C * self.S

    @property
    def P(self) -> int:
        """Compartments per neuron: the innermost extent of X and grad_x."""
        return self.B * self.comps_per_branch

    def with_(self, **kw) -> "DendSNConfig":
        return dataclasses.replace(self, **kw)

    def to_c(self) -> dendsn_cfg:
        return dendsn_cfg(
            T=self.T, batch=self.batch, C=self.C, S=self.S, B=self.B,
            comps_per_branch=self.comps_per_branch, stateful=int(self.stateful),
            detach_reset=int(self.detach_reset),
            ckpt_every=self.ckpt_every if self.ckpt_every > 0 else max(1, min(self.T, 2**31 - 1)),
            io=IO[self.io], psi=PSI[self.psi], sg=SG[self.sg], sg_scale=self.sg_scale,
            beta=self.beta, v_th=self.v_th, batch_groups=self.batch_groups, residual=int(self.residual),
            layout=LAYOUT[self.layout],
        )


_lib = None

_SIGS = {
    "dendsn_ckpt_bytes": (ctypes.c_int, [ctypes.POINTER(dendsn_cfg), ctypes.POINTER(ctypes.c_size_t)]),
    "dendsn_bwd_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(dendsn_cfg), ctypes.POINTER(ctypes.c_size_t)]),
    "dendsn_forward": (ctypes.c_int, [ctypes.POINTER(dendsn_cfg)] + [ctypes.c_void_p] * 11),
    "dendsn_backward": (ctypes.c_int, [ctypes.POINTER(dendsn_cfg)] + [ctypes.c_void_p] * 17
                        + [ctypes.c_size_t, ctypes.c_void_p]),
    "dendsn_backward_noalloc": (ctypes.c_int, [ctypes.POINTER(dendsn_cfg)] + [ctypes.c_void_p] * 17),
    "dendsn_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "dendsn_last_error": (ctypes.c_char_p, []),
}

EXPORTS = tuple(_SIGS)


def lib():
    """Load libdendsn.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build the HIP library first "
                "(python -m paper_2412_06355_amd.build)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(status: int):
    if status != 0:
        raise DendSNError(status, lib().dendsn_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    import torch

    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


# ---------------------------------------------------------------------------
# Entry points with the C names
# ---------------------------------------------------------------------------
def dendsn_status_str(status: int) -> str:
    return lib().dendsn_status_str(status).decode()


def dendsn_last_error() -> str:
    return lib().dendsn_last_error().decode()


def dendsn_ckpt_bytes(cfg: DendSNConfig) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().dendsn_ckpt_bytes(ctypes.byref(cfg.to_c()), ctypes.byref(out)))
    return out.value


def dendsn_bwd_workspace_bytes(cfg: DendSNConfig) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().dendsn_bwd_workspace_bytes(ctypes.byref(cfg.to_c()), ctypes.byref(out)))
    return out.value


def dendsn_forward(cfg: DendSNConfig, x, alpha, beta, kappa, xi, zeta, mask, spikes, v_soma, ckpt,
                   stream=None):
    c = cfg.to_c()
    st = stream if stream is not None else _stream(x.device)
    _check(lib().dendsn_forward(ctypes.byref(c), _ptr(x), _ptr(alpha), _ptr(beta), _ptr(kappa), _ptr(xi),
                                _ptr(zeta), _ptr(mask), _ptr(spikes), _ptr(v_soma), _ptr(ckpt), st))


def dendsn_backward(cfg: DendSNConfig, x, alpha, beta, kappa, xi, zeta, mask, ckpt, grad_spikes, grad_v_soma,
                    grad_x, grad_alpha, grad_beta, grad_kappa, grad_xi, grad_zeta, workspace, stream=None):
    c = cfg.to_c()
    st = stream if stream is not None else _stream(x.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().dendsn_backward(ctypes.byref(c), _ptr(x), _ptr(alpha), _ptr(beta), _ptr(kappa), _ptr(xi),
                                 _ptr(zeta), _ptr(mask), _ptr(ckpt), _ptr(grad_spikes), _ptr(grad_v_soma),
                                 _ptr(grad_x), _ptr(grad_alpha), _ptr(grad_beta), _ptr(grad_kappa),
                                 _ptr(grad_xi), _ptr(grad_zeta), _ptr(workspace), ctypes.c_size_t(ws_bytes),
                                 st))


def dendsn_backward_noalloc(cfg: DendSNConfig, x, alpha, beta, kappa, xi, zeta, mask, ckpt, grad_spikes,
                            grad_v_soma, grad_x, grad_alpha, grad_beta, grad_kappa, grad_xi, grad_zeta,
                            stream=None):
    c = cfg.to_c()
    st = stream if stream is not None else _stream(x.device)
    _check(lib().dendsn_backward_noalloc(ctypes.byref(c), _ptr(x), _ptr(alpha), _ptr(beta), _ptr(kappa),
                                         _ptr(xi), _ptr(zeta), _ptr(mask), _ptr(ckpt), _ptr(grad_spikes),
                                         _ptr(grad_v_soma), _ptr(grad_x), _ptr(grad_alpha), _ptr(grad_beta),
                                         _ptr(grad_kappa), _ptr(grad_xi), _ptr(grad_zeta), st))


# ---------------------------------------------------------------------------
# Conveniences that allocate outputs and check tensor shapes / dtypes
# ---------------------------------------------------------------------------
def _io_dtype(cfg):
    import torch

    return {"f32": torch.float32, "bf16": torch.bfloat16}[cfg.io]


def _expect(t, name, shape, dtype, device, optional=False):
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != {tuple(shape)}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype} != {dtype}")
    if t.device != device:
        raise ValueError(f"{name}: on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _x_shape(cfg, x):
    """[T, N, P]; in the channel-major layout any contiguous shape that starts
    with T and holds T N P elements in [T, batch, C, P, S] order (for example
    the producing conv layer's [T, batch, C P, H, W])."""
    if cfg.layout == "channel_major":
        n = cfg.N * cfg.P
        return tuple(x.shape) if (x.dim() >= 2 and x.shape[0] == cfg.T and x.numel() == cfg.T * n) \
            else (cfg.T, cfg.batch, cfg.C, cfg.P, cfg.S)
    return (cfg.T, cfg.N, cfg.P)


def _check_params(cfg, x, alpha, kappa, xi, zeta, mask, beta=None):
    import torch

    dev = x.device
    _expect(x, "x", _x_shape(cfg, x), _io_dtype(cfg), dev)
    _expect(alpha, "alpha", (1,), torch.float32, dev, optional=not cfg.stateful)
    _expect(beta, "beta", (1,), torch.float32, dev, optional=True)
    _expect(kappa, "kappa", (cfg.C, cfg.B), torch.float32, dev)
    _expect(xi, "xi", (cfg.C, cfg.P), torch.float32, dev, optional=True)
    _expect(zeta, "zeta", (cfg.C, cfg.B), torch.float32, dev, optional=True)
    _expect(mask, "mask", (cfg.C, cfg.B), torch.uint8, dev, optional=True)


def _check_ckpt(cfg, ckpt, device):
    """The checkpoint buffer the backward reads: when this cfg has interior
    checkpoints, a contiguous float32 tensor on the layer's device holding at
    least dendsn_ckpt_bytes(cfg) bytes (a buffer written for another cfg would
    be read past its end)."""
    import torch

    need = dendsn_ckpt_bytes(cfg)
    if need == 0:
        return
    if ckpt is None:
        raise ValueError(f"ckpt is required: this layer has interior checkpoints ({need} bytes)")
    if ckpt.dtype != torch.float32 or ckpt.device != device or not ckpt.is_contiguous():
        raise ValueError(f"ckpt must be a contiguous float32 tensor on {device}")
    if ckpt.numel() * 4 < need:
        raise ValueError(f"ckpt holds {ckpt.numel() * 4} bytes, this layer needs {need}")


def forward(cfg: DendSNConfig, x, alpha, kappa, xi=None, zeta=None, mask=None, *, beta=None,
            want_v_soma: bool = False, save_ckpt: bool = True):
    """Returns (spikes [T,N] io, v_soma [T,N] fp32 or None, ckpt buffer or None).
    ``beta``: optional learnable somatic decay [1] on the device (else cfg.beta)."""
    import torch

    _check_params(cfg, x, alpha, kappa, xi, zeta, mask, beta)
    dev = x.device
    spikes = torch.empty((cfg.T, cfg.N), dtype=_io_dtype(cfg), device=dev)
    v_soma = torch.empty((cfg.T, cfg.N), dtype=torch.float32, device=dev) if want_v_soma else None
    nb = dendsn_ckpt_bytes(cfg)
    ckpt = torch.empty((nb // 4,), dtype=torch.float32, device=dev) if (save_ckpt and nb) else None
    dendsn_forward(cfg, x, alpha, beta, kappa, xi, zeta, mask, spikes, v_soma, ckpt)
    return spikes, v_soma, ckpt


def backward(cfg: DendSNConfig, x, alpha, kappa, xi, zeta, mask, ckpt, grad_spikes, grad_v_soma=None,
             workspace=None, *, beta=None):
    """Returns a dict with grad_x (x's shape and layout) and grad_alpha [1], grad_beta [1],
    grad_kappa, grad_zeta [C,B] and grad_xi [C,P] (fp32)."""
    import torch

    _check_params(cfg, x, alpha, kappa, xi, zeta, mask, beta)
    dev = x.device
    _expect(grad_spikes, "grad_spikes", (cfg.T, cfg.N), _io_dtype(cfg), dev)
    _expect(grad_v_soma, "grad_v_soma", (cfg.T, cfg.N), torch.float32, dev, optional=True)
    _check_ckpt(cfg, ckpt, dev)
    out = dict(
        grad_x=torch.empty(x.shape, dtype=_io_dtype(cfg), device=dev),
        grad_alpha=torch.empty((1,), dtype=torch.float32, device=dev),
        grad_beta=torch.empty((1,), dtype=torch.float32, device=dev),
        grad_kappa=torch.empty((cfg.C, cfg.B), dtype=torch.float32, device=dev),
        grad_xi=torch.empty((cfg.C, cfg.P), dtype=torch.float32, device=dev),
        grad_zeta=torch.empty((cfg.C, cfg.B), dtype=torch.float32, device=dev),
    )
    if workspace is None:
        nb = dendsn_bwd_workspace_bytes(cfg)
        workspace = torch.empty(((nb + 3) // 4,), dtype=torch.float32, device=dev)
    dendsn_backward(cfg, x, alpha, beta, kappa, xi, zeta, mask, ckpt, grad_spikes, grad_v_soma,
                    out["grad_x"], out["grad_alpha"], out["grad_beta"], out["grad_kappa"], out["grad_xi"],
                    out["grad_zeta"], workspace)
    return out
