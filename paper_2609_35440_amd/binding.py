"""Thin ctypes binding of ``libsolo_readout.so`` (declared in include/solo_readout.h).

Argument marshalling only: every step of the computation runs in the library's
HIP kernels.  PyTorch provides the device memory and the stream.  There is no
fallback: if the library is missing the call raises.
"""
from __future__ import annotations

import collections
import ctypes
import os
import re
from typing import Optional

__all__ = [
    "SoloError",
    "ReadoutResult",
    "load_library",
    "library_path",
    "abi_version",
    "status_string",
    "workspace_size",
    "kernel_family",
    "readout_fwd_bwd",
    "readout_fwd_bwd_raw",
    "SOLO_BF16",
    "SOLO_F32",
    "STATUS",
]

SOLO_BF16 = 0
SOLO_F32 = 1
STATUS = {
    "SOLO_OK": 0,
    "SOLO_ERR_NULL": 1,
    "SOLO_ERR_SHAPE": 2,
    "SOLO_ERR_DTYPE": 3,
    "SOLO_ERR_ALIGN": 4,
    "SOLO_ERR_WORKSPACE": 5,
    "SOLO_ERR_ARG": 6,
    "SOLO_ERR_HIP": 7,
}

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB = None

ReadoutResult = collections.namedtuple("ReadoutResult", ["losses", "dh", "dW", "dgain", "row_loss"])


class SoloError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"solo_readout status {status}: {msg}")
        self.status = status


def library_path() -> str:
    return os.environ.get("SOLO_READOUT_LIB", os.path.join(_PKG, "libsolo_readout.so"))


def load_library():
    """Load the HIP library once; raise if it has not been built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    try:
        # load torch's HIP runtime first so the library binds to the same one
        import torch  # noqa: F401
    except ImportError:
        pass
    path = library_path()
    if not os.path.exists(path):
        raise SoloError(-1, f"HIP library not found at {path}; build it with `python -m paper_2609_35440_amd.build`")
    lib = ctypes.CDLL(path)
    c_int, c_size, c_float, vp = ctypes.c_int, ctypes.c_size_t, ctypes.c_float, ctypes.c_void_p
    lib.solo_readout_abi_version.restype = c_int
    lib.solo_readout_abi_version.argtypes = []
    lib.solo_status_string.restype = ctypes.c_char_p
    lib.solo_status_string.argtypes = [c_int]
    lib.solo_readout_workspace_size.restype = c_size
    lib.solo_readout_workspace_size.argtypes = [c_int] * 6
    lib.solo_readout_kernel_family.restype = ctypes.c_char_p
    lib.solo_readout_kernel_family.argtypes = [c_int] * 5
    common = [
        c_int, c_int, c_int, c_int, c_int, c_float,  # K T d V dtype eps
        vp, vp, vp, vp, c_int,                      # h gain W targets final_module_dW
        vp, vp, vp, vp, vp,                         # losses row_loss dh dW dgain
        vp, c_size, vp,                             # workspace bytes stream
    ]
    lib.solo_readout_fwd_bwd.restype = c_int
    lib.solo_readout_fwd_bwd.argtypes = common
    lib.solo_readout_fwd_bwd_profiled.restype = c_int
    lib.solo_readout_fwd_bwd_profiled.argtypes = common + [ctypes.POINTER(vp)]
    _LIB = lib
    return lib


def header_functions() -> list:
    """Names of the functions declared in include/solo_readout.h."""
    hdr = os.path.join(os.path.dirname(_PKG), "include", "solo_readout.h")
    with open(hdr) as f:
        text = f.read()
    return re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(solo_\w+)\s*\(", text, re.M)


def abi_version() -> int:
    return load_library().solo_readout_abi_version()


def status_string(status: int) -> str:
    return load_library().solo_status_string(int(status)).decode()


def workspace_size(K: int, T: int, d: int, V: int, dtype: int, final_module_dW: bool = True) -> int:
    return int(load_library().solo_readout_workspace_size(K, T, d, V, dtype, int(final_module_dW)))


def kernel_family(K: int, T: int, d: int, V: int, dtype: int) -> str:
    return load_library().solo_readout_kernel_family(K, T, d, V, dtype).decode()


NUM_STAGES = 6
STAGE_NAMES = ["prep_readout", "row_rstd", "local_loss", "module_loss", "readout_grad", "dgain_reduce"]


def readout_fwd_bwd_raw(K, T, d, V, dtype, eps, h, gain, W, targets, final_module_dW, losses, row_loss, dh, dW,
                        dgain, workspace, workspace_bytes, stream, stage_events=None) -> int:
    """Direct call with integer pointers (0 for NULL); returns the status code.

    ``stage_events``: optional sequence of NUM_STAGES hipEvent_t handles (ints,
    0 for none), recorded after each stage (the profiled entry point).
    """
    lib = load_library()
    args = (int(K), int(T), int(d), int(V), int(dtype), float(eps),
            h or None, gain or None, W or None, targets or None, int(final_module_dW),
            losses or None, row_loss or None, dh or None, dW or None, dgain or None,
            workspace or None, int(workspace_bytes), stream or None)
    if stage_events is None:
        return int(lib.solo_readout_fwd_bwd(*args))
    arr = (ctypes.c_void_p * NUM_STAGES)(*[(e or None) for e in stage_events])
    return int(lib.solo_readout_fwd_bwd_profiled(*args, arr))


def _dtype_code(t):
    import torch

    if t == torch.bfloat16:
        return SOLO_BF16
    if t == torch.float32:
        return SOLO_F32
    raise TypeError(f"unsupported dtype {t}; use torch.bfloat16 or torch.float32")


def readout_fwd_bwd(h, gain, W, targets, final_module_dW: bool = True, eps: float = 1e-6, *,
                    row_loss: bool = False, workspace=None, out: Optional[ReadoutResult] = None,
                    stream=None, stage_events=None) -> ReadoutResult:
    """Shared-readout local loss of K modules and its local gradients.

    h [K, T, d], gain [d], W [V, d]: bf16 or fp32 CUDA/HIP tensors (same dtype);
    targets [K, T] integer.  Returns ReadoutResult(losses [K] fp32, dh like h,
    dW [V, d] fp32 or None, dgain [d] fp32 or None, row_loss [K, T] fp32 or None).
    The work is enqueued on ``stream`` (default: torch's current stream).
    """
    import torch

    if h.dim() != 3 or W.dim() != 2 or gain.dim() != 1 or targets.dim() != 2:
        raise ValueError("expected h [K,T,d], gain [d], W [V,d], targets [K,T]")
    K, T, d = h.shape
    V = W.shape[0]
    if W.shape[1] != d or gain.shape[0] != d or tuple(targets.shape) != (K, T):
        raise ValueError(f"shape mismatch: h {tuple(h.shape)}, gain {tuple(gain.shape)}, W {tuple(W.shape)}, "
                         f"targets {tuple(targets.shape)}")
    if not (h.dtype == gain.dtype == W.dtype):
        raise TypeError("h, gain and W must share one dtype")
    if not (h.is_cuda and gain.is_cuda and W.is_cuda and targets.is_cuda):
        raise ValueError("all inputs must be GPU tensors")
    dt = _dtype_code(h.dtype)
    dev = h.device
    h = h.contiguous()
    gain = gain.contiguous()
    W = W.contiguous()
    if targets.dtype != torch.int32:
        targets = targets.to(torch.int32)
    targets = targets.contiguous()

    fdw = bool(final_module_dW)
    if out is None:
        out = ReadoutResult(
            losses=torch.empty(K, dtype=torch.float32, device=dev),
            dh=torch.empty_like(h),
            dW=torch.empty((V, d), dtype=torch.float32, device=dev) if fdw else None,
            dgain=torch.empty(d, dtype=torch.float32, device=dev) if fdw else None,
            row_loss=torch.empty((K, T), dtype=torch.float32, device=dev) if row_loss else None,
        )
    ws_bytes = workspace_size(K, T, d, V, dt, fdw)
    if ws_bytes == 0:
        raise SoloError(STATUS["SOLO_ERR_SHAPE"], status_string(STATUS["SOLO_ERR_SHAPE"]))
    if workspace is None or workspace.numel() * workspace.element_size() < ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    st = readout_fwd_bwd_raw(
        K, T, d, V, dt, eps, h.data_ptr(), gain.data_ptr(), W.data_ptr(), targets.data_ptr(), fdw,
        out.losses.data_ptr(), out.row_loss.data_ptr() if out.row_loss is not None else 0, out.dh.data_ptr(),
        out.dW.data_ptr() if fdw else 0, out.dgain.data_ptr() if fdw else 0,
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), stream.cuda_stream, stage_events)
    if st != 0:
        raise SoloError(st, status_string(st))
    return out
