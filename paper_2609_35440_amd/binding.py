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
    "readout_fwd_bwd_noalloc_raw",
    "scratch_limit",
    "SoloReadoutArgs",
    "GeneralResult",
    "EvalResult",
    "general_workspace_size",
    "exit_eval_workspace_size",
    "readout_general",
    "readout_general_raw",
    "exit_eval",
    "exit_eval_raw",
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
GeneralResult = collections.namedtuple(
    "GeneralResult", ["losses", "dh", "dW", "dWbar", "dgain", "dtau", "dbias", "row_loss"])
EvalResult = collections.namedtuple("EvalResult", ["losses", "row_loss", "top1"])


class SoloReadoutArgs(ctypes.Structure):
    """Mirror of ``solo_readout_args`` (same field order and C alignment)."""

    _fields_ = [
        ("K", ctypes.c_int), ("T", ctypes.c_int), ("d", ctypes.c_int), ("V", ctypes.c_int),
        ("dtype", ctypes.c_int), ("eps", ctypes.c_float),
        ("h", ctypes.c_void_p), ("gain", ctypes.c_void_p), ("W", ctypes.c_void_p), ("Wbar", ctypes.c_void_p),
        ("tau", ctypes.c_void_p), ("bias", ctypes.c_void_p), ("targets", ctypes.c_void_p),
        ("gain_per_module", ctypes.c_int), ("readout_per_head", ctypes.c_int),
        ("final_module_dW", ctypes.c_int), ("heads_train_readout", ctypes.c_int),
        ("losses", ctypes.c_void_p), ("row_loss", ctypes.c_void_p), ("dh", ctypes.c_void_p),
        ("dW", ctypes.c_void_p), ("dWbar", ctypes.c_void_p), ("dgain", ctypes.c_void_p),
        ("dtau", ctypes.c_void_p), ("dbias", ctypes.c_void_p), ("top1", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
        ("hip_stream", ctypes.c_void_p), ("stage_events", ctypes.c_void_p),
        ("rot", ctypes.c_void_p),
    ]


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
    lib.solo_readout_scratch_limit.restype = c_size
    lib.solo_readout_scratch_limit.argtypes = []
    lib.solo_readout_fwd_bwd_noalloc.restype = c_int
    lib.solo_readout_fwd_bwd_noalloc.argtypes = common[:16] + [vp]
    pargs = [ctypes.POINTER(SoloReadoutArgs)]
    for name in ("solo_readout_general_workspace_size", "solo_readout_exit_eval_workspace_size"):
        getattr(lib, name).restype = c_size
        getattr(lib, name).argtypes = pargs
    for name in ("solo_readout_general", "solo_readout_exit_eval"):
        getattr(lib, name).restype = c_int
        getattr(lib, name).argtypes = pargs
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
STAGE_NAMES = ["row_rstd", "local_loss", "module_sums", "readout_grad", "bias_grad", "dgain_reduce"]


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


def scratch_limit() -> int:
    """Bytes of the library's static scratch (the allocation-free entry point)."""
    return int(load_library().solo_readout_scratch_limit())


def readout_fwd_bwd_noalloc_raw(K, T, d, V, dtype, eps, h, gain, W, targets, final_module_dW, losses, row_loss, dh,
                                dW, dgain, stream) -> int:
    """solo_readout_fwd_bwd_noalloc with integer pointers (0 for NULL); returns the status code."""
    lib = load_library()
    return int(lib.solo_readout_fwd_bwd_noalloc(
        int(K), int(T), int(d), int(V), int(dtype), float(eps), h or None, gain or None, W or None, targets or None,
        int(final_module_dW), losses or None, row_loss or None, dh or None, dW or None, dgain or None,
        stream or None))


def _dtype_code(t):
    import torch

    if t == torch.bfloat16:
        return SOLO_BF16
    if t == torch.float32:
        return SOLO_F32
    raise TypeError(f"unsupported dtype {t}; use torch.bfloat16 or torch.float32")


def _check_targets(targets):
    import torch

    if targets.dtype.is_floating_point or targets.dtype.is_complex or targets.dtype == torch.bool:
        raise TypeError(f"targets must be an integer tensor, got {targets.dtype}")


def _check_device(dev, tensors):
    for name, t in tensors.items():
        if t is not None and t.device != dev:
            raise ValueError(f"{name} is on {t.device}, expected {dev} (all tensors on one GPU)")


def _check_out(out, spec, dev):
    """Every output this call writes must match (shape, dtype), sit on ``dev`` and be
    contiguous: the kernels write its full extent through its data pointer.  Returns
    name -> tensor for the outputs written, None for the others (whose pointers stay NULL)."""
    used = {}
    for name, (shape, dtype) in spec.items():
        t = getattr(out, name)
        used[name] = None
        if shape is None:
            continue
        if t is None:
            raise ValueError(f"out.{name} is required for this call")
        if tuple(t.shape) != tuple(shape) or t.dtype != dtype or t.device != dev or not t.is_contiguous():
            raise ValueError(f"out.{name}: expected contiguous {dtype} {tuple(shape)} on {dev}, "
                             f"got {'contiguous' if t.is_contiguous() else 'non-contiguous'} {t.dtype} "
                             f"{tuple(t.shape)} on {t.device}")
        used[name] = t
    return used


def _workspace(workspace, ws_bytes, dev):
    import torch

    if workspace is not None:
        if workspace.device != dev or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on the inputs' GPU")
        if workspace.numel() * workspace.element_size() >= ws_bytes:
            return workspace
    return torch.empty(ws_bytes, dtype=torch.uint8, device=dev)


def _streams(stream, dev):
    """The stream the call is enqueued on, and torch's current stream, on which the
    input conversions and new tensors of this call were made.  A different call
    stream first waits for the current one."""
    import torch

    cur = torch.cuda.current_stream(dev)
    if stream is None:
        return cur, cur
    if stream.device != dev:
        raise ValueError(f"stream is on {stream.device}, expected {dev}")
    if stream != cur:
        stream.wait_stream(cur)
    return stream, cur


def _hand_over(stream, cur, tensors):
    """Tensors made on ``cur`` and used on another ``stream``: tell the caching
    allocator, so that their memory is not reused before the stream has finished."""
    if stream == cur:
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


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
    _check_targets(targets)
    dt = _dtype_code(h.dtype)
    dev = h.device
    _check_device(dev, {"gain": gain, "W": W, "targets": targets})
    h = h.contiguous()
    gain = gain.contiguous()
    W = W.contiguous()
    targets = targets.to(torch.int32).contiguous()

    fdw = bool(final_module_dW)
    f32 = torch.float32
    made = []
    if out is None:
        out = ReadoutResult(
            losses=torch.empty(K, dtype=f32, device=dev),
            dh=torch.empty_like(h),
            dW=torch.empty((V, d), dtype=f32, device=dev) if fdw else None,
            dgain=torch.empty(d, dtype=f32, device=dev) if fdw else None,
            row_loss=torch.empty((K, T), dtype=f32, device=dev) if row_loss else None,
        )
        made = list(out)
    none = (None, None)
    used = _check_out(out, {"losses": ((K,), f32), "dh": ((K, T, d), h.dtype),
                            "dW": ((V, d), f32) if fdw else none, "dgain": ((d,), f32) if fdw else none,
                            "row_loss": ((K, T), f32) if out.row_loss is not None else none}, dev)
    ws_bytes = workspace_size(K, T, d, V, dt, fdw)
    if ws_bytes == 0:
        raise SoloError(STATUS["SOLO_ERR_SHAPE"], status_string(STATUS["SOLO_ERR_SHAPE"]))
    workspace = _workspace(workspace, ws_bytes, dev)
    stream, cur = _streams(stream, dev)
    _hand_over(stream, cur, [h, gain, W, targets, workspace] + made)
    st = readout_fwd_bwd_raw(
        K, T, d, V, dt, eps, h.data_ptr(), gain.data_ptr(), W.data_ptr(), targets.data_ptr(), fdw,
        used["losses"].data_ptr(), _ptr(used["row_loss"]) or 0, used["dh"].data_ptr(),
        _ptr(used["dW"]) or 0, _ptr(used["dgain"]) or 0,
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), stream.cuda_stream, stage_events)
    if st != 0:
        raise SoloError(st, status_string(st))
    return out


def general_workspace_size(args: SoloReadoutArgs) -> int:
    return int(load_library().solo_readout_general_workspace_size(ctypes.byref(args)))


def exit_eval_workspace_size(args: SoloReadoutArgs) -> int:
    return int(load_library().solo_readout_exit_eval_workspace_size(ctypes.byref(args)))


def readout_general_raw(args: SoloReadoutArgs) -> int:
    """Direct call with a filled SoloReadoutArgs; returns the status code."""
    return int(load_library().solo_readout_general(ctypes.byref(args)))


def exit_eval_raw(args: SoloReadoutArgs) -> int:
    return int(load_library().solo_readout_exit_eval(ctypes.byref(args)))


def _ptr(t):
    return t.data_ptr() if t is not None else None


def _fill_inputs(h, gain, W, targets, Wbar, tau, bias, eps, rot=None):
    """Validate shapes and build the input part of SoloReadoutArgs (tensors kept alive by the caller)."""
    import torch

    if h.dim() != 3 or W.dim() != 2 or gain.dim() not in (1, 2) or targets.dim() != 2:
        raise ValueError("expected h [K,T,d], gain [d] or [K,d], W [V,d], targets [K,T]")
    K, T, d = h.shape
    V = W.shape[0]
    if W.shape[1] != d or gain.shape[-1] != d or (gain.dim() == 2 and gain.shape[0] != K) \
            or tuple(targets.shape) != (K, T):
        raise ValueError(f"shape mismatch: h {tuple(h.shape)}, gain {tuple(gain.shape)}, W {tuple(W.shape)}, "
                         f"targets {tuple(targets.shape)}")
    if Wbar is not None and tuple(Wbar.shape) not in ((V, d), (K - 1, V, d)):
        raise ValueError(f"Wbar must be [V,d] or [K-1,V,d], got {tuple(Wbar.shape)}")
    if tau is not None and tuple(tau.shape) != (K,):
        raise ValueError("tau must be [K]")
    if bias is not None and tuple(bias.shape) != (K, V):
        raise ValueError("bias must be [K,V]")
    if rot is not None:
        if tuple(rot.shape) != (K - 1, d, d):
            raise ValueError(f"rot must be [K-1,d,d], got {tuple(rot.shape)}")
        if Wbar is not None and Wbar.dim() == 3:
            raise ValueError("rot rotates one shared readout: Wbar must be None or [V,d]")
    dts = {h.dtype, gain.dtype, W.dtype} | ({Wbar.dtype} if Wbar is not None else set()) \
        | ({rot.dtype} if rot is not None else set())
    if len(dts) != 1:
        raise TypeError("h, gain, W, Wbar and rot must share one dtype")
    for t in (h, gain, W, targets, Wbar, tau, bias, rot):
        if t is not None and not t.is_cuda:
            raise ValueError("all inputs must be GPU tensors")
    _check_targets(targets)
    _check_device(h.device, {"gain": gain, "W": W, "targets": targets, "Wbar": Wbar, "tau": tau, "bias": bias,
                             "rot": rot})
    keep = {
        "h": h.contiguous(), "gain": gain.contiguous(), "W": W.contiguous(),
        "Wbar": Wbar.contiguous() if Wbar is not None else None,
        "tau": tau.to(torch.float32).contiguous() if tau is not None else None,
        "bias": bias.to(torch.float32).contiguous() if bias is not None else None,
        "targets": targets.to(torch.int32).contiguous(),
        "rot": rot.contiguous() if rot is not None else None,
    }
    a = SoloReadoutArgs()
    a.K, a.T, a.d, a.V = K, T, d, V
    a.dtype = _dtype_code(h.dtype)
    a.eps = float(eps)
    for name in ("h", "gain", "W", "Wbar", "tau", "bias", "targets", "rot"):
        setattr(a, name, _ptr(keep[name]))
    a.gain_per_module = int(gain.dim() == 2)
    a.readout_per_head = int(Wbar is not None and Wbar.dim() == 3)
    return a, keep


def readout_general(h, gain, W, targets, *, Wbar=None, tau=None, bias=None, rot=None, final_module_dW: bool = True,
                    heads_train_readout: bool = False, want_dtau: bool = False, want_dbias: bool = False,
                    eps: float = 1e-6, row_loss: bool = False, workspace=None, stream=None,
                    stage_events=None, out: Optional[GeneralResult] = None) -> GeneralResult:
    """The loss with temperatures, biases, per-module gains and readout sources
    (``solo_readout_general``).  ``gain`` [d] or [K, d]; ``Wbar`` None, [V, d] or
    [K-1, V, d] (same dtype as h); ``tau`` [K] and ``bias`` [K, V] float32 or None;
    ``rot`` [K-1, d, d] (same dtype as h) or None: head k reads (Wbar or W) R_k (ROT).
    Returns GeneralResult; gradients that were not requested are None.  ``out``
    (a GeneralResult from an earlier call with the same arguments) reuses its tensors.
    """
    import torch

    a, keep = _fill_inputs(h, gain, W, targets, Wbar, tau, bias, eps, rot)
    K, T, d, V = a.K, a.T, a.d, a.V
    dev = h.device
    f32 = dict(dtype=torch.float32, device=dev)
    fdw = bool(final_module_dW)
    priv = bool(heads_train_readout)
    made = []
    if out is None:
        out = GeneralResult(
            losses=torch.empty(K, **f32),
            dh=torch.empty_like(keep["h"]),
            dW=torch.empty((V, d), **f32) if fdw else None,
            dWbar=torch.empty((K - 1, V, d), **f32) if (priv and K > 1) else None,
            dgain=(torch.empty((K, d), **f32) if a.gain_per_module else (torch.empty(d, **f32) if fdw else None)),
            dtau=torch.empty(K, **f32) if want_dtau else None,
            dbias=torch.empty((K, V), **f32) if want_dbias else None,
            row_loss=torch.empty((K, T), **f32) if row_loss else None,
        )
        made = list(out)
    fl = torch.float32
    none = (None, None)
    used = _check_out(out, {
        "losses": ((K,), fl), "dh": ((K, T, d), keep["h"].dtype),
        "dW": ((V, d), fl) if fdw else none,
        "dWbar": ((K - 1, V, d), fl) if (priv and K > 1) else none,
        "dgain": ((K, d), fl) if a.gain_per_module else (((d,), fl) if fdw else none),
        "dtau": ((K,), fl) if want_dtau else none,
        "dbias": ((K, V), fl) if want_dbias else none,
        "row_loss": ((K, T), fl) if out.row_loss is not None else none}, dev)
    a.final_module_dW = int(fdw)
    a.heads_train_readout = int(priv)
    for name in ("losses", "dh", "dW", "dWbar", "dgain", "dtau", "dbias", "row_loss"):
        setattr(a, name, _ptr(used[name]))
    ws_bytes = general_workspace_size(a)
    if ws_bytes == 0:
        raise SoloError(STATUS["SOLO_ERR_SHAPE"], status_string(STATUS["SOLO_ERR_SHAPE"]))
    workspace = _workspace(workspace, ws_bytes, dev)
    a.workspace = workspace.data_ptr()
    a.workspace_bytes = workspace.numel() * workspace.element_size()
    stream, cur = _streams(stream, dev)
    _hand_over(stream, cur, list(keep.values()) + [workspace] + made)
    a.hip_stream = stream.cuda_stream or None
    evs = None
    if stage_events is not None:
        evs = (ctypes.c_void_p * NUM_STAGES)(*[(e or None) for e in stage_events])
        a.stage_events = ctypes.cast(evs, ctypes.c_void_p)
    st = readout_general_raw(a)
    if st != 0:
        raise SoloError(st, status_string(st))
    return out


def exit_eval(h, gain, W, targets, *, Wbar=None, tau=None, bias=None, rot=None, eps: float = 1e-6,
              row_loss: bool = True,
              top1: bool = True, workspace=None, stream=None, stage_events=None,
              out: Optional[EvalResult] = None) -> EvalResult:
    """Forward-only exit evaluation (``solo_readout_exit_eval``): losses [K],
    row_loss [K, T] and top1 [K, T] int32 (argmax of the logits, lowest index on ties)."""
    import torch

    a, keep = _fill_inputs(h, gain, W, targets, Wbar, tau, bias, eps, rot)
    K, T = a.K, a.T
    dev = h.device
    made = []
    if out is None:
        out = EvalResult(
            losses=torch.empty(K, dtype=torch.float32, device=dev),
            row_loss=torch.empty((K, T), dtype=torch.float32, device=dev) if row_loss else None,
            top1=torch.empty((K, T), dtype=torch.int32, device=dev) if top1 else None,
        )
        made = list(out)
    used = _check_out(out, {"losses": ((K,), torch.float32),
                            "row_loss": ((K, T), torch.float32) if out.row_loss is not None else (None, None),
                            "top1": ((K, T), torch.int32) if out.top1 is not None else (None, None)}, dev)
    a.losses = _ptr(used["losses"])
    a.row_loss = _ptr(used["row_loss"])
    a.top1 = _ptr(used["top1"])
    ws_bytes = exit_eval_workspace_size(a)
    if ws_bytes == 0:
        raise SoloError(STATUS["SOLO_ERR_SHAPE"], status_string(STATUS["SOLO_ERR_SHAPE"]))
    workspace = _workspace(workspace, ws_bytes, dev)
    a.workspace = workspace.data_ptr()
    a.workspace_bytes = workspace.numel() * workspace.element_size()
    stream, cur = _streams(stream, dev)
    _hand_over(stream, cur, list(keep.values()) + [workspace] + made)
    a.hip_stream = stream.cuda_stream or None
    evs = None
    if stage_events is not None:
        evs = (ctypes.c_void_p * NUM_STAGES)(*[(e or None) for e in stage_events])
        a.stage_events = ctypes.cast(evs, ctypes.c_void_p)
    st = exit_eval_raw(a)
    if st != 0:
        raise SoloError(st, status_string(st))
    return out
