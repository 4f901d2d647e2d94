"""MI355X (gfx950) implementation of the AsymSpec fused decision step.

The compute lives in ``libasymspec.so`` (hand-written HIP for CDNA4); this
module only marshals arguments: torch tensors in, device pointers and the
current HIP stream out to the C ABI declared in ``include/asymspec.h``.
There is no fallback: if the library is missing, every call raises.
"""

from __future__ import annotations

import ctypes
import os

__all__ = ["fuse_verify", "workspace_size", "Workspace", "load_library", "status_string",
           "workspace_timeouts", "set_wait_limit",
           "BF16", "FP32", "GATE_CDA", "GATE_FIXED", "GATE_KL", "GATE_LAMBDA",
           "DELTA_AB", "DELTA_A", "DELTA_TB", "FUSE_BONUS", "EARLY_EXIT", "AsymSpecError"]

BF16 = 0
FP32 = 1
GATE_CDA = 0
GATE_FIXED = 1
GATE_KL = 2
GATE_LAMBDA = 3
DELTA_AB = 0
DELTA_A = 1
DELTA_TB = 2
FUSE_BONUS = 1
EARLY_EXIT = 2

OK = 0
E_ARG = -1
E_ALIGN = -2
E_WORKSPACE = -3
E_DEVICE = -4

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libasymspec.so")
_lib = None


class AsymSpecError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"asymspec error {status}: {msg}")
        self.status = status


class _Params(ctypes.Structure):
    _fields_ = [("beta", ctypes.c_float), ("gamma", ctypes.c_float),
                ("gate_mode", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("delta_mode", ctypes.c_int32), ("lam", ctypes.c_float),
                ("early_rows", ctypes.c_int32)]


def load_library(path: str | None = None):
    """Load (once) and return the ctypes handle of libasymspec.so."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise ImportError(f"{p} is missing: build it with `python -m paper_2608_26004_amd.build` "
                          "(hipcc --offload-arch=gfx950)")
    lib = ctypes.CDLL(p)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.asymspec_workspace_size.argtypes = [i32, i32, i32, i32]
    lib.asymspec_workspace_size.restype = sz
    lib.asymspec_workspace_clear.argtypes = [vp, sz, vp]
    lib.asymspec_workspace_clear.restype = i32
    lib.asymspec_fuse_verify.argtypes = [vp, vp, vp, i32, vp, vp, vp, vp, i32, i32, i32,
                                         ctypes.POINTER(_Params), vp, vp, vp, vp, vp, vp, sz, vp]
    lib.asymspec_fuse_verify.restype = i32
    lib.asymspec_fuse_verify_xvocab.argtypes = [vp, vp, vp, i32, vp, i32, vp, vp, vp, vp, i32, i32, i32,
                                                ctypes.POINTER(_Params), vp, vp, vp, vp, vp, vp, sz, vp]
    lib.asymspec_fuse_verify_xvocab.restype = i32
    lib.asymspec_workspace_size_xvocab.argtypes = [i32, i32, i32, i32, i32]
    lib.asymspec_workspace_size_xvocab.restype = sz
    lib.asymspec_status_string.argtypes = [i32]
    lib.asymspec_status_string.restype = ctypes.c_char_p
    lib.asymspec_version.argtypes = []
    lib.asymspec_version.restype = i32
    lib.asymspec_workspace_timeouts.argtypes = [vp, sz, vp, ctypes.POINTER(ctypes.c_uint32)]
    lib.asymspec_workspace_timeouts.restype = i32
    lib.asymspec_set_wait_limit.argtypes = [ctypes.c_ulonglong]
    lib.asymspec_set_wait_limit.restype = i32
    lib.asymspec_fuse_verify_noalloc.argtypes = [vp, vp, vp, i32, vp, vp, vp, vp, i32, i32, i32,
                                                 ctypes.POINTER(_Params), vp, vp, vp, vp, vp, vp]
    lib.asymspec_fuse_verify_noalloc.restype = i32
    lib.asymspec_noalloc_timeouts.argtypes = [vp, ctypes.POINTER(ctypes.c_uint32)]
    lib.asymspec_noalloc_timeouts.restype = i32
    if path is None:
        _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().asymspec_status_string(status).decode()


def workspace_size(B: int, K: int, V: int, dtype: int) -> int:
    return int(load_library().asymspec_workspace_size(B, K, V, dtype))


def _ptr(x):
    return None if x is None else ctypes.c_void_p(x.data_ptr())


def _stream_handle(device):
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


class Workspace:
    """A zero-filled device workspace reused across calls of one shape class
    (grows on demand).  Calls sharing one Workspace must not overlap."""

    def __init__(self, device=None):
        self.device = device
        self.buf = None

    def get(self, nbytes: int, device):
        import torch
        if self.buf is None or self.buf.numel() < nbytes or self.buf.device != device:
            # a replaced buffer goes back to torch's caching allocator, which
            # does not reuse it before the work recorded on it has finished
            self.buf = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=device)
        self.buf.record_stream(torch.cuda.current_stream(device))
        return self.buf

    def timeouts(self) -> int:
        """Timed-out waits counted in this workspace since it was allocated
        (synchronises the current stream); nonzero means some request's
        decision was not completed (its accept_len is -1)."""
        if self.buf is None:
            return 0
        return workspace_timeouts(self.buf)


# one default workspace per (device, stream): calls on different streams
# may overlap and must not share one
_default_ws = {}


def workspace_timeouts(buf) -> int:
    """The timeout count of a workspace tensor (see Workspace.timeouts)."""
    lib = load_library()
    n = ctypes.c_uint32(0)
    st = lib.asymspec_workspace_timeouts(_ptr(buf), buf.numel() * buf.element_size(),
                                         _stream_handle(buf.device), ctypes.byref(n))
    if st != OK:
        raise AsymSpecError(st, status_string(st))
    return int(n.value)


def set_wait_limit(ticks: int) -> None:
    """Bound of every wait between workgroups for later calls, in 10 ns
    ticks (0: the default 0.2 s); a test hook for the error path."""
    st = load_library().asymspec_set_wait_limit(int(ticks))
    if st != OK:
        raise AsymSpecError(st, status_string(st))


def fuse_verify(t, a, b, draft_tokens, draft_probs, uniforms, temperature,
                beta: float = 1.0, gamma: float = 0.5, gate_mode: int = GATE_CDA,
                return_gate: bool = False, workspace: Workspace | None = None, out=None,
                delta_mode: int = DELTA_AB, lam: float = 0.1, fuse_bonus: bool = False,
                return_full: bool = False, vocab_map=None, early_exit: int = 0):
    """One AsymSpec decision step on the current HIP stream.

    t, a, b: [B, K+1, V] torch.bfloat16 or torch.float32 on the GPU
    draft_tokens: [B, K] int32; draft_probs: [B, K] float32 or None;
    uniforms: [B, K+1] float32; temperature: [B] float32 (<= 0: greedy).
    gate_mode: GATE_CDA (the paper), GATE_FIXED, GATE_KL or GATE_LAMBDA (with
    scale lam); delta_mode: DELTA_AB (the paper), DELTA_A or DELTA_TB;
    fuse_bonus: take the bonus token from f_K rather than t_K (FUSE_BONUS);
    return_full: also return every element's log-probability under its row's
    distribution, [B, K+1, V] float32 (a second pass over the logits);
    vocab_map: for a drafter of another model family, [V] int32 on the GPU
    (drafter id of each verifier token, -1 if not shared); a and b are then
    [B, K+1, Vd] in the drafter's vocabulary;
    early_exit: 0 reads every row; n > 0 reads the first n rows, then the
    others only if none of those is surely rejected (EARLY_EXIT); the
    per-draft outputs of rows not read are NaN.
    Returns (accept_len [B] int32 (-1 marks a request whose decision did not
             complete on the device: see Workspace.timeouts), next_token [B] int32,
             fused_logprobs [B, K+1] float32[, gate [B, K, 2] float32]
             [, full [B, K+1, V] float32])."""
    import torch
    lib = load_library()
    if t.dtype == torch.bfloat16:
        dt = BF16
    elif t.dtype == torch.float32:
        dt = FP32
    else:
        raise TypeError(f"logits must be bfloat16 or float32, got {t.dtype}")
    if t.dim() != 3:
        raise ValueError("logits must be [B, K+1, V]")
    B, Kp1, V = t.shape
    K = Kp1 - 1
    dev = t.device
    Vd = V
    if vocab_map is not None:
        if vocab_map.dtype != torch.int32 or tuple(vocab_map.shape) != (V,) or vocab_map.device != dev:
            raise ValueError("vocab_map must be int32 [V] on the logits' device")
        if a.dim() != 3 or tuple(a.shape[:2]) != (B, Kp1):
            raise ValueError("a must be [B, K+1, Vd]")
        Vd = a.shape[2]
    for name, x in (("a", a), ("b", b)):
        if tuple(x.shape) != (B, Kp1, Vd) or x.dtype != t.dtype or x.device != dev:
            raise ValueError(f"{name} must be [B, K+1, {Vd}] with t's dtype and device")
    extra = (vocab_map,) if vocab_map is not None else ()
    for x in (t, a, b, draft_tokens, uniforms, temperature) + extra + ((draft_probs,) if draft_probs is not None else ()):
        if not x.is_contiguous():
            raise ValueError("all tensors must be contiguous")
    if draft_tokens.dtype != torch.int32 or tuple(draft_tokens.shape) != (B, K):
        raise ValueError("draft_tokens must be int32 [B, K]")
    if uniforms.dtype != torch.float32 or tuple(uniforms.shape) != (B, K + 1):
        raise ValueError("uniforms must be float32 [B, K+1]")
    if temperature.dtype != torch.float32 or tuple(temperature.shape) != (B,):
        raise ValueError("temperature must be float32 [B]")
    if draft_probs is not None and (draft_probs.dtype != torch.float32 or tuple(draft_probs.shape) != (B, K)):
        raise ValueError("draft_probs must be float32 [B, K] or None")
    if out is None:
        acc = torch.empty(B, dtype=torch.int32, device=dev)
        nxt = torch.empty(B, dtype=torch.int32, device=dev)
        flp = torch.empty(B, K + 1, dtype=torch.float32, device=dev)
        gate = torch.empty(B, K, 2, dtype=torch.float32, device=dev) if return_gate else None
        full = torch.empty(B, K + 1, V, dtype=torch.float32, device=dev) if return_full else None
    else:
        acc, nxt, flp, gate = out[:4]
        full = out[4] if len(out) > 4 else None
    ws_bytes = (workspace_size(B, K, V, dt) if vocab_map is None
                else int(lib.asymspec_workspace_size_xvocab(B, K, V, Vd, dt)))
    if ws_bytes == 0:
        raise AsymSpecError(E_ARG, "invalid shape")
    if workspace is None:
        key = (dev, torch.cuda.current_stream(dev).cuda_stream)
        workspace = _default_ws.setdefault(key, Workspace(dev))
    wsbuf = workspace.get(ws_bytes, dev)
    flags = (FUSE_BONUS if fuse_bonus else 0) | (EARLY_EXIT if early_exit else 0)
    params = _Params(float(beta), float(gamma), int(gate_mode), flags, int(delta_mode), float(lam),
                     int(early_exit))
    tail = (_ptr(draft_tokens), _ptr(draft_probs), _ptr(uniforms), _ptr(temperature),
            B, K, V, ctypes.byref(params), _ptr(acc), _ptr(nxt), _ptr(flp), _ptr(gate), _ptr(full),
            _ptr(wsbuf), wsbuf.numel(), _stream_handle(dev))
    if vocab_map is None:
        st = lib.asymspec_fuse_verify(_ptr(t), _ptr(a), _ptr(b), dt, *tail)
    else:
        st = lib.asymspec_fuse_verify_xvocab(_ptr(t), _ptr(a), _ptr(b), dt, _ptr(vocab_map), Vd, *tail)
    if st != OK:
        raise AsymSpecError(st, status_string(st))
    res = (acc, nxt, flp)
    if return_gate:
        res += (gate,)
    if return_full:
        res += (full,)
    return res
