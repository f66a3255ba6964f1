"""Thin ctypes binding of liblinsimp.so (the C ABI in include/linsimp.h,
include/linsimp_head.h and include/linsimp_bank.h).

Argument marshalling only: torch tensors are turned into device pointers and
the current HIP stream is passed through.  Every step of the computation runs
in the library's HIP kernels; there is no CPU or PyTorch fallback, and every
entry point raises if the library is not built or a tensor is not on the GPU.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "liblinsimp.so")
_lib = None

F32, BF16 = 0, 1
EPS = 1e-30


class LinSimpError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"linsimp status {status}: {message}")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("H", ctypes.c_int64), ("n", ctypes.c_int64),
                ("D", ctypes.c_int32), ("Dv", ctypes.c_int32), ("m", ctypes.c_int32),
                ("w", ctypes.c_int32), ("dtype", ctypes.c_int32), ("eps", ctypes.c_float)]


class HeadOpts(ctypes.Structure):
    _fields_ = [("norm_eps", ctypes.c_float), ("rms_eps", ctypes.c_float), ("gate", ctypes.c_int32)]


GATE_HEAD, GATE_CHANNEL = 0, 1
NORM_EPS, RMS_EPS = 1e-12, 1e-6

BWD_REUSE_STATES = 1

EXPORTS = ("linsimp_workspace_size", "linsimp_fwd", "linsimp_fwd_static", "linsimp_bwd", "linsimp_bwd_ex",
           "linsimp_prefill",
           "linsimp_decode_step", "linsimp_decode_chunk", "linsimp_timing_enable",
           "linsimp_timing_read", "linsimp_last_error", "linsimp_version")
HEAD_EXPORTS = ("linsimp_head_saved_size", "linsimp_head_workspace_size", "linsimp_head_fwd",
                "linsimp_head_bwd", "linsimp_head_bwd_ex")
BANK_EXPORTS = ("linsimp_feature_bank",)


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load liblinsimp.so (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run paper_2608_09307_amd.build.build()")
    L = ctypes.CDLL(_LIB_PATH)
    vp, sz, i32, i64, f32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    pd = ctypes.POINTER(Dims)
    L.linsimp_workspace_size.argtypes = [pd, ctypes.c_int]
    L.linsimp_workspace_size.restype = sz
    L.linsimp_fwd.argtypes = [pd] + [vp] * 8 + [vp, sz, vp]
    L.linsimp_fwd.restype = ctypes.c_int
    L.linsimp_fwd_static.argtypes = [pd] + [vp] * 8 + [vp]
    L.linsimp_fwd_static.restype = ctypes.c_int
    L.linsimp_bwd.argtypes = [pd] + [vp] * 14 + [vp, sz, vp]
    L.linsimp_bwd.restype = ctypes.c_int
    L.linsimp_bwd_ex.argtypes = [pd] + [vp] * 14 + [i32, vp, sz, vp]
    L.linsimp_bwd_ex.restype = ctypes.c_int
    L.linsimp_prefill.argtypes = [pd] + [vp] * 11 + [vp, sz, vp]
    L.linsimp_prefill.restype = ctypes.c_int
    L.linsimp_decode_step.argtypes = [i64, i32, i32, i32, i32, i32, i32, f32] + [vp] * 13 + [vp]
    L.linsimp_decode_step.restype = ctypes.c_int
    L.linsimp_decode_chunk.argtypes = [i64, i32, i32, i32, i32, i32, i32, i32, f32] + [vp] * 13 + [vp]
    L.linsimp_decode_chunk.restype = ctypes.c_int
    L.linsimp_timing_enable.argtypes = [ctypes.c_int]
    L.linsimp_timing_enable.restype = ctypes.c_int
    L.linsimp_timing_read.argtypes = [ctypes.c_char_p, ctypes.c_int, ctypes.POINTER(ctypes.c_float),
                                      ctypes.POINTER(ctypes.c_int), ctypes.c_int]
    L.linsimp_timing_read.restype = ctypes.c_int
    L.linsimp_last_error.argtypes = []
    L.linsimp_last_error.restype = ctypes.c_char_p
    L.linsimp_version.argtypes = []
    L.linsimp_version.restype = ctypes.c_int
    po = ctypes.POINTER(HeadOpts)
    L.linsimp_head_saved_size.argtypes = [pd]
    L.linsimp_head_saved_size.restype = sz
    L.linsimp_head_workspace_size.argtypes = [pd, ctypes.c_int]
    L.linsimp_head_workspace_size.restype = sz
    L.linsimp_head_fwd.argtypes = [pd, po] + [vp] * 10 + [sz, vp, sz, vp]
    L.linsimp_head_fwd.restype = ctypes.c_int
    L.linsimp_head_bwd.argtypes = [pd, po] + [vp] * 17 + [vp, sz, vp]
    L.linsimp_head_bwd.restype = ctypes.c_int
    L.linsimp_head_bwd_ex.argtypes = [pd, po] + [vp] * 17 + [i32, vp, sz, vp]
    L.linsimp_head_bwd_ex.restype = ctypes.c_int
    L.linsimp_feature_bank.argtypes = [i32, i32, i32, vp, vp, vp, i32, vp]
    L.linsimp_feature_bank.restype = ctypes.c_int
    _lib = L
    return L


def _check(rc: int):
    if rc != 0:
        raise LinSimpError(rc, lib().linsimp_last_error().decode())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t: Optional[torch.Tensor], name: str):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _expect(pairs, device=None):
    """Check (tensor, name, shape, dtype) tuples before their pointers go to
    the C ABI, which sees bare pointers and trusts the sizes it is given: a
    tensor of the wrong shape would be read or written out of bounds.  Shape
    and dtype are checked first, then that every tensor is on the first one's
    device and that this is the current device (the launch stream's)."""
    for t, name, shape, dtype in pairs:
        if t is None:
            raise ValueError(f"{name} is required")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
        if t.dtype != dtype:
            raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    dev = device if device is not None else pairs[0][0].device
    for t, name, _, _ in pairs:
        if t.device != dev:
            raise ValueError(f"{name} is on {t.device}, expected {dev}")
    if dev.type == "cuda" and dev.index is not None and dev.index != torch.cuda.current_device():
        raise ValueError(f"tensors are on {dev} but the current device is cuda:{torch.cuda.current_device()}")


def _layer_shapes(q, v, omega):
    if q.dim() != 4 or v.dim() != 4 or omega.dim() != 3:
        raise ValueError("q, v must be [B, H, n, D|Dv] and omega [H, m, D]")
    B, H, n, D = q.shape
    return B, H, n, D, v.shape[-1], omega.shape[1]


def _layer_inputs(q, k, v, r, u, omega):
    B, H, n, D, Dv, m = _layer_shapes(q, v, omega)
    dt = q.dtype
    return [(q, "q", (B, H, n, D), dt), (k, "k", (B, H, n, D), dt), (v, "v", (B, H, n, Dv), dt),
            (r, "r", (B, H, n, D), dt), (u, "u", (B, H, n, Dv), dt),
            (omega, "omega", (H, m, D), torch.float32)]


def make_dims(B, H, n, D, Dv, m, w, dtype, eps=EPS) -> Dims:
    return Dims(B, H, n, D, Dv, m, w, dtype, eps)


def dims_of(q: torch.Tensor, v: torch.Tensor, omega: torch.Tensor, w: int, eps: float = EPS) -> Dims:
    B, H, n, D = q.shape
    return make_dims(B, H, n, D, v.shape[-1], omega.shape[1], w, _dtype_code(q), eps)


def workspace_size(d: Dims, backward: bool) -> int:
    return int(lib().linsimp_workspace_size(ctypes.byref(d), 1 if backward else 0))


def alloc_workspace(d: Dims, backward: bool, device) -> torch.Tensor:
    nbytes = workspace_size(d, backward)
    if nbytes == 0:
        _check(lib().linsimp_workspace_size(ctypes.byref(d), 1 if backward else 0) or -2)
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off: off + nbytes]


def fwd(q, k, v, r, u, omega, w, eps=EPS, out=None, stats=None, workspace=None,
        want_stats=True):
    """Forward pass; returns (out, stats).  See linsimp_fwd."""
    chk = _layer_inputs(q, k, v, r, u, omega)
    d = dims_of(q, v, omega, w, eps)
    if out is None:
        out = torch.empty(q.shape[:3] + (v.shape[-1],), dtype=q.dtype, device=q.device)
    if stats is None and want_stats:
        stats = torch.empty(q.shape[:3] + (2,), dtype=torch.float32, device=q.device)
    chk.append((out, "out", q.shape[:3] + (v.shape[-1],), q.dtype))
    if stats is not None:
        chk.append((stats, "stats", q.shape[:3] + (2,), torch.float32))
    _expect(chk)
    if workspace is None:
        workspace = alloc_workspace(d, False, q.device)
    _check(lib().linsimp_fwd(ctypes.byref(d), _ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"),
                             _ptr(r, "r"), _ptr(u, "u"), _ptr(omega, "omega"), _ptr(out, "out"),
                             _ptr(stats, "stats"), _ptr(workspace, "workspace"),
                             workspace.numel(), _stream()))
    return out, stats


FWD_STATIC_MAX_BYTES = 64 << 20      # LINSIMP_FWD_STATIC_MAX_BYTES


def fwd_static(q, k, v, r, u, omega, w, eps=EPS, out=None, stats=None, want_stats=True):
    """Forward pass with the library's static scratch instead of a workspace
    (linsimp_fwd_static: nothing is allocated by the library; ``out`` and
    ``stats`` are allocated here unless given); returns (out, stats)."""
    chk = _layer_inputs(q, k, v, r, u, omega)
    d = dims_of(q, v, omega, w, eps)
    if out is None:
        out = torch.empty(q.shape[:3] + (v.shape[-1],), dtype=q.dtype, device=q.device)
    if stats is None and want_stats:
        stats = torch.empty(q.shape[:3] + (2,), dtype=torch.float32, device=q.device)
    chk.append((out, "out", q.shape[:3] + (v.shape[-1],), q.dtype))
    if stats is not None:
        chk.append((stats, "stats", q.shape[:3] + (2,), torch.float32))
    _expect(chk)
    _check(lib().linsimp_fwd_static(ctypes.byref(d), _ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"),
                                    _ptr(r, "r"), _ptr(u, "u"), _ptr(omega, "omega"), _ptr(out, "out"),
                                    _ptr(stats, "stats"), _stream()))
    return out, stats


def bwd(q, k, v, r, u, omega, w, out, stats, dout, eps=EPS, grads=None, workspace=None,
        reuse_states=False):
    """Backward pass; returns (dq, dk, dv, dr, du).  See linsimp_bwd; with
    ``reuse_states`` (linsimp_bwd_ex, LINSIMP_BWD_REUSE_STATES) ``workspace``
    must be the backward-sized workspace the matching fwd call used."""
    chk = _layer_inputs(q, k, v, r, u, omega)
    d = dims_of(q, v, omega, w, eps)
    if grads is None:
        grads = tuple(torch.empty_like(x) for x in (q, k, v, r, u))
    dq, dk, dv, dr, du = grads
    ov = q.shape[:3] + (v.shape[-1],)
    chk += [(out, "out", ov, q.dtype), (stats, "stats", q.shape[:3] + (2,), torch.float32),
            (dout, "dout", ov, q.dtype)]
    chk += [(g, "d" + nm, x.shape, x.dtype) for g, nm, x in zip(grads, "qkvru", (q, k, v, r, u))]
    _expect(chk)
    if workspace is None:
        if reuse_states:
            raise ValueError("reuse_states needs the workspace of the matching forward call")
        workspace = alloc_workspace(d, True, q.device)
    _check(lib().linsimp_bwd_ex(ctypes.byref(d), _ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"),
                                _ptr(r, "r"), _ptr(u, "u"), _ptr(omega, "omega"), _ptr(out, "out"),
                                _ptr(stats, "stats"), _ptr(dout, "dout"), _ptr(dq, "dq"),
                                _ptr(dk, "dk"), _ptr(dv, "dv"), _ptr(dr, "dr"), _ptr(du, "du"),
                                BWD_REUSE_STATES if reuse_states else 0,
                                _ptr(workspace, "workspace"), workspace.numel(), _stream()))
    return dq, dk, dv, dr, du


def timing_enable(on: bool = True):
    """Bracket every library kernel launch with HIP events (see linsimp_timing_enable)."""
    _check(lib().linsimp_timing_enable(1 if on else 0))


def timing_read(max_kernels: int = 64):
    """Per-kernel {name: (total_ms, launches)} since the previous read."""
    names = ctypes.create_string_buffer(4096)
    tot = (ctypes.c_float * max_kernels)()
    cnt = (ctypes.c_int * max_kernels)()
    nk = lib().linsimp_timing_read(names, 4096, tot, cnt, max_kernels)
    if nk < 0:
        _check(nk)
    keys = names.value.decode().split("\n")[:nk]
    return {k: (float(tot[i]), int(cnt[i])) for i, k in enumerate(keys)}


def prefill(k, v, r, u, omega, w, eps=EPS, workspace=None):
    """Decode state after a prefix (k, v, r, u: [S, H, n, *]).  Returns a dict
    with M [S,H,m,Dv], a [S,H,m], rho [S,H] (log2 frame), ring_r, ring_u, pos."""
    S, H, n, D, Dv, m = _layer_shapes(k, v, omega)
    _expect([(k, "k", (S, H, n, D), k.dtype), (v, "v", (S, H, n, Dv), k.dtype),
             (r, "r", (S, H, n, D), k.dtype), (u, "u", (S, H, n, Dv), k.dtype),
             (omega, "omega", (H, m, D), torch.float32)])
    d = make_dims(S, H, n, D, Dv, m, w, _dtype_code(k), eps)
    dev = k.device
    st = {"M": torch.empty(S, H, m, Dv, dtype=torch.float32, device=dev),
          "a": torch.empty(S, H, m, dtype=torch.float32, device=dev),
          "rho": torch.empty(S, H, dtype=torch.float32, device=dev),
          "ring_r": torch.empty(S, H, w, D, dtype=k.dtype, device=dev),
          "ring_u": torch.empty(S, H, w, Dv, dtype=k.dtype, device=dev),
          "pos": torch.empty(S, dtype=torch.int64, device=dev)}
    if workspace is None:
        workspace = alloc_workspace(d, False, dev)
    _check(lib().linsimp_prefill(ctypes.byref(d), _ptr(k, "k"), _ptr(v, "v"), _ptr(r, "r"),
                                 _ptr(u, "u"), _ptr(omega, "omega"), _ptr(st["M"], "M"),
                                 _ptr(st["a"], "a"), _ptr(st["rho"], "rho"),
                                 _ptr(st["ring_r"], "ring_r"), _ptr(st["ring_u"], "ring_u"),
                                 _ptr(st["pos"], "pos"), _ptr(workspace, "workspace"),
                                 workspace.numel(), _stream()))
    return st


def _decode_checks(state, q, k, v, r, u, omega, w, out, tok):
    """Shapes of a decode call: tok is () for one token, (T,) for a chunk."""
    if q.dim() != 3 + len(tok) or omega.dim() != 3:
        raise ValueError("q must be [S, H, *tok, D] and omega [H, m, D]")
    S, H, D = q.shape[0], q.shape[1], q.shape[-1]
    Dv, m, dt = v.shape[-1], omega.shape[1], q.dtype
    f32 = torch.float32
    _expect([(q, "q", (S, H, *tok, D), dt), (k, "k", (S, H, *tok, D), dt), (v, "v", (S, H, *tok, Dv), dt),
             (r, "r", (S, H, *tok, D), dt), (u, "u", (S, H, *tok, Dv), dt),
             (omega, "omega", (H, m, D), f32), (state["M"], "M", (S, H, m, Dv), f32),
             (state["a"], "a", (S, H, m), f32), (state["rho"], "rho", (S, H), f32),
             (state["ring_r"], "ring_r", (S, H, w, D), dt), (state["ring_u"], "ring_u", (S, H, w, Dv), dt),
             (state["pos"], "pos", (S,), torch.int64), (out, "out", (S, H, *tok, Dv), dt)])
    return S, H, D, Dv, m


def decode_step(state, q, k, v, r, u, omega, w, eps=EPS, out=None):
    """One decode step for S sequences (q, k, v, r, u: [S, H, *]); updates
    ``state`` in place and returns out [S, H, Dv]."""
    if out is None:
        out = torch.empty(q.shape[:2] + (v.shape[-1],), dtype=q.dtype, device=q.device)
    S, H, D, Dv, m = _decode_checks(state, q, k, v, r, u, omega, w, out, ())
    _check(lib().linsimp_decode_step(S, H, D, Dv, m, w, _dtype_code(q), eps, _ptr(q, "q"),
                                     _ptr(k, "k"), _ptr(v, "v"), _ptr(r, "r"), _ptr(u, "u"),
                                     _ptr(omega, "omega"), _ptr(state["M"], "M"),
                                     _ptr(state["a"], "a"), _ptr(state["rho"], "rho"),
                                     _ptr(state["ring_r"], "ring_r"),
                                     _ptr(state["ring_u"], "ring_u"), _ptr(state["pos"], "pos"),
                                     _ptr(out, "out"), _stream()))
    return out


def decode_chunk(state, q, k, v, r, u, omega, w, eps=EPS, out=None):
    """T consecutive decode steps for S sequences (q, k, v, r, u: [S, H, T, *]);
    updates ``state`` in place and returns out [S, H, T, Dv]."""
    if out is None:
        out = torch.empty(q.shape[:3] + (v.shape[-1],), dtype=q.dtype, device=q.device)
    T = q.shape[2]
    S, H, D, Dv, m = _decode_checks(state, q, k, v, r, u, omega, w, out, (T,))
    _check(lib().linsimp_decode_chunk(S, H, T, D, Dv, m, w, _dtype_code(q), eps, _ptr(q, "q"),
                                      _ptr(k, "k"), _ptr(v, "v"), _ptr(r, "r"), _ptr(u, "u"),
                                      _ptr(omega, "omega"), _ptr(state["M"], "M"),
                                      _ptr(state["a"], "a"), _ptr(state["rho"], "rho"),
                                      _ptr(state["ring_r"], "ring_r"),
                                      _ptr(state["ring_u"], "ring_u"), _ptr(state["pos"], "pos"),
                                      _ptr(out, "out"), _stream()))
    return out


# ---------------------------------------------------------------------------
# Full head (include/linsimp_head.h)
# ---------------------------------------------------------------------------

def _aligned_bytes(nbytes: int, device) -> torch.Tensor:
    buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-buf.data_ptr()) % 256
    return buf[off: off + nbytes]


def head_opts(gate_kind=GATE_HEAD, norm_eps=NORM_EPS, rms_eps=RMS_EPS) -> HeadOpts:
    return HeadOpts(norm_eps, rms_eps, gate_kind)


def _gate_kind(gate: torch.Tensor, v: torch.Tensor) -> int:
    return GATE_CHANNEL if gate.dim() == 4 else GATE_HEAD


def _head_params(q, v, tau, gate):
    H = q.shape[1]
    gshape, gdt = ((q.shape[:3] + (v.shape[-1],), q.dtype) if gate.dim() == 4 else ((H,), torch.float32))
    return [(tau, "tau", (H,), torch.float32), (gate, "gate", gshape, gdt)]


def head_fwd(q, k, v, r, u, omega, w, tau, gate, eps=EPS, norm_eps=NORM_EPS, rms_eps=RMS_EPS,
             y=None, saved=None, workspace=None):
    """Forward of one full head; returns (y, saved).  ``gate`` is gamma [H]
    float32 (per-head gate) or logits [B, H, n, Dv] (channel-wise gate).
    See linsimp_head_fwd."""
    d = dims_of(q, v, omega, w, eps)
    o = head_opts(_gate_kind(gate, v), norm_eps, rms_eps)
    L = lib()
    if y is None:
        y = torch.empty(q.shape[:3] + (v.shape[-1],), dtype=q.dtype, device=q.device)
    _expect(_layer_inputs(q, k, v, r, u, omega) + _head_params(q, v, tau, gate)
            + [(y, "y", q.shape[:3] + (v.shape[-1],), q.dtype)])
    if saved is None:
        nb = int(L.linsimp_head_saved_size(ctypes.byref(d)))
        if nb == 0:
            _check(-2)
        saved = _aligned_bytes(nb, q.device)
    if workspace is None:
        nb = int(L.linsimp_head_workspace_size(ctypes.byref(d), 0))
        if nb == 0:
            _check(-2)
        workspace = _aligned_bytes(nb, q.device)
    _check(L.linsimp_head_fwd(ctypes.byref(d), ctypes.byref(o), _ptr(q, "q"), _ptr(k, "k"),
                              _ptr(v, "v"), _ptr(r, "r"), _ptr(u, "u"), _ptr(omega, "omega"),
                              _ptr(tau, "tau"), _ptr(gate, "gate"), _ptr(y, "y"),
                              _ptr(saved, "saved"), saved.numel(), _ptr(workspace, "workspace"),
                              workspace.numel(), _stream()))
    return y, saved


def head_bwd(q, k, v, r, u, omega, w, tau, gate, saved, dy, eps=EPS, norm_eps=NORM_EPS,
             rms_eps=RMS_EPS, workspace=None, reuse_states=False):
    """Backward of one full head; returns (dq, dk, dv, dr, du, dtau, dgate).
    See linsimp_head_bwd; with ``reuse_states`` (linsimp_head_bwd_ex)
    ``workspace`` must be the backward-sized one the matching head_fwd used."""
    d = dims_of(q, v, omega, w, eps)
    o = head_opts(_gate_kind(gate, v), norm_eps, rms_eps)
    L = lib()
    _expect(_layer_inputs(q, k, v, r, u, omega) + _head_params(q, v, tau, gate)
            + [(dy, "dy", q.shape[:3] + (v.shape[-1],), q.dtype)])
    grads = [torch.empty_like(x) for x in (q, k, v, r, u)]
    dtau = torch.empty_like(tau)
    dgate = torch.empty_like(gate)
    if workspace is None:
        if reuse_states:
            raise ValueError("reuse_states needs the workspace of the matching head_fwd call")
        nb = int(L.linsimp_head_workspace_size(ctypes.byref(d), 1))
        if nb == 0:
            _check(-2)
        workspace = _aligned_bytes(nb, q.device)
    _check(L.linsimp_head_bwd_ex(ctypes.byref(d), ctypes.byref(o), _ptr(q, "q"), _ptr(k, "k"),
                                 _ptr(v, "v"), _ptr(r, "r"), _ptr(u, "u"), _ptr(omega, "omega"),
                                 _ptr(tau, "tau"), _ptr(gate, "gate"), _ptr(saved, "saved"),
                                 _ptr(dy, "dy"), *[_ptr(g, "grad") for g in grads],
                                 _ptr(dtau, "dtau"), _ptr(dgate, "dgate"),
                                 BWD_REUSE_STATES if reuse_states else 0,
                                 _ptr(workspace, "workspace"), workspace.numel(), _stream()))
    return (*grads, dtau, dgate)


# ---------------------------------------------------------------------------
# Orthogonal random-feature bank (include/linsimp_bank.h)
# ---------------------------------------------------------------------------

def feature_bank(gauss, radii, m, sign_correct=True, omega=None):
    """Bank [H, m, D] float32 from draws gauss [H, nb, D, D] and radii
    [H, nb, D] (float32, on the GPU).  See linsimp_feature_bank."""
    H, nb, D, _ = gauss.shape
    if gauss.dtype != torch.float32 or radii.dtype != torch.float32:
        raise TypeError("gauss and radii must be float32")
    if radii.shape != (H, nb, D) or nb != (m + D - 1) // D:
        raise ValueError("gauss must be [H, ceil(m/D), D, D] and radii [H, ceil(m/D), D]")
    if omega is None:
        omega = torch.empty(H, m, D, dtype=torch.float32, device=gauss.device)
    _check(lib().linsimp_feature_bank(H, m, D, _ptr(gauss, "gauss"), _ptr(radii, "radii"),
                                      _ptr(omega, "omega"), 1 if sign_correct else 0, _stream()))
    return omega
