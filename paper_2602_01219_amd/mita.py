"""Python binding of libmita (the gfx950 MiTA forward library).

Argument marshalling only: every step of the forward runs in the HIP kernels
behind the C ABI declared in include/mita.h. Tensors are torch device tensors
(torch provides device memory and the current HIP stream); the functions
allocate outputs and workspaces with torch when they are not given.

There is no CPU fallback: if libmita.so is missing or no GPU is visible the
calls raise.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmita.so")

MITA_OK, MITA_ERR_INVALID_ARG, MITA_ERR_UNSUPPORTED, MITA_ERR_WORKSPACE, MITA_ERR_HIP = range(5)
MITA_F32, MITA_BF16 = 0, 1
MITA_FLAG_STAGED_GATHER = 0x1
MITA_FLAG_FULL_SCORES = 0x2
WS_FORWARD, WS_SCORES, WS_TOPK, WS_ROUTE, WS_ATTEND, WS_BACKWARD, WS_TOME = range(7)
NUM_STAGES = 6
MAX_LAUNCHES = 32
STAGES = ("landmarks", "scores", "topk", "gather", "route", "attend")
MAX_N = 65536
MAX_S = 4

EXPORTED = ("mita_check", "mita_workspace_size", "mita_status_string", "mita_last_error", "mita_forward",
            "mita_landmarks", "mita_scores", "mita_topk", "mita_gather", "mita_route", "mita_attend",
            "mita_timer_create", "mita_timer_destroy", "mita_timer_reset", "mita_timer_read",
            "mita_forward_timed", "mita_forward_fallbacks", "mita_select_plan", "mita_timer_launches",
            "mita_forward_noalloc", "mita_landmarks_select", "mita_forward_lm", "mita_forward_lm_timed",
            "mita_backward", "mita_backward_timed", "mita_landmarks_tome")


class CfgStruct(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("B", "H", "N", "d", "grid_h", "grid_w", "M", "lm_h", "lm_w", "k", "s", "use_shared",
                 "use_routed", "dtype")] + [("scale", ctypes.c_float), ("flags", ctypes.c_uint32)]


class MitaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"mita status {status}: {msg}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libmita.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} not found: build it with `python -m paper_2602_01219_amd.build`")
    lib = ctypes.CDLL(path)
    P, I, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    cfgp = ctypes.POINTER(CfgStruct)
    sig = {
        "mita_check": (I, [cfgp]),
        "mita_workspace_size": (Z, [cfgp, I]),
        "mita_status_string": (ctypes.c_char_p, [I]),
        "mita_last_error": (ctypes.c_char_p, []),
        "mita_forward": (I, [cfgp, P, P, P, P, P, Z, P]),
        "mita_forward_timed": (I, [cfgp, P, P, P, P, P, Z, P, P]),
        "mita_forward_noalloc": (I, [cfgp, P, P, P, P, P]),
        "mita_forward_fallbacks": (I, [cfgp, P, Z, ctypes.POINTER(ctypes.c_int64), P]),
        "mita_select_plan": (I, [cfgp] + [ctypes.POINTER(ctypes.c_int32)] * 4),
        "mita_landmarks": (I, [cfgp, P, P, P]),
        "mita_landmarks_select": (I, [cfgp, P, P, P, P]),
        "mita_forward_lm": (I, [cfgp, P, P, P, P, P, P, Z, P]),
        "mita_forward_lm_timed": (I, [cfgp, P, P, P, P, P, P, Z, P, P]),
        "mita_backward": (I, [cfgp, P, P, P, P, P, P, P, P, P, Z, P]),
        "mita_landmarks_tome": (I, [cfgp, P, P, P, P, Z, P]),
        "mita_backward_timed": (I, [cfgp, P, P, P, P, P, P, P, P, P, Z, P, P]),
        "mita_scores": (I, [cfgp, P, P, P, P, P, P, Z, P]),
        "mita_topk": (I, [cfgp, P, P, P, Z, P]),
        "mita_gather": (I, [cfgp, P, P, P, P, P, P]),
        "mita_route": (I, [cfgp, P, P, P, P, P, P, Z, P]),
        "mita_attend": (I, [cfgp, P, P, P, P, P, P, P, P, P, Z, P]),
        "mita_timer_create": (I, [ctypes.POINTER(P), I]),
        "mita_timer_destroy": (I, [P]),
        "mita_timer_reset": (I, [P]),
        "mita_timer_read": (I, [P, ctypes.POINTER(ctypes.c_float), I, ctypes.POINTER(I)]),
        "mita_timer_launches": (I, [P, I, I, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_int32),
                                    ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_int32)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != MITA_OK:
        lib = load_library()
        raise MitaError(status, lib.mita_last_error().decode() or lib.mita_status_string(status).decode())


@dataclass(frozen=True)
class Config:
    """Problem description (mirrors mita_cfg_t)."""
    B: int
    H: int
    N: int
    d: int
    grid_h: int
    grid_w: int
    M: int
    lm_h: int
    lm_w: int
    k: int
    dtype: str = "bf16"          # "f32" | "bf16"
    use_shared: int = 1
    use_routed: int = 1
    s: int = 1
    scale: float = 0.0           # 0 -> 1/sqrt(d)
    staged_gather: bool = False
    full_scores: bool = False    # store S and select from it instead of the fused selection

    @staticmethod
    def from_workload(wl, **kw) -> "Config":
        c = dict(B=wl.B, H=wl.H, N=wl.N, d=wl.d, grid_h=wl.grid_h, grid_w=wl.grid_w, M=wl.M, lm_h=wl.lm_h,
                 lm_w=wl.lm_w, k=wl.k, dtype=wl.dtype, use_shared=wl.use_shared, use_routed=wl.use_routed)
        c.update(kw)
        return Config(**c)

    def struct(self) -> CfgStruct:
        return CfgStruct(self.B, self.H, self.N, self.d, self.grid_h, self.grid_w, self.M, self.lm_h, self.lm_w,
                         self.k, self.s, self.use_shared, self.use_routed,
                         MITA_F32 if self.dtype == "f32" else MITA_BF16, float(self.scale),
                         (MITA_FLAG_STAGED_GATHER if self.staged_gather else 0)
                         | (MITA_FLAG_FULL_SCORES if self.full_scores else 0))

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def eff_scale(self) -> float:
        return self.scale if self.scale else 1.0 / math.sqrt(self.d)


def _p(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def check(cfg: Config) -> int:
    return load_library().mita_check(ctypes.byref(cfg.struct()))


def workspace_size(cfg: Config, which: int = WS_FORWARD) -> int:
    return int(load_library().mita_workspace_size(ctypes.byref(cfg.struct()), which))


def _ws(cfg, which, ws, device):
    n = workspace_size(cfg, which)
    if ws is None and n:
        ws = torch.empty(n, dtype=torch.uint8, device=device)
    return ws, (ws.numel() if ws is not None else 0)


def _dev(t):
    if not t.is_cuda:
        raise ValueError("tensors must be on the GPU")
    return t.device


def forward(cfg: Config, q, k, v, o=None, ws=None, stream=None, timer: "Timer" = None, q_lm=None):
    """MiTA forward: o [B, H, N, d]. With q_lm [B, H, M, d] given (e.g. from
    landmarks_select), the forward uses those landmark queries instead of
    pooling them (mita_forward_lm)."""
    lib = load_library()
    dev = _dev(q)
    if o is None:
        o = torch.empty_like(q)
    ws, nws = _ws(cfg, WS_FORWARD, ws, dev)
    c = cfg.struct()
    if q_lm is not None:
        if timer is None:
            st = lib.mita_forward_lm(ctypes.byref(c), _p(q), _p(k), _p(v), _p(q_lm), _p(o), _p(ws), nws,
                                     _stream(stream))
        else:
            st = lib.mita_forward_lm_timed(ctypes.byref(c), _p(q), _p(k), _p(v), _p(q_lm), _p(o), _p(ws), nws,
                                           _stream(stream), timer.handle)
        _check(st)
        return o
    if timer is None:
        st = lib.mita_forward(ctypes.byref(c), _p(q), _p(k), _p(v), _p(o), _p(ws), nws, _stream(stream))
    else:
        st = lib.mita_forward_timed(ctypes.byref(c), _p(q), _p(k), _p(v), _p(o), _p(ws), nws, _stream(stream),
                                    timer.handle)
    _check(st)
    return o


def backward(cfg: Config, q, k, v, o, dO, dq=None, dk=None, dv=None, ws=None, stream=None,
             timer: "Timer" = None):
    """Gradients (dq, dk, dv) [B, H, N, d] of the forward's output o for the
    upstream gradient dO, the top-k sets and routing held fixed
    (mita_backward)."""
    lib = load_library()
    dev = _dev(q)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    ws, nws = _ws(cfg, WS_BACKWARD, ws, dev)
    c = cfg.struct()
    args = [ctypes.byref(c), _p(q), _p(k), _p(v), _p(o), _p(dO), _p(dq), _p(dk), _p(dv), _p(ws), nws, _stream(stream)]
    if timer is None:
        _check(lib.mita_backward(*args))
    else:
        _check(lib.mita_backward_timed(*args, timer.handle))
    return dq, dk, dv


NOALLOC_SCRATCH_BYTES = 64 << 20


def forward_noalloc(cfg: Config, q, k, v, o=None, stream=None):
    """MiTA forward with the library's static scratch as workspace (no
    allocation by the library; only the output is allocated here if not
    given). Raises MitaError(MITA_ERR_WORKSPACE) if the forward needs more
    than NOALLOC_SCRATCH_BYTES of workspace."""
    lib = load_library()
    _dev(q)
    if o is None:
        o = torch.empty_like(q)
    _check(lib.mita_forward_noalloc(ctypes.byref(cfg.struct()), _p(q), _p(k), _p(v), _p(o), _stream(stream)))
    return o


def forward_fallbacks(cfg: Config, ws, stream=None) -> int:
    """Landmark rows whose fused top-k selection fell back to the full score
    row in the last forward on workspace ws (synchronises the stream)."""
    n = ctypes.c_int64()
    _check(load_library().mita_forward_fallbacks(ctypes.byref(cfg.struct()), _p(ws), ws.numel(), ctypes.byref(n),
                                                 _stream(stream)))
    return n.value


def select_plan(cfg: Config) -> dict:
    """How the forward selects the top-k sets (host only): fused in the score
    pass (with its sample size, pivot rank and list cap) or from the stored
    score matrix."""
    v = [ctypes.c_int32() for _ in range(4)]
    _check(load_library().mita_select_plan(ctypes.byref(cfg.struct()), *[ctypes.byref(x) for x in v]))
    return dict(zip(("fused", "ns", "rank", "cap"), (x.value for x in v)))


def landmarks(cfg: Config, q, q_lm=None, stream=None):
    lib = load_library()
    if q_lm is None:
        q_lm = torch.empty((cfg.B, cfg.H, cfg.M, cfg.d), dtype=q.dtype, device=_dev(q))
    _check(lib.mita_landmarks(ctypes.byref(cfg.struct()), _p(q), _p(q_lm), _stream(stream)))
    return q_lm


def landmarks_select(cfg: Config, q, sel, q_lm=None, stream=None):
    """Random-selection landmarks: q_lm[b, h, i] = q[b, h, sel[b, h, i]];
    sel: [B, H, M] int32 device tensor of drawn token indices."""
    lib = load_library()
    if sel.dtype != torch.int32 or tuple(sel.shape) != (cfg.B, cfg.H, cfg.M) or not sel.is_contiguous():
        raise ValueError("sel must be a contiguous [B, H, M] int32 tensor")
    if q_lm is None:
        q_lm = torch.empty((cfg.B, cfg.H, cfg.M, cfg.d), dtype=q.dtype, device=_dev(q))
    _check(lib.mita_landmarks_select(ctypes.byref(cfg.struct()), _p(q), _p(sel), _p(q_lm), _stream(stream)))
    return q_lm


def landmarks_tome(cfg: Config, q, q_lm=None, want_assign=True, ws=None, stream=None):
    """Token-merging landmarks: (q_lm [B, H, M, d], assign [B, H, N] int32 or
    None), mita_landmarks_tome."""
    lib = load_library()
    dev = _dev(q)
    if q_lm is None:
        q_lm = torch.empty((cfg.B, cfg.H, cfg.M, cfg.d), dtype=q.dtype, device=dev)
    assign = torch.empty((cfg.B, cfg.H, cfg.N), dtype=torch.int32, device=dev) if want_assign else None
    ws, nws = _ws(cfg, WS_TOME, ws, dev)
    _check(lib.mita_landmarks_tome(ctypes.byref(cfg.struct()), _p(q), _p(q_lm), _p(assign), _p(ws), nws,
                                   _stream(stream)))
    return q_lm, assign


def scores(cfg: Config, q_lm, k, v=None, want_scores=True, want_v_lm=True, ws=None, stream=None):
    """Returns (scores [B,H,M,N] fp32 or None, v_lm [B,H,M,d] or None)."""
    lib = load_library()
    dev = _dev(q_lm)
    S = torch.empty((cfg.B, cfg.H, cfg.M, cfg.N), dtype=torch.float32, device=dev) if want_scores else None
    v_lm = torch.empty((cfg.B, cfg.H, cfg.M, cfg.d), dtype=q_lm.dtype, device=dev) if want_v_lm else None
    ws, nws = _ws(cfg, WS_SCORES, ws, dev) if want_v_lm else (None, 0)
    _check(lib.mita_scores(ctypes.byref(cfg.struct()), _p(q_lm), _p(k), _p(v), _p(S), _p(v_lm), _p(ws), nws,
                           _stream(stream)))
    return S, v_lm


def topk(cfg: Config, S, idx=None, stream=None):
    lib = load_library()
    if idx is None:
        idx = torch.empty((cfg.B, cfg.H, cfg.M, cfg.k), dtype=torch.int32, device=_dev(S))
    _check(lib.mita_topk(ctypes.byref(cfg.struct()), _p(S), _p(idx), None, 0, _stream(stream)))
    return idx


def gather(cfg: Config, k, v, idx, stream=None):
    lib = load_library()
    shape = (cfg.B, cfg.H, cfg.M, cfg.k, cfg.d)
    kx = torch.empty(shape, dtype=k.dtype, device=_dev(k))
    vx = torch.empty(shape, dtype=v.dtype, device=_dev(v))
    _check(lib.mita_gather(ctypes.byref(cfg.struct()), _p(k), _p(v), _p(idx), _p(kx), _p(vx), _stream(stream)))
    return kx, vx


def route(cfg: Config, q, q_lm, ws=None, stream=None):
    """Returns (expert, perm, offsets) int32: with s = 1 expert [B,H,N],
    perm [B,H,N], offsets [B,H,M+1]; with s > 1 expert [B,H,N,s] (rank
    order), perm [B,H,N*s] (pair ids n*s+j grouped into 2M groups),
    offsets [B,H,2M+1]."""
    lib = load_library()
    dev = _dev(q)
    s = cfg.s if cfg.use_routed else 1
    G = 2 * cfg.M if s > 1 else cfg.M
    expert = torch.empty((cfg.B, cfg.H, cfg.N) + ((s,) if s > 1 else ()), dtype=torch.int32, device=dev)
    perm = torch.empty((cfg.B, cfg.H, cfg.N * s), dtype=torch.int32, device=dev)
    offsets = torch.empty((cfg.B, cfg.H, G + 1), dtype=torch.int32, device=dev)
    ws, nws = _ws(cfg, WS_ROUTE, ws, dev)
    _check(lib.mita_route(ctypes.byref(cfg.struct()), _p(q), _p(q_lm), _p(expert), _p(perm), _p(offsets), _p(ws),
                          nws, _stream(stream)))
    return expert, perm, offsets


def attend(cfg: Config, q, q_lm, v_lm, k_x, v_x, perm, offsets, o=None, ws=None, stream=None):
    lib = load_library()
    dev = _dev(q)
    if o is None:
        o = torch.empty_like(q)
    ws, nws = _ws(cfg, WS_ATTEND, ws, dev)
    _check(lib.mita_attend(ctypes.byref(cfg.struct()), _p(q), _p(q_lm), _p(v_lm), _p(k_x), _p(v_x), _p(perm),
                           _p(offsets), _p(o), _p(ws), nws, _stream(stream)))
    return o


class Timer:
    """HIP-event stage timer for mita_forward_timed."""

    def __init__(self, max_calls: int):
        self.lib = load_library()
        h = ctypes.c_void_p()
        _check(self.lib.mita_timer_create(ctypes.byref(h), int(max_calls)))
        self.handle = h
        self.max_calls = max_calls

    def reset(self):
        _check(self.lib.mita_timer_reset(self.handle))

    def launches(self):
        """Waits for the events; returns a list (one per call) of
        (kernel name, stage index, ms) tuples, one per kernel launched."""
        out = []
        n_calls = len(self.read())
        for c in range(n_calls):
            names = (ctypes.c_char_p * MAX_LAUNCHES)()
            stages = (ctypes.c_int32 * MAX_LAUNCHES)()
            ms = (ctypes.c_float * MAX_LAUNCHES)()
            n = ctypes.c_int32()
            _check(self.lib.mita_timer_launches(self.handle, c, MAX_LAUNCHES, names, stages, ms, ctypes.byref(n)))
            out.append([(names[i].decode(), stages[i], ms[i]) for i in range(n.value)])
        return out

    def read(self):
        """Waits for the events; returns a list (one per call) of per-stage ms
        lists (each stage the sum of its launches' times)."""
        n = ctypes.c_int()
        buf = (ctypes.c_float * (self.max_calls * NUM_STAGES))()
        _check(self.lib.mita_timer_read(self.handle, buf, len(buf), ctypes.byref(n)))
        return [[buf[c * NUM_STAGES + s] for s in range(NUM_STAGES)] for c in range(n.value)]

    def close(self):
        if self.handle:
            self.lib.mita_timer_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
