"""Python binding of libwavezip.so (argument marshalling only).

Every call forwards torch device tensors' pointers and the current HIP stream
to the C ABI declared in include/wavezip.h; all computation happens in the
library's gfx950 kernels.  If the library is missing this module raises
instead of falling back to anything else: build it with
`python -m paper_2607_23265_amd.csrc.build`.
"""
import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwavezip.so")

WZ_F32, WZ_BF16 = 0, 1
WZ_SELECT, WZ_INTERP = 0, 1
WZ_HAAR, WZ_DB4, WZ_BIOR44 = 0, 1, 2
BASIS = {"haar": WZ_HAAR, "db4": WZ_DB4, "bior4.4": WZ_BIOR44}
_STATUS = {0: "WZ_OK", 1: "WZ_ERR_NULL", 2: "WZ_ERR_ALIGN", 3: "WZ_ERR_SHAPE", 4: "WZ_ERR_DTYPE",
           5: "WZ_ERR_PARAM", 6: "WZ_ERR_BUDGET", 7: "WZ_ERR_WORKSPACE", 8: "WZ_ERR_DEVICE",
           9: "WZ_ERR_SCRATCH"}
EXPORTS = ("wz_workspace_bytes", "wz_relevance", "wz_relevance_pass", "wz_temporal_budget",
           "wz_spatial_dwt_condense", "wz_condense", "wz_condense_batch", "wz_condense_queries",
           "wz_condense_noalloc", "wz_noalloc_scratch_bytes", "wz_status_str", "wz_probe_stream_read")


class WZError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {_STATUS.get(status, status)}")


class Config(ctypes.Structure):
    """Mirror of wz_config."""
    _fields_ = [("T", ctypes.c_int32), ("H", ctypes.c_int32), ("W", ctypes.c_int32),
                ("C", ctypes.c_int32), ("Q", ctypes.c_int32), ("in_dtype", ctypes.c_int32),
                ("out_dtype", ctypes.c_int32), ("levels", ctypes.c_int32), ("B", ctypes.c_int64),
                ("lambda_", ctypes.c_float), ("tau", ctypes.c_float), ("assign", ctypes.c_int32),
                ("spatial_levels", ctypes.c_int32), ("temporal_basis", ctypes.c_int32),
                ("spatial_basis", ctypes.c_int32)]


_lib = None


def lib():
    """Load libwavezip.so (once) and declare its entry points."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing; build it with `python -m paper_2607_23265_amd.csrc.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, S = ctypes.c_void_p, ctypes.c_size_t
    cfgp = ctypes.POINTER(Config)
    L.wz_workspace_bytes.argtypes = [cfgp]
    L.wz_workspace_bytes.restype = S
    L.wz_relevance.argtypes = [cfgp, P, P, P, P, P, P, S, P]
    L.wz_relevance_pass.argtypes = [cfgp, P, P, P, P, S, P]
    L.wz_condense_batch.argtypes = [cfgp, ctypes.c_int32, P, P, P, P, P, P, P, S, P]
    L.wz_condense_queries.argtypes = [cfgp, ctypes.c_int32, P, P, P, P, P, P, P, S, P]
    L.wz_temporal_budget.argtypes = [cfgp, P, P, P, P, P, P]
    L.wz_spatial_dwt_condense.argtypes = [cfgp, P, P, P, P, P, P]
    L.wz_condense.argtypes = [cfgp, P, P, P, P, P, P, P, S, P]
    L.wz_condense_noalloc.argtypes = [cfgp, P, P, P, P, P, P, P]
    L.wz_probe_stream_read.argtypes = [P, S, P, P]
    L.wz_probe_stream_read.restype = ctypes.c_int
    L.wz_noalloc_scratch_bytes.argtypes = []
    L.wz_noalloc_scratch_bytes.restype = S
    for f in ("wz_relevance", "wz_relevance_pass", "wz_temporal_budget", "wz_spatial_dwt_condense", "wz_condense",
              "wz_condense_batch", "wz_condense_queries", "wz_condense_noalloc"):
        getattr(L, f).restype = ctypes.c_int
    L.wz_status_str.argtypes = [ctypes.c_int]
    L.wz_status_str.restype = ctypes.c_char_p
    _lib = L
    return L


@dataclass
class Problem:
    T: int
    H: int
    W: int
    C: int
    Q: int
    B: int
    in_dtype: int = WZ_BF16
    out_dtype: int = WZ_F32
    levels: int = 1
    lam: float = 1.5
    tau: float = 0.0
    assign: int = 0  # WZ_SELECT; WZ_INTERP for the budget-guided interpolation
    spatial_levels: int = 1  # 2: the two-level spatial modulator (selection only)
    temporal_basis: int = WZ_HAAR  # WZ_DB4 / WZ_BIOR44: filter bank of the temporal allocator
    spatial_basis: int = WZ_HAAR   # WZ_DB4 / WZ_BIOR44: filter bank of the spatial modulator

    def config(self):
        return Config(self.T, self.H, self.W, self.C, self.Q, self.in_dtype, self.out_dtype, self.levels,
                      self.B, self.lam, self.tau, self.assign, self.spatial_levels, self.temporal_basis,
                      self.spatial_basis)

    @property
    def N(self):
        return self.H * self.W


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check(st, where):
    if st != 0:
        raise WZError(st, where)


def _require_device(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("arguments must be contiguous GPU tensors")


def workspace_bytes(p: Problem):
    return int(lib().wz_workspace_bytes(ctypes.byref(p.config())))


def new_workspace(p: Problem, device):
    """A workspace for `p` (its contents on entry are ignored by the library)."""
    n = workspace_bytes(p)
    if n == 0:
        raise WZError(3, "wz_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def relevance(p: Problem, X, query, ws=None):
    """wz_relevance -> (tok_score [T*N], frame_rel [T], frame_delta [T]) float32."""
    _require_device(X, query)
    dev = X.device
    ws = new_workspace(p, dev) if ws is None else ws
    a = torch.empty(p.T * p.N, dtype=torch.float32, device=dev)
    r = torch.empty(p.T, dtype=torch.float32, device=dev)
    d = torch.empty(p.T, dtype=torch.float32, device=dev)
    cfg = p.config()
    _check(lib().wz_relevance(ctypes.byref(cfg), _ptr(X), _ptr(query), _ptr(a), _ptr(r), _ptr(d), _ptr(ws),
                              ws.numel(), _stream(dev)), "wz_relevance")
    return a, r, d


def relevance_pass(p: Problem, X, query, tok_score, ws):
    """wz_relevance_pass: the pass over X alone, into caller-owned tok_score and ws."""
    _require_device(X, query, tok_score, ws)
    cfg = p.config()
    _check(lib().wz_relevance_pass(ctypes.byref(cfg), _ptr(X), _ptr(query), _ptr(tok_score), _ptr(ws),
                                   ws.numel(), _stream(X.device)), "wz_relevance_pass")


def temporal_budget(p: Problem, frame_rel, frame_delta):
    """wz_temporal_budget -> (budget [T] int32, offset [T+1] int32, rel_rect [T] float32)."""
    _require_device(frame_rel, frame_delta)
    dev = frame_rel.device
    b = torch.empty(p.T, dtype=torch.int32, device=dev)
    o = torch.empty(p.T + 1, dtype=torch.int32, device=dev)
    rr = torch.empty(p.T, dtype=torch.float32, device=dev)
    cfg = p.config()
    _check(lib().wz_temporal_budget(ctypes.byref(cfg), _ptr(frame_rel), _ptr(frame_delta), _ptr(b), _ptr(o),
                                    _ptr(rr), _stream(dev)), "wz_temporal_budget")
    return b, o, rr


def _out_tokens(p: Problem, dev):
    dt = torch.float32 if p.out_dtype == WZ_F32 else torch.bfloat16
    return torch.empty((max(p.B, 1), p.C), dtype=dt, device=dev), torch.empty(max(p.B, 1), dtype=torch.int32,
                                                                               device=dev)


def spatial_dwt_condense(p: Problem, X, tok_score, offset):
    """wz_spatial_dwt_condense -> (tokens [B, C], index [B]); rows from offset[T] on are unwritten."""
    _require_device(X, tok_score, offset)
    dev = X.device
    tok, idx = _out_tokens(p, dev)
    cfg = p.config()
    _check(lib().wz_spatial_dwt_condense(ctypes.byref(cfg), _ptr(X), _ptr(tok_score), _ptr(offset), _ptr(tok),
                                         _ptr(idx), _stream(dev)),
           "wz_spatial_dwt_condense")
    return tok, idx


def condense(p: Problem, X, query, ws=None, out=None):
    """wz_condense -> (tokens [B, C], index [B], budget [T], offset [T+1])."""
    _require_device(X, query)
    dev = X.device
    ws = new_workspace(p, dev) if ws is None else ws
    tok, idx = _out_tokens(p, dev) if out is None else out
    b = torch.empty(p.T, dtype=torch.int32, device=dev)
    o = torch.empty(p.T + 1, dtype=torch.int32, device=dev)
    cfg = p.config()
    _check(lib().wz_condense(ctypes.byref(cfg), _ptr(X), _ptr(query), _ptr(tok), _ptr(idx), _ptr(b), _ptr(o),
                             _ptr(ws), ws.numel(), _stream(dev)), "wz_condense")
    return tok, idx, b, o


def condense_noalloc(p: Problem, X, query, out=None):
    """wz_condense_noalloc (no workspace: the library's static scratch) -> (tokens, index, budget, offset)."""
    _require_device(X, query)
    dev = X.device
    tok, idx = _out_tokens(p, dev) if out is None else out
    b = torch.empty(p.T, dtype=torch.int32, device=dev)
    o = torch.empty(p.T + 1, dtype=torch.int32, device=dev)
    cfg = p.config()
    _check(lib().wz_condense_noalloc(ctypes.byref(cfg), _ptr(X), _ptr(query), _ptr(tok), _ptr(idx), _ptr(b), _ptr(o),
                                     _stream(dev)), "wz_condense_noalloc")
    return tok, idx, b, o


def probe_stream_read(data, sink):
    """wz_probe_stream_read: one plain streaming read of a device tensor (a measurement aid)."""
    _require_device(data, sink)
    _check(lib().wz_probe_stream_read(_ptr(data), data.numel() * data.element_size(), _ptr(sink), _stream(data.device)),
           "wz_probe_stream_read")


def condense_batch(p: Problem, X, query, ws=None, out=None):
    """wz_condense_batch over V videos: X [V, T, H, W, C], query [V, Q, C] ->
    (tokens [V, B, C], index [V, B], budget [V, T], offset [V, T+1])."""
    _require_device(X, query)
    dev = X.device
    V = X.shape[0]
    ws = torch.empty(V * workspace_bytes(p), dtype=torch.uint8, device=dev) if ws is None else ws
    dt = torch.float32 if p.out_dtype == WZ_F32 else torch.bfloat16
    if out is None:
        out = (torch.empty((V, max(p.B, 1), p.C), dtype=dt, device=dev),
               torch.empty((V, max(p.B, 1)), dtype=torch.int32, device=dev))
    tok, idx = out
    b = torch.empty((V, p.T), dtype=torch.int32, device=dev)
    o = torch.empty((V, p.T + 1), dtype=torch.int32, device=dev)
    cfg = p.config()
    _check(lib().wz_condense_batch(ctypes.byref(cfg), V, _ptr(X), _ptr(query), _ptr(tok), _ptr(idx), _ptr(b),
                                   _ptr(o), _ptr(ws), ws.numel(), _stream(dev)), "wz_condense_batch")
    return tok, idx, b, o


def condense_queries(p: Problem, X, query, ws=None, out=None):
    """wz_condense_queries: G queries over one video, X [T, H, W, C], query [G, Q, C] ->
    (tokens [G, B, C], index [G, B], budget [G, T], offset [G, T+1])."""
    _require_device(X, query)
    dev = X.device
    G = query.shape[0]
    ws = torch.empty(G * workspace_bytes(p), dtype=torch.uint8, device=dev) if ws is None else ws
    dt = torch.float32 if p.out_dtype == WZ_F32 else torch.bfloat16
    if out is None:
        out = (torch.empty((G, max(p.B, 1), p.C), dtype=dt, device=dev),
               torch.empty((G, max(p.B, 1)), dtype=torch.int32, device=dev))
    tok, idx = out
    b = torch.empty((G, p.T), dtype=torch.int32, device=dev)
    o = torch.empty((G, p.T + 1), dtype=torch.int32, device=dev)
    cfg = p.config()
    _check(lib().wz_condense_queries(ctypes.byref(cfg), G, _ptr(X), _ptr(query), _ptr(tok), _ptr(idx), _ptr(b),
                                     _ptr(o), _ptr(ws), ws.numel(), _stream(dev)), "wz_condense_queries")
    return tok, idx, b, o


def to_device(inp, device="cuda:0"):
    """Move a generated input set (paper_2607_23265_amd.synth.Inputs) to the GPU."""
    if inp.wl.dtype == "bf16":
        X = torch.from_numpy(inp.X.view("int16")).to(device).view(torch.bfloat16)
        q = torch.from_numpy(inp.query.view("int16")).to(device).view(torch.bfloat16)
    else:
        X = torch.from_numpy(inp.X).to(device)
        q = torch.from_numpy(inp.query).to(device)
    return X.contiguous(), q.contiguous()


def problem_of(wl, out_dtype=WZ_F32, assign=0, spatial_levels=1, temporal_basis=WZ_HAAR, spatial_basis=WZ_HAAR):
    """Problem description of a workload (paper_2607_23265_amd.synth.Workload)."""
    return Problem(T=wl.T, H=wl.H, W=wl.W, C=wl.C, Q=wl.Q, B=wl.B,
                   in_dtype=WZ_BF16 if wl.dtype == "bf16" else WZ_F32, out_dtype=out_dtype,
                   levels=wl.levels, lam=wl.lam, tau=wl.tau, assign=assign, spatial_levels=spatial_levels,
                   temporal_basis=temporal_basis, spatial_basis=spatial_basis)
