"""Python binding of libbkv.so, the MI355X (gfx950) BeaconKV eviction step.

Argument marshalling only: every step of the path runs in the HIP kernels
behind include/bkv.h.  torch supplies device memory and the stream (work is
enqueued on torch's current stream).  Tensor shapes, dtypes, devices and
contiguity are checked here because the C ABI takes bare pointers and
cannot see them.  There is no fallback: the library is loaded on first use,
and if it is not built that first use raises ImportError.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libbkv.so")
_lib = None

OK, ERR_INVALID, ERR_SHAPE, ERR_DTYPE, ERR_WORKSPACE, ERR_HIP, ERR_DEVICE = range(7)
F32, BF16 = 0, 1
OP_BEACON_UPDATE, OP_SCORE, OP_TOPK, OP_COMPACT, OP_EVICT = range(5)

EXPORTS = ("bkv_validate", "bkv_workspace_bytes", "bkv_workspace_init", "bkv_device_status",
           "bkv_beacon_update", "bkv_score", "bkv_topk", "bkv_compact", "bkv_evict",
           "bkv_score_ex", "bkv_evict_ex", "bkv_fps", "bkv_fps_gather", "bkv_status_string",
           "bkv_abi_version", "bkv_compact_fill", "bkv_evict_noalloc")
SCORE_MEAN, SCORE_CAUSAL = 1, 2


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("B", "Hq", "Hkv", "D", "N", "N_cap", "W", "C", "budget", "n_prefix", "dtype")]

    @property
    def G(self):
        return self.Hq // self.Hkv

    @property
    def P(self):
        return self.B * self.Hkv

    @property
    def n_keep(self):
        return min(self.budget, self.N)

    def replace(self, **kw):
        d = Dims()
        for n, _ in self._fields_:
            setattr(d, n, kw.get(n, getattr(self, n)))
        return d

    def __repr__(self):
        return "Dims(" + ", ".join(f"{n}={getattr(self, n)}" for n, _ in self._fields_) + ")"


def dims(B, Hq, Hkv, D, N, W, C, budget, n_prefix=0, dtype="bf16", N_cap=None) -> Dims:
    d = Dims()
    d.B, d.Hq, d.Hkv, d.D, d.N = B, Hq, Hkv, D, N
    d.N_cap = N if N_cap is None else N_cap
    d.W, d.C, d.budget, d.n_prefix = W, C, budget, n_prefix
    d.dtype = {"bf16": BF16, "fp32": F32, BF16: BF16, F32: F32}[dtype]
    return d


_P = ctypes.c_void_p
_D = ctypes.POINTER(Dims)
_S = ctypes.c_size_t
_I = ctypes.c_int32
_SIGS = {
    "bkv_validate": ([_D, ctypes.c_int32], ctypes.c_int),
    "bkv_workspace_bytes": ([_D, ctypes.c_int32], _S),
    "bkv_workspace_init": ([_D, _P, _S, _P], ctypes.c_int),
    "bkv_device_status": ([_P, _S, _P], ctypes.c_int),
    "bkv_beacon_update": ([_D, _P, ctypes.c_int32, _P, _P, _P, _P], ctypes.c_int),
    "bkv_score": ([_D, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _S, _P], ctypes.c_int),
    "bkv_topk": ([_D, _P, _P, _P, _S, _P], ctypes.c_int),
    "bkv_compact": ([_D, _P, _P, _P, _P, _S, _P], ctypes.c_int),
    "bkv_evict": ([_D, _P, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P, _S, _P], ctypes.c_int),
    "bkv_score_ex": ([_D, _I, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _S, _P], ctypes.c_int),
    "bkv_evict_ex": ([_D, _I, _P, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P, _S, _P], ctypes.c_int),
    "bkv_evict_noalloc": ([_D, _I, _P, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P, _P], ctypes.c_int),
    "bkv_fps": ([_I] * 5 + [_P, _I, _P, _P], ctypes.c_int),
    "bkv_fps_gather": ([_I] * 5 + [_P, _I, _P, _I, _I, _P, _P, _P], ctypes.c_int),
    "bkv_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "bkv_abi_version": ([], ctypes.c_int32),
}


def lib():
    """The loaded libbkv.so (loaded on first use; ImportError if not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_04971_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


class BkvError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


def status_string(st: int) -> str:
    return lib().bkv_status_string(st).decode()


def abi_version() -> int:
    return int(lib().bkv_abi_version())


def _check(st: int, where: str):
    if st != OK:
        raise BkvError(st, where)


def validate(d: Dims, op: int) -> int:
    """Host-only validation (no GPU needed); returns the bkv_status code."""
    return int(lib().bkv_validate(ctypes.byref(d), op))


def workspace_bytes(d: Dims, op: int = OP_EVICT) -> int:
    return int(lib().bkv_workspace_bytes(ctypes.byref(d), op))


# ---- marshalling helpers ---------------------------------------------------
def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _tdtype(d: Dims):
    return torch.bfloat16 if d.dtype == BF16 else torch.float32


def _ptr(t, shape=None, dtype=None, name="tensor", optional=False):
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _ws(ws):
    if ws is None:
        return None, 0
    if not isinstance(ws, torch.Tensor) or ws.device.type != "cuda" or not ws.is_contiguous():
        raise ValueError("workspace must be a contiguous CUDA tensor")
    return ctypes.c_void_p(ws.data_ptr()), ws.numel() * ws.element_size()


# ---- workspace -----------------------------------------------------------------
def workspace(d: Dims, op: int = OP_EVICT, device="cuda") -> torch.Tensor:
    """Allocate (through torch) and initialise a workspace for `op` on `d`."""
    n = workspace_bytes(d, op)
    ws = torch.empty(max(n, 256), dtype=torch.uint8, device=device)
    workspace_init(d, ws)
    return ws


def workspace_init(d: Dims, ws: torch.Tensor):
    p, n = _ws(ws)
    _check(lib().bkv_workspace_init(ctypes.byref(d), p, n, _stream()), "bkv_workspace_init")


def device_status(ws: torch.Tensor) -> int:
    """Synchronise the current stream and return the workspace's device status."""
    p, n = _ws(ws)
    return int(lib().bkv_device_status(p, n, _stream()))


# ---- operations ------------------------------------------------------------------
def beacon_update(d: Dims, q_new, beacons, counts, assign=None):
    """(a1) in place on beacons [B,Hkv,C,D] fp32 and counts [B,Hkv,C] int32."""
    T = q_new.shape[2]
    st = lib().bkv_beacon_update(
        ctypes.byref(d), _ptr(q_new, (d.B, d.Hq, T, d.D), _tdtype(d), "q_new"), T,
        _ptr(beacons, (d.B, d.Hkv, d.C, d.D), torch.float32, "beacons"),
        _ptr(counts, (d.B, d.Hkv, d.C), torch.int32, "counts"),
        _ptr(assign, (d.B, d.Hkv, T * d.G), torch.int32, "assign", optional=True), _stream())
    _check(st, "bkv_beacon_update")


def _rope(rope_cos, rope_sin, d):
    return (_ptr(rope_cos, (d.D // 2,), torch.float32, "rope_cos", optional=True),
            _ptr(rope_sin, (d.D // 2,), torch.float32, "rope_sin", optional=True))


def _flags(mean, causal):
    return (SCORE_MEAN if mean else 0) | (SCORE_CAUSAL if causal else 0)


def score(d: Dims, K, q_win, beacons, counts, scores, ws, row_lse=None, rope_cos=None, rope_sin=None,
          scale: float = 0.0, mean: bool = False, causal: bool = False):
    """(a2)+(a3): scores [B,Hkv,N] fp32 (and row_lse [B,Hkv,C+G*W]) written.
    mean / causal select the scoring options of bkv_score_ex."""
    rc, rs = _rope(rope_cos, rope_sin, d)
    wp, wn = _ws(ws)
    st = lib().bkv_score_ex(
        ctypes.byref(d), _flags(mean, causal), _ptr(K, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "K"),
        _ptr(q_win, (d.B, d.Hq, d.W, d.D), _tdtype(d), "q_win"),
        _ptr(beacons, (d.B, d.Hkv, d.C, d.D), torch.float32, "beacons"),
        _ptr(counts, (d.B, d.Hkv, d.C), torch.int32, "counts"), rc, rs, float(scale),
        _ptr(scores, (d.B, d.Hkv, d.N), torch.float32, "scores"),
        _ptr(row_lse, (d.B, d.Hkv, d.C + d.G * d.W), torch.float32, "row_lse", optional=True), wp, wn,
        _stream())
    _check(st, "bkv_score_ex")


def topk(d: Dims, scores, kept, ws=None):
    """(a4): kept [B,Hkv,min(budget,N)] int32 written, ascending."""
    wp, wn = _ws(ws)
    st = lib().bkv_topk(ctypes.byref(d), _ptr(scores, (d.B, d.Hkv, d.N), torch.float32, "scores"),
                       _ptr(kept, (d.B, d.Hkv, d.n_keep), torch.int32, "kept"), wp, wn, _stream())
    _check(st, "bkv_topk")


def compact(d: Dims, K, V, kept, ws):
    """(a5): rows i < n of K and V become rows kept[i], in place."""
    wp, wn = _ws(ws)
    st = lib().bkv_compact(ctypes.byref(d), _ptr(K, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "K"),
                          _ptr(V, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "V"),
                          _ptr(kept, (d.B, d.Hkv, d.n_keep), torch.int32, "kept"), wp, wn, _stream())
    _check(st, "bkv_compact")


def compact_fill(d: Dims, K, V, kept, src_of, ws):
    """Hole-filling compaction in place: kept rows below n stay, the holes
    below n take the kept rows past n; src_of [B,Hkv,n] int32 receives the
    old row now at each row."""
    wp, wn = _ws(ws)
    st = lib().bkv_compact_fill(ctypes.byref(d), _ptr(K, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "K"),
                                _ptr(V, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "V"),
                                _ptr(kept, (d.B, d.Hkv, d.n_keep), torch.int32, "kept"),
                                _ptr(src_of, (d.B, d.Hkv, d.n_keep), torch.int32, "src_of"), wp, wn, _stream())
    _check(st, "bkv_compact_fill")


def evict(d: Dims, K, V, q_win, beacons, counts, ws, kept=None, scores=None, row_lse=None, rope_cos=None,
          rope_sin=None, scale: float = 0.0, mean: bool = False, causal: bool = False):
    """(a6): score -> select -> compact one layer in place (scoring options
    as in score)."""
    rc, rs = _rope(rope_cos, rope_sin, d)
    wp, wn = _ws(ws)
    st = lib().bkv_evict_ex(
        ctypes.byref(d), _flags(mean, causal), _ptr(K, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "K"),
        _ptr(V, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "V"),
        _ptr(q_win, (d.B, d.Hq, d.W, d.D), _tdtype(d), "q_win"),
        _ptr(beacons, (d.B, d.Hkv, d.C, d.D), torch.float32, "beacons"),
        _ptr(counts, (d.B, d.Hkv, d.C), torch.int32, "counts"), rc, rs, float(scale),
        _ptr(kept, (d.B, d.Hkv, d.n_keep), torch.int32, "kept", optional=True),
        _ptr(scores, (d.B, d.Hkv, d.N), torch.float32, "scores", optional=True),
        _ptr(row_lse, (d.B, d.Hkv, d.C + d.G * d.W), torch.float32, "row_lse", optional=True), wp, wn,
        _stream())
    _check(st, "bkv_evict_ex")


def evict_noalloc(d: Dims, K, V, q_win, beacons, counts, kept=None, scores=None, row_lse=None, rope_cos=None,
                  rope_sin=None, scale: float = 0.0, mean: bool = False, causal: bool = False, status=None):
    """evict() with the library's fixed device array as its workspace: no
    workspace argument, nothing allocated.  status, an optional int32 tensor
    of one element, receives the call's device status (OK or ERR_DEVICE)."""
    rc, rs = _rope(rope_cos, rope_sin, d)
    st = lib().bkv_evict_noalloc(
        ctypes.byref(d), _flags(mean, causal), _ptr(K, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "K"),
        _ptr(V, (d.B, d.Hkv, d.N_cap, d.D), _tdtype(d), "V"),
        _ptr(q_win, (d.B, d.Hq, d.W, d.D), _tdtype(d), "q_win"),
        _ptr(beacons, (d.B, d.Hkv, d.C, d.D), torch.float32, "beacons"),
        _ptr(counts, (d.B, d.Hkv, d.C), torch.int32, "counts"), rc, rs, float(scale),
        _ptr(kept, (d.B, d.Hkv, d.n_keep), torch.int32, "kept", optional=True),
        _ptr(scores, (d.B, d.Hkv, d.N), torch.float32, "scores", optional=True),
        _ptr(row_lse, (d.B, d.Hkv, d.C + d.G * d.W), torch.float32, "row_lse", optional=True),
        _ptr(status, (1,), torch.int32, "status", optional=True), _stream())
    _check(st, "bkv_evict_noalloc")


# ---- Continual FPS -------------------------------------------------------------
_FPS_DT = {torch.bfloat16: BF16, torch.float32: F32}


def _fps_src(q, n, name):
    if not isinstance(q, torch.Tensor) or q.dim() < 2:
        raise ValueError(f"{name} must be a tensor [..., rows, D]")
    if q.dtype not in _FPS_DT:
        raise ValueError(f"{name} must be bfloat16 or float32, got {q.dtype}")
    rows, D = q.shape[-2], q.shape[-1]
    H = q.numel() // max(1, rows * D) if rows * D else 0
    n = rows if n is None else int(n)
    return _ptr(q, name=name), H, rows, D, n


def fps(q, m: int, n: int | None = None, picks=None):
    """Farthest point sampling (Appendix D.1, Algorithm 1) of the first n rows
    (default: all) of every head of q [..., rows, D]: returns picks
    [..., min(m, n)] int32 in selection order."""
    qp, H, rows, D, n = _fps_src(q, n, "q")
    k = max(0, min(int(m), n))
    shape = tuple(q.shape[:-2]) + (k,)
    if picks is None:
        picks = torch.empty(shape, dtype=torch.int32, device=q.device)
    pp = _ptr(picks, shape, torch.int32, "picks")
    _check(lib().bkv_fps(H, n, int(m), D, _FPS_DT[q.dtype], qp, rows, pp, _stream()), "bkv_fps")
    return picks


def fps_gather(src, m: int, dst=None, n: int | None = None, picks=None, counts=None):
    """FPS of the first n rows of every head of src [..., rows, D], then rows
    0..k-1 of dst [..., dst_rows, D] (default: src itself, in place) become
    the picked rows in selection order, k = min(m, n) (Section 4.2, Eq.
    fps_q).  dst may be float32 for a bfloat16 src.  picks [..., k] and
    counts [..., dst_rows] are optional outputs.  Returns dst."""
    sp, H, rows, D, n = _fps_src(src, n, "src")
    k = max(0, min(int(m), n))
    if dst is None:
        dst = src
    if dst.dtype not in _FPS_DT or dst.dim() != src.dim() or dst.shape[:-2] != src.shape[:-2] \
            or dst.shape[-1] != D:
        raise ValueError("dst must be [..., dst_rows, D] with the leading shape and D of src")
    dst_rows = dst.shape[-2]
    lead = tuple(src.shape[:-2])
    pp = _ptr(picks, lead + (k,), torch.int32, "picks", optional=True)
    cp = _ptr(counts, lead + (dst_rows,), torch.int32, "counts", optional=True)
    st = lib().bkv_fps_gather(H, n, int(m), D, _FPS_DT[src.dtype], sp, rows, _ptr(dst, name="dst"),
                              _FPS_DT[dst.dtype], dst_rows, pp, cp, _stream())
    _check(st, "bkv_fps_gather")
    return dst
