"""CPU oracle of the BeaconKV eviction step -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may
import this package.  The GPU library never does; the two share no code.

The arithmetic lives in bkv_oracle.c (plain C, double precision, one
function per step of the method, each citing the passage it follows).
This module only marshals whole tensors into per-(batch, kv-head) calls:

  * a bf16 tensor is handed over as its raw 16-bit patterns, fp32 as is;
  * kv-head h owns query heads h*G .. h*G+G-1 (contiguous GQA grouping),
    which are contiguous in a [B, Hq, T, D] tensor;
  * heads are independent, so a thread pool may run them side by side
    (ctypes releases the GIL during each call).

Inputs may be numpy arrays or CPU torch tensors (bf16 or fp32).
"""
from __future__ import annotations

import ctypes
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

F32, BF16 = 0, 1

_p = ctypes.c_void_p
_i = ctypes.c_int
_f = ctypes.c_float


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from oracle.build import build  # build only when nothing is built yet
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.orc_beacon_update.argtypes = [_i, _i, _i, _i, _i, _p, _p, _p, _p, _p]
    lib.orc_beacon_update.restype = _i
    lib.orc_rope_row.argtypes = [_i, _p, _p, _p, _i, _p]
    lib.orc_rope_row.restype = None
    lib.orc_assemble_rows.argtypes = [_i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _p]
    lib.orc_assemble_rows.restype = _i
    lib.orc_score.argtypes = [_i, _i, _i, _p, _p, _i, ctypes.c_double, _p, _p]
    lib.orc_score.restype = _i
    lib.orc_score_head.argtypes = [_i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _f, _p, _p]
    lib.orc_score_head.restype = _i
    lib.orc_topk.argtypes = [_i, _p, _i, _i, _i, _p]
    lib.orc_topk.restype = _i
    lib.orc_compact.argtypes = [_i, _i, _i, _p, _p, _p]
    lib.orc_compact.restype = _i
    lib.orc_compact_fill.argtypes = [_i, _i, _i, _i, _p, _p, _p, _p]
    lib.orc_compact_fill.restype = _i
    lib.orc_fps.argtypes = [_i, _i, _i, _i, _p, _p, ctypes.c_double, _p, _p]
    lib.orc_fps.restype = _i
    lib.orc_evict_head.argtypes = [_i, _i, _i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p,
                                   _p, _f, _p, _p, _p]
    lib.orc_evict_head.restype = _i
    lib.orc_score_ex.argtypes = [_i, _i, _i, _p, _p, _i, ctypes.c_double, _i, _p, _p, _p]
    lib.orc_score_ex.restype = _i
    lib.orc_score_head_ex.argtypes = [_i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _f, _i, _i, _p, _p]
    lib.orc_score_head_ex.restype = _i
    lib.orc_evict_head_ex.argtypes = [_i, _i, _i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p,
                                      _p, _f, _i, _i, _p, _p, _p]
    lib.orc_evict_head_ex.restype = _i
    _lib = lib
    return lib


def _raw(x):
    """Return (contiguous numpy array, dtype code) for a bf16/fp32 tensor."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().contiguous()
            if x.dtype == torch.bfloat16:
                return x.view(torch.int16).numpy().view(np.uint16), BF16
            if x.dtype == torch.float32:
                return x.numpy(), F32
            if x.dtype == torch.int32:
                return x.numpy(), None
            raise TypeError(f"oracle: unsupported tensor dtype {x.dtype}")
    except ImportError:
        pass
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return x, BF16
    if x.dtype == np.float32:
        return x, F32
    if x.dtype == np.int32:
        return x, None
    if x.dtype == np.float64:
        return x.astype(np.float32), F32
    raise TypeError(f"oracle: unsupported array dtype {x.dtype}")


def _ptr(a: np.ndarray, offset_elems: int = 0):
    return ctypes.c_void_p(a.ctypes.data + offset_elems * a.itemsize)


def _run(fn, items, threads):
    if threads <= 1:
        return [fn(it) for it in items]
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(fn, items))


# ---------------------------------------------------------------------------
def beacon_update(q_new, beacons, counts, Hkv: int, threads: int = 1):
    """(a1) for every (b, kv-head): q_new [B,Hq,T,D] (bf16 or fp32) pre-RoPE,
    beacons [B,Hkv,C,D] fp32, counts [B,Hkv,C] int32.  Returns a dict with the
    updated beacons and counts (copies), the chosen slot of every query
    (assign [B,Hkv,T*G], order t-major then g) and the near-tie flags."""
    lib = _load()
    q, dt = _raw(q_new)
    B, Hq, T, D = q.shape
    G = Hq // Hkv
    bc = np.array(_raw(beacons)[0], dtype=np.float32, copy=True)
    cn = np.array(_raw(counts)[0], dtype=np.int32, copy=True)
    C = bc.shape[2]
    assign = np.zeros((B, Hkv, T * G), np.int32)
    tie = np.zeros((B, Hkv, T * G), np.int32)

    def one(bh):
        b, h = bh
        rc = lib.orc_beacon_update(dt, D, C, G, T, _ptr(q, ((b * Hq) + h * G) * T * D),
                                   _ptr(bc, (b * Hkv + h) * C * D), _ptr(cn, (b * Hkv + h) * C),
                                   _ptr(assign, (b * Hkv + h) * T * G),
                                   _ptr(tie, (b * Hkv + h) * T * G))
        if rc:
            raise RuntimeError(f"orc_beacon_update failed ({rc})")

    _run(one, [(b, h) for b in range(B) for h in range(Hkv)], threads)
    return {"beacons": bc, "counts": cn, "assign": assign, "near_tie": tie.astype(bool)}


def rope_row(beta, cos_t=None, sin_t=None, to_bf16: bool = False):
    """(a2) one fp32 row rotated by the step's cos/sin table (rotate-half)."""
    lib = _load()
    b = np.ascontiguousarray(beta, dtype=np.float32)
    D = b.shape[0]
    out = np.zeros(D, np.float32)
    c = None if cos_t is None else np.ascontiguousarray(cos_t, dtype=np.float32)
    s = None if sin_t is None else np.ascontiguousarray(sin_t, dtype=np.float32)
    lib.orc_rope_row(D, _ptr(b), None if c is None else _ptr(c), None if s is None else _ptr(s),
                     int(to_bf16), _ptr(out))
    return out


_AGG = {"max": 0, "mean": 1}


def score_rows(Y, Khead, scale: float, agg: str = "max", limit=None):
    """(a3) on explicit float64 rows Y [R,D] and keys Khead [N,D] (fp32 or
    bf16 raw); returns (lse [R], s [N]).  agg "mean" takes Eq. (6)'s mean
    form; limit [R] (optional) lets row r see keys j <= limit[r] only."""
    lib = _load()
    Yd = np.ascontiguousarray(Y, dtype=np.float64)
    k, dt = _raw(Khead)
    R = Yd.shape[0]
    N, D = k.shape
    lse = np.zeros(max(R, 1), np.float64)
    s = np.zeros(max(N, 1), np.float64)
    lim = None if limit is None else np.ascontiguousarray(limit, dtype=np.int32)
    rc = lib.orc_score_ex(R, N, D, _ptr(Yd), _ptr(k), dt, float(scale), _AGG[agg],
                          None if lim is None else _ptr(lim), _ptr(lse), _ptr(s))
    if rc:
        raise RuntimeError(f"orc_score failed ({rc})")
    return lse[:R], s[:N]


def score(K, q_win, beacons, counts, N: int, rope_cos=None, rope_sin=None, scale: float = 0.0,
          heads=None, threads: int = 1, agg: str = "max", causal: bool = False):
    """(a2)+(a3) for every (b, kv-head) or the listed `heads` [(b, h), ...].
    K [B,Hkv,N_cap,D], q_win [B,Hq,W,D] post-RoPE, beacons [B,Hkv,C,D] fp32,
    counts [B,Hkv,C].  Returns (scores [B,Hkv,N] float64, row_lse
    [B,Hkv,C+G*W] float64, slot-indexed, -inf for empty beacon slots); heads
    not listed read NaN."""
    lib = _load()
    k, dt = _raw(K)
    qw, dq = _raw(q_win)
    if dq != dt:
        raise TypeError("oracle: K and q_win must share a dtype")
    bc = np.ascontiguousarray(_raw(beacons)[0], dtype=np.float32)
    cn = np.ascontiguousarray(_raw(counts)[0], dtype=np.int32)
    B, Hkv, Ncap, D = k.shape
    Hq, W = qw.shape[1], qw.shape[2]
    G = Hq // Hkv
    C = bc.shape[2]
    cs = None if rope_cos is None else np.ascontiguousarray(rope_cos, dtype=np.float32)
    sn = None if rope_sin is None else np.ascontiguousarray(rope_sin, dtype=np.float32)
    scores = np.full((B, Hkv, N), np.nan)
    lse = np.full((B, Hkv, C + G * W), np.nan)
    if heads is None:
        heads = [(b, h) for b in range(B) for h in range(Hkv)]

    def one(bh):
        b, h = bh
        s_h = np.zeros(max(N, 1), np.float64)
        l_h = np.zeros(max(C + G * W, 1), np.float64)
        rc = lib.orc_score_head_ex(dt, D, N, C, G, W, _ptr(k, (b * Hkv + h) * Ncap * D),
                                   _ptr(qw, (b * Hq + h * G) * W * D), _ptr(bc, (b * Hkv + h) * C * D),
                                   _ptr(cn, (b * Hkv + h) * C), None if cs is None else _ptr(cs),
                                   None if sn is None else _ptr(sn), float(scale), _AGG[agg], int(bool(causal)),
                                   _ptr(l_h), _ptr(s_h))
        if rc:
            raise RuntimeError(f"orc_score_head failed ({rc})")
        scores[b, h] = s_h[:N]
        lse[b, h] = l_h[:C + G * W]

    _run(one, list(heads), threads)
    return scores, lse


def topk_head(s, budget: int, W: int, n_prefix: int):
    """(a4) on one head's scores (float64 vector); returns kept (int32)."""
    lib = _load()
    sv = np.ascontiguousarray(s, dtype=np.float64)
    N = sv.shape[0]
    kept = np.zeros(max(min(budget, N), 1), np.int32)
    n = lib.orc_topk(N, _ptr(sv), budget, W, n_prefix, _ptr(kept))
    if n < 0:
        raise RuntimeError(f"orc_topk failed ({n})")
    return kept[:n]


def topk(scores, budget: int, W: int, n_prefix: int = 0):
    """(a4) for every head of scores [B,Hkv,N]; returns kept [B,Hkv,min(budget,N)]."""
    s = np.asarray(scores, dtype=np.float64)
    B, Hkv, N = s.shape
    out = np.zeros((B, Hkv, min(budget, N)), np.int32)
    for b in range(B):
        for h in range(Hkv):
            out[b, h] = topk_head(s[b, h], budget, W, n_prefix)
    return out


def compact(K, V, kept):
    """(a5) on copies of K and V [B,Hkv,N_cap,D] with kept [B,Hkv,n];
    returns (K', V') as raw numpy arrays of the input's storage type."""
    lib = _load()
    k, dt = _raw(K)
    v, dv = _raw(V)
    k = k.copy()
    v = v.copy()
    kp = np.ascontiguousarray(kept, dtype=np.int32)
    B, Hkv, Ncap, D = k.shape
    n = kp.shape[2]
    es = 2 if dt == BF16 else 4
    for b in range(B):
        for h in range(Hkv):
            rc = lib.orc_compact(es, D, n, _ptr(kp, (b * Hkv + h) * n), _ptr(k, (b * Hkv + h) * Ncap * D),
                                 _ptr(v, (b * Hkv + h) * Ncap * D))
            if rc:
                raise RuntimeError(f"orc_compact failed ({rc})")
    return k, v


def compact_fill(K, V, kept, N: int):
    """Hole-filling compaction on copies of K and V [B,Hkv,N_cap,D] with
    kept [B,Hkv,n]: kept rows below n stay, the holes below n take the kept
    rows at or above n in ascending order.  Returns (K', V' raw numpy,
    src_of [B,Hkv,n] int32, moved [B,Hkv] rows moved)."""
    lib = _load()
    k, dt = _raw(K)
    v, _ = _raw(V)
    k = k.copy()
    v = v.copy()
    kp = np.ascontiguousarray(kept, dtype=np.int32)
    B, Hkv, Ncap, D = k.shape
    n = kp.shape[2]
    es = 2 if dt == BF16 else 4
    src_of = np.empty((B, Hkv, n), np.int32)
    moved = np.empty((B, Hkv), np.int64)
    for b in range(B):
        for h in range(Hkv):
            rc = lib.orc_compact_fill(es, D, N, n, _ptr(kp, (b * Hkv + h) * n), _ptr(k, (b * Hkv + h) * Ncap * D),
                                      _ptr(v, (b * Hkv + h) * Ncap * D), _ptr(src_of, (b * Hkv + h) * n))
            if rc < 0:
                raise RuntimeError(f"orc_compact_fill failed ({rc})")
            moved[b, h] = rc
    return k, v, src_of, moved


def evict(K, V, q_win, beacons, counts, N: int, budget: int, W: int, n_prefix: int = 0,
          rope_cos=None, rope_sin=None, scale: float = 0.0, heads=None, threads: int = 1, agg: str = "max",
          causal: bool = False):
    """(a6) = (a2)->(a5) for every head or the listed `heads`, on copies.
    Returns dict(K, V (raw numpy, compacted), scores, row_lse, kept); heads
    not listed keep their input rows and read NaN / -1."""
    lib = _load()
    k, dt = _raw(K)
    v, _ = _raw(V)
    k = k.copy()
    v = v.copy()
    qw, _ = _raw(q_win)
    bc = np.ascontiguousarray(_raw(beacons)[0], dtype=np.float32)
    cn = np.ascontiguousarray(_raw(counts)[0], dtype=np.int32)
    B, Hkv, Ncap, D = k.shape
    Hq = qw.shape[1]
    G = Hq // Hkv
    C = bc.shape[2]
    cs = None if rope_cos is None else np.ascontiguousarray(rope_cos, dtype=np.float32)
    sn = None if rope_sin is None else np.ascontiguousarray(rope_sin, dtype=np.float32)
    nk = min(budget, N)
    scores = np.full((B, Hkv, N), np.nan)
    lse = np.full((B, Hkv, C + G * W), np.nan)
    kept = np.full((B, Hkv, nk), -1, np.int32)
    if heads is None:
        heads = [(b, h) for b in range(B) for h in range(Hkv)]

    def one(bh):
        b, h = bh
        s_h = np.zeros(max(N, 1), np.float64)
        l_h = np.zeros(max(C + G * W, 1), np.float64)
        kp = np.zeros(max(nk, 1), np.int32)
        n = lib.orc_evict_head_ex(dt, D, N, C, G, W, budget, n_prefix,
                                  _ptr(k, (b * Hkv + h) * Ncap * D), _ptr(v, (b * Hkv + h) * Ncap * D),
                                  _ptr(qw, (b * Hq + h * G) * W * D), _ptr(bc, (b * Hkv + h) * C * D),
                                  _ptr(cn, (b * Hkv + h) * C), None if cs is None else _ptr(cs),
                                  None if sn is None else _ptr(sn), float(scale), _AGG[agg], int(bool(causal)),
                                  _ptr(l_h), _ptr(s_h), _ptr(kp))
        if n < 0:
            raise RuntimeError(f"orc_evict_head failed ({n})")
        scores[b, h] = s_h[:N]
        lse[b, h] = l_h[:C + G * W]
        kept[b, h] = kp[:nk]

    _run(one, list(heads), threads)
    return {"K": k, "V": v, "scores": scores, "row_lse": lse, "kept": kept}


def fps(q, m: int, forced=None, tie_tol: float = 0.0, threads: int = 1):
    """Farthest point sampling (Appendix D.1, Algorithm 1) of every head of
    q [H, n, D] (bf16 or fp32): returns (picks [H, min(m, n)] int32 in
    selection order, near_tie [H, min(m, n)] bool).  With `forced`
    [H, min(m, n)], each forced pick is checked to be within tie_tol of the
    step's minimum and then followed (ValueError at the first that is not)."""
    lib = _load()
    x, dt = _raw(q)
    H, n, D = x.shape
    k = max(0, min(m, n))
    picks = np.zeros((H, k), np.int32)
    tie = np.zeros((H, k), np.int32)
    fo = None if forced is None else np.ascontiguousarray(np.asarray(forced), dtype=np.int32)
    errors = {}

    def one(h):
        rc = lib.orc_fps(dt, D, n, m, _ptr(x, h * n * D), None if fo is None else _ptr(fo, h * k), float(tie_tol),
                         _ptr(picks, h * k) if k else None, _ptr(tie, h * k) if k else None)
        if rc < 0:
            errors[h] = -rc - 1

    _run(one, list(range(H)), threads)
    if errors:
        h = min(errors)
        raise ValueError(f"head {h}: forced pick at step {errors[h]} is not within {tie_tol} of the minimum")
    return picks, tie.astype(bool)
