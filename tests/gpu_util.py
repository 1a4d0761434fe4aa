"""Shared helpers for the GPU parity tests (inputs, comparison rules).

Comparison rules against the CPU oracle:
  * scores and row normalisers: |gpu - oracle| <= 1e-3 in natural-log units
    (1e-3 relative on the attention weight exp(s));
  * kept indices: let theta be the oracle score of the weakest chosen
    candidate; candidates within 1e-3 of theta form the tie band.  Outside
    the band GPU and oracle keep exactly the same indices; inside it they
    keep the same number.  Band size and in-band differences are reported;
  * compacted K/V: bit-exact, row for row, wherever the kept index agrees;
  * integer work (selection fed identical scores, compaction fed identical
    indices, beacon counts): bit-exact.
"""
import numpy as np
import torch

import oracle
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth

SCORE_TOL = 1e-3


def say(msg):
    print(f"[gpu] {msg}", flush=True)


def dims_of(w: synth.Workload, N=None, N_cap=None, budget=None, n_prefix=None) -> bkv.Dims:
    N = w.N if N is None else N
    return bkv.dims(B=w.B, Hq=w.Hq, Hkv=w.Hkv, D=w.D, N=N, N_cap=N if N_cap is None else N_cap, W=w.W, C=w.C,
                    budget=w.budget if budget is None else budget,
                    n_prefix=w.n_prefix if n_prefix is None else n_prefix, dtype=w.dtype)


def to_dev(x: dict) -> dict:
    return {k: v.cuda() for k, v in x.items()}


def host(t: torch.Tensor):
    return t.detach().cpu()


def raw_bits(t: torch.Tensor) -> np.ndarray:
    t = host(t).contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.view(torch.int32).numpy()


def assert_scores_close(got: np.ndarray, want: np.ndarray, what="scores"):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    both_inf = np.isneginf(got) & np.isneginf(want)
    assert not np.isnan(got).any(), f"{what}: NaN in GPU output"
    with np.errstate(invalid="ignore"):
        err = np.where(both_inf, 0.0, np.abs(got - want))
    worst = np.unravel_index(np.argmax(err), err.shape)
    assert err.max() <= SCORE_TOL, f"{what}: max |diff| {err.max():.3g} at {worst} (gpu {got[worst]}, ref {want[worst]})"
    return float(err.max())


def compare_kept(kept_gpu: np.ndarray, kept_ref: np.ndarray, s_ref: np.ndarray, N: int, W: int, n_prefix: int,
                 budget: int):
    """Tie-band rule per head; returns (band size total, in-band differences)."""
    band_total, diff_total = 0, 0
    for idx in np.ndindex(kept_ref.shape[:-1]):
        g, r, s = kept_gpu[idx], kept_ref[idx], s_ref[idx]
        assert len(g) == len(r) == min(budget, N)
        assert np.all(np.diff(g) > 0), f"head {idx}: kept not strictly ascending"
        if N <= budget:
            assert np.array_equal(g, r)
            continue
        forced = np.zeros(N, bool)
        forced[:n_prefix] = True
        forced[N - W:] = True
        chosen = np.setdiff1d(r, np.flatnonzero(forced))
        if len(chosen) == 0:
            assert np.array_equal(g, r)
            continue
        theta = s[chosen].min()
        band = (~forced) & (np.abs(s - theta) <= SCORE_TOL)
        gs, rs = set(g.tolist()), set(r.tolist())
        out_g = {j for j in gs if not band[j]}
        out_r = {j for j in rs if not band[j]}
        assert out_g == out_r, f"head {idx}: kept differs outside the tie band: {sorted(out_g ^ out_r)[:10]}"
        in_g = {j for j in gs if band[j]}
        in_r = {j for j in rs if band[j]}
        assert len(in_g) == len(in_r)
        band_total += int(band.sum())
        diff_total += len(in_g ^ in_r) // 2
    return band_total, diff_total


def assert_rows_match(K_gpu: torch.Tensor, K_ref_raw: np.ndarray, kept_gpu: np.ndarray, kept_ref: np.ndarray,
                      n_keep: int, what="K"):
    """Compacted rows bit-exact wherever GPU and oracle kept the same index."""
    g = raw_bits(K_gpu)
    r = np.asarray(K_ref_raw)
    if r.dtype == np.float32:
        r = r.view(np.int32)
    same = kept_gpu == kept_ref  # [..., n_keep]
    gv, rv = g[..., :n_keep, :], r[..., :n_keep, :]
    bad = (gv != rv).any(-1) & same
    assert not bad.any(), f"{what}: {int(bad.sum())} compacted rows differ (first at {np.argwhere(bad)[0]})"
