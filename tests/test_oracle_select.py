"""Pins for the oracle's selection (a4), compaction (a5) and the whole
eviction (a6), CPU only.

Expected values come from hand-worked fixtures, an exhaustive search over
all subsets on tiny inputs, numpy's take for the gather, and the
invariants of the selection rule checked with hypothesis.
"""
import itertools
import math

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle
from golden_io import load, scalar


def test_all_equal_scores():
    fx = load("topk_all_equal.txt")
    N = int(scalar(fx, "N"))
    kept = oracle.topk_head(np.zeros(N), int(scalar(fx, "budget")), int(scalar(fx, "W")),
                            int(scalar(fx, "n_prefix")))
    assert kept.tolist() == [int(v) for v in fx["kept"][0]]


def test_closed_form_eviction():
    fx = load("score_closed_form.txt")
    D = int(scalar(fx, "D"))
    keys = np.array([[float(v) for v in r] for r in fx["key"]], np.float32)
    beacon = np.array([math.sqrt(2) * math.log(2), 0], np.float32).reshape(1, 1, 1, D)
    recent = np.array([0, math.sqrt(2) * math.log(3)], np.float32).reshape(1, 1, 1, D)
    N = keys.shape[0]
    V = np.arange(N * D, dtype=np.float32).reshape(1, 1, N, D)
    out = oracle.evict(keys.reshape(1, 1, N, D), V, recent, beacon, np.ones((1, 1, 1), np.int32), N=N,
                       budget=int(scalar(fx, "budget")), W=int(scalar(fx, "W")))
    want = [int(v) for v in fx["kept"][0]]
    assert out["kept"][0, 0].tolist() == want
    np.testing.assert_array_equal(out["K"][0, 0, :len(want)], keys[want])
    np.testing.assert_array_equal(out["V"][0, 0, :len(want)], V[0, 0, want])


def test_max_aggregation_not_mean():
    # rows with given attention weights: keys = identity, rows = log(p)/scale
    fx = load("max_vs_mean.txt")
    P = np.array([[float(v) for v in r] for r in fx["row"]])
    scale = 0.5
    lse, s = oracle.score_rows(np.log(P) / scale, np.eye(3, dtype=np.float32), scale)
    np.testing.assert_allclose(lse, 0.0, atol=1e-12)
    np.testing.assert_allclose(np.exp(s), P.max(axis=0), rtol=1e-12)
    budget, W = int(scalar(fx, "budget")), int(scalar(fx, "W"))
    assert oracle.topk_head(s, budget, W, 0).tolist() == [int(v) for v in fx["kept_max"][0]]
    # the fixture discriminates: mean aggregation would pick the other token
    assert oracle.topk_head(np.log(P.mean(axis=0)), budget, W, 0).tolist() == \
        [int(v) for v in fx["kept_mean"][0]]


def _brute_topk(s, budget, W, n_prefix):
    N = len(s)
    if N <= budget:
        return list(range(N))
    forced = set(range(n_prefix)) | set(range(N - W, N))
    cand = [j for j in range(N) if j not in forced]
    ksel = budget - len(forced)
    rank = lambda j: (-s[j], j)  # (score descending, index ascending)
    hits = []
    for sub in itertools.combinations(cand, ksel):
        rest = [j for j in cand if j not in sub]
        if all(rank(a) < rank(b) for a in sub for b in rest):
            hits.append(sorted(forced | set(sub)))
    assert len(hits) == 1
    return hits[0]


@pytest.mark.parametrize("seed", range(40))
def test_exhaustive_subsets_tiny(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 11))
    W = int(rng.integers(0, 3))
    n_prefix = int(rng.integers(0, 3))
    budget = int(rng.integers(W + n_prefix, W + n_prefix + 5)) if W + n_prefix > 0 else int(rng.integers(1, 6))
    s = rng.integers(-3, 1, size=N).astype(np.float64)  # many ties
    assert oracle.topk_head(s, budget, W, n_prefix).tolist() == _brute_topk(s, budget, W, n_prefix)


def test_negative_zero_ties_positive_zero():
    s = np.array([-1.0, 0.0, -0.0, -0.0, -1.0])
    assert oracle.topk_head(s, 2, 0, 0).tolist() == [1, 2]


@settings(max_examples=200, deadline=None)
@given(st.integers(1, 300), st.integers(0, 8), st.integers(0, 4), st.integers(0, 400),
       st.integers(0, 2**31 - 1))
def test_selection_invariants(N, W, n_prefix, extra, seed):
    budget = W + n_prefix + extra
    if budget == 0:
        budget = 1
    rng = np.random.default_rng(seed)
    s = np.round(rng.normal(size=N), 1)
    kept = oracle.topk_head(s, budget, W, n_prefix)
    assert len(kept) == min(budget, N)
    assert np.all(np.diff(kept) > 0)
    if N > budget:
        ks = set(kept.tolist())
        forced = set(range(n_prefix)) | set(range(N - W, N))
        assert forced <= ks
        chosen = [j for j in ks if j not in forced]
        rejected = [j for j in range(N) if j not in ks]
        if chosen and rejected:
            worst = min(chosen, key=lambda j: (s[j], -j))
            best_rej = max(rejected, key=lambda j: (s[j], -j))
            assert (s[worst], -worst) > (s[best_rej], -best_rej)


def test_gather_equals_take_bf16_bits():
    rng = np.random.default_rng(0)
    B, H, Ncap, D, n = 2, 3, 40, 8, 11
    K = rng.integers(0, 2**16, size=(B, H, Ncap, D), dtype=np.uint16)  # any bits, NaNs included
    V = rng.integers(0, 2**16, size=(B, H, Ncap, D), dtype=np.uint16)
    kept = np.stack([np.stack([np.sort(rng.choice(33, n, replace=False)) for _ in range(H)]) for _ in range(B)])
    kept = kept.astype(np.int32)
    K2, V2 = oracle.compact(K, V, kept)
    for b in range(B):
        for h in range(H):
            np.testing.assert_array_equal(K2[b, h, :n], np.take(K[b, h], kept[b, h], axis=0))
            np.testing.assert_array_equal(V2[b, h, :n], np.take(V[b, h], kept[b, h], axis=0))
            np.testing.assert_array_equal(K2[b, h, n:], K[b, h, n:])


def test_gather_overlapping_rows_fp32():
    K = np.arange(4 * 2, dtype=np.float32).reshape(1, 1, 4, 2)
    kept = np.array([[[0, 2, 3]]], np.int32)
    K2, _ = oracle.compact(K, K.copy(), kept)
    np.testing.assert_array_equal(K2[0, 0], K[0, 0, [0, 2, 3, 3]])


def test_whole_eviction_matches_steps():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(9)
    B, Hkv, G, N, D, W, C, budget = 1, 2, 2, 40, 8, 3, 3, 12
    K = torch.from_numpy(rng.normal(size=(B, Hkv, N, D)).astype(np.float32)).to(torch.bfloat16)
    V = torch.from_numpy(rng.normal(size=(B, Hkv, N, D)).astype(np.float32)).to(torch.bfloat16)
    qw = torch.from_numpy(rng.normal(size=(B, Hkv * G, W, D)).astype(np.float32)).to(torch.bfloat16)
    bc = rng.normal(size=(B, Hkv, C, D)).astype(np.float32)
    cn = np.array([[[1, 0, 2], [3, 1, 1]]], np.int32)
    ang = rng.uniform(-3, 3, size=D // 2)
    c, s = np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)
    out = oracle.evict(K, V, qw, bc, cn, N=N, budget=budget, W=W, n_prefix=2, rope_cos=c, rope_sin=s)
    sc, lse = oracle.score(K, qw, bc, cn, N=N, rope_cos=c, rope_sin=s)
    np.testing.assert_array_equal(out["scores"], sc)
    kept = oracle.topk(sc, budget, W, 2)
    np.testing.assert_array_equal(out["kept"], kept)
    K2, V2 = oracle.compact(K, V, kept)
    np.testing.assert_array_equal(out["K"], K2)
    np.testing.assert_array_equal(out["V"], V2)
