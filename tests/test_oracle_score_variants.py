"""Pins for the oracle's scoring variants, CPU only: Eq. (6)'s mean form next
to the max form, and recent queries that see only the keys up to their own
position.

Expected values come from a hand-worked example (tests/golden/
score_variants.txt), the max-versus-mean selection fixture, a numpy brute
force over masked softmaxes, and invariants (one row: mean = max; limits
past the last key change nothing; max - ln R <= mean <= max)."""
import math

import numpy as np
import pytest

import oracle
from golden_io import load, scalar

SQRT2 = math.sqrt(2.0)


def _fixture():
    fx = load("score_variants.txt")
    keys = np.array([[float(v) for v in r] for r in fx["key"]], np.float32)
    rows = np.array([[SQRT2 * math.log(float(a)), SQRT2 * math.log(float(b))] for a, b in fx["row_sqrt2_ln"]])
    limit = np.array([int(v) for v in fx["limit"][0]], np.int32)
    return fx, keys, rows, limit


@pytest.mark.parametrize("agg,causal", [("max", False), ("max", True), ("mean", False), ("mean", True)])
def test_hand_worked_variants(agg, causal):
    fx, keys, rows, limit = _fixture()
    lse, s = oracle.score_rows(rows, keys, 1.0 / SQRT2, agg=agg, limit=limit if causal else None)
    name = agg + ("_causal" if causal else "")
    want = np.array([float(v) for v in fx[name][0]])
    np.testing.assert_allclose(np.exp(s), want, rtol=1e-12)
    want_lse = np.log([float(v) for v in fx["lse_exp_causal" if causal else "lse_exp"][0]])
    np.testing.assert_allclose(lse, want_lse, rtol=1e-12)


@pytest.mark.parametrize("agg,causal", [("max", True), ("mean", False), ("mean", True)])
def test_hand_worked_variants_through_head_scoring(agg, causal):
    # the same example as one kv-head: one beacon slot, one query head with
    # W = 2 recent queries (oldest first), fp32; pins the slot order and the
    # recent positions N - W + w that the causal limits come from
    fx, keys, rows, _ = _fixture()
    K = keys[None, None]                                   # [1, 1, 3, 2]
    q_win = rows[1:].astype(np.float32)[None, None]        # [1, 1, 2, 2]
    beacons = rows[:1].astype(np.float32)[None, None]      # [1, 1, 1, 2]
    counts = np.ones((1, 1, 1), np.int32)
    s, lse = oracle.score(K, q_win, beacons, counts, N=3, scale=1.0 / SQRT2, agg=agg, causal=causal)
    name = agg + ("_causal" if causal else "")
    want = np.array([float(v) for v in fx[name][0]])
    np.testing.assert_allclose(np.exp(s[0, 0]), want, rtol=1e-6)  # rows rounded to fp32
    want_lse = np.log([float(v) for v in fx["lse_exp_causal" if causal else "lse_exp"][0]])
    np.testing.assert_allclose(lse[0, 0], want_lse, rtol=1e-6)


def test_mean_aggregation_selects_the_other_token():
    # the max-versus-mean fixture: the mean form keeps the token the max
    # form drops (Table 2's comparison)
    fx = load("max_vs_mean.txt")
    P = np.array([[float(v) for v in r] for r in fx["row"]])
    scale = 0.5
    _, s = oracle.score_rows(np.log(P) / scale, np.eye(3, dtype=np.float32), scale, agg="mean")
    np.testing.assert_allclose(np.exp(s), P.mean(axis=0), rtol=1e-12)
    budget, W = int(scalar(fx, "budget")), int(scalar(fx, "W"))
    assert oracle.topk_head(s, budget, W, 0).tolist() == [int(v) for v in fx["kept_mean"][0]]


def _brute(Y, K, scale, agg, limit):
    L = scale * (Y @ K.T)  # [R, N]
    R, N = L.shape
    mask = np.ones_like(L, bool) if limit is None else (np.arange(N)[None, :] <= np.asarray(limit)[:, None])
    Lm = np.where(mask, L, -np.inf)
    with np.errstate(divide="ignore", invalid="ignore"):
        m = Lm.max(axis=1, keepdims=True)
        m = np.where(np.isfinite(m), m, 0.0)
        Pw = np.where(mask, np.exp(Lm - m), 0.0)
        Z = Pw.sum(axis=1, keepdims=True)
        Pw = np.divide(Pw, Z, out=np.zeros_like(Pw), where=Z > 0)
        if agg == "max":
            return np.log(Pw.max(axis=0))
        return np.log(Pw.mean(axis=0))


@pytest.mark.parametrize("agg", ["max", "mean"])
@pytest.mark.parametrize("seed", range(6))
def test_brute_force_masked_softmax(agg, seed):
    rng = np.random.default_rng(seed)
    R, N, D = int(rng.integers(1, 9)), int(rng.integers(1, 40)), 8
    Y = rng.standard_normal((R, D)) * 2
    K = rng.standard_normal((N, D)).astype(np.float32)
    limit = rng.integers(-1, N + 2, R).astype(np.int32)
    for lim in (None, limit):
        _, s = oracle.score_rows(Y, K, 0.7, agg=agg, limit=lim)
        want = _brute(Y, K.astype(np.float64), 0.7, agg, lim)
        np.testing.assert_allclose(s, want, rtol=1e-10, atol=1e-12)


def test_one_row_mean_equals_max():
    rng = np.random.default_rng(3)
    Y, K = rng.standard_normal((1, 16)), rng.standard_normal((50, 16)).astype(np.float32)
    _, smax = oracle.score_rows(Y, K, 0.25)
    _, smean = oracle.score_rows(Y, K, 0.25, agg="mean")
    np.testing.assert_allclose(smean, smax, rtol=0, atol=1e-13)


def test_limits_past_the_last_key_change_nothing():
    rng = np.random.default_rng(4)
    Y, K = rng.standard_normal((5, 16)), rng.standard_normal((30, 16)).astype(np.float32)
    for agg in ("max", "mean"):
        l0, s0 = oracle.score_rows(Y, K, 0.25, agg=agg)
        l1, s1 = oracle.score_rows(Y, K, 0.25, agg=agg, limit=np.array([29, 30, 100, 29, 29]))
        np.testing.assert_array_equal(s0, s1)
        np.testing.assert_array_equal(l0, l1)


def test_mean_lies_between_max_minus_log_rows_and_max():
    rng = np.random.default_rng(5)
    Y, K = rng.standard_normal((7, 16)) * 3, rng.standard_normal((60, 16)).astype(np.float32)
    limit = rng.integers(0, 60, 7)
    _, smax = oracle.score_rows(Y, K, 0.25, limit=limit)
    _, smean = oracle.score_rows(Y, K, 0.25, agg="mean", limit=limit)
    assert np.all(smean <= smax + 1e-12)
    assert np.all(smean >= smax - math.log(7) - 1e-12)


def test_a_row_that_sees_nothing():
    # a recent query older than every key (limit -1) has lse -inf and adds
    # weight 0; a key no row sees scores -inf
    Y = np.array([[1.0, 0.0], [0.0, 1.0]])
    K = np.array([[1, 0], [0, 1], [1, 1]], np.float32)
    lse, s = oracle.score_rows(Y, K, 1.0, agg="mean", limit=np.array([-1, 1]))
    assert lse[0] == -np.inf and np.isfinite(lse[1])
    w1 = np.exp([0.0, 1.0]) / np.exp([0.0, 1.0]).sum()
    np.testing.assert_allclose(np.exp(s[:2]), w1 / 2, rtol=1e-12)  # mean over both rows
    assert s[2] == -np.inf
    _, smax = oracle.score_rows(Y, K, 1.0, agg="max", limit=np.array([-1, 1]))
    np.testing.assert_allclose(np.exp(smax[:2]), w1, rtol=1e-12)
    assert smax[2] == -np.inf
