"""Pins for the oracle's hole-filling compaction (CPU only).

The paper's Algorithm 2 gathers the kept rows in token order (orc_compact,
pinned in its own tests); the hole-filling layout keeps the same set in
rows [0, n) but moves only the kept rows at or above n.  It is pinned by a
hand-worked example and by properties that hold for any input: the same
rows as the order-preserving compaction (sorted by their old positions),
kept rows below n never move, the number of moves is the least any layout
of the kept set can make, holes take the tail rows in ascending order, and
rows from n on are untouched."""
import itertools

import numpy as np
import pytest

import oracle


def _kv(P, N, D, seed):
    rng = np.random.default_rng(seed)
    K = rng.integers(-2**31, 2**31 - 1, (1, P, N, D), dtype=np.int64).astype(np.int32).view(np.float32)
    V = rng.integers(-2**31, 2**31 - 1, (1, P, N, D), dtype=np.int64).astype(np.int32).view(np.float32)
    return K, V


def test_hand_worked():
    # N = 10, keep 5: kept = (1, 3, 4, 7, 9).  Kept rows below 5 (1, 3, 4)
    # stay; the holes below 5 are positions 0 and 2, which take the kept
    # rows at or above 5 in order: 0 <- 7, 2 <- 9.
    K, V = _kv(1, 10, 4, 0)
    kept = np.array([[[1, 3, 4, 7, 9]]], np.int32)
    Kf, Vf, src_of, moved = oracle.compact_fill(K, V, kept, N=10)
    assert src_of[0, 0].tolist() == [7, 1, 9, 3, 4]
    assert moved[0, 0] == 2
    for j, s in enumerate([7, 1, 9, 3, 4]):
        assert np.array_equal(Kf[0, 0, j].view(np.int32), K[0, 0, s].view(np.int32))
        assert np.array_equal(Vf[0, 0, j].view(np.int32), V[0, 0, s].view(np.int32))


def _check_properties(K, V, kept, N):
    n = kept.shape[2]
    Kf, Vf, src_of, moved = oracle.compact_fill(K, V, kept, N=N)
    Ko, Vo = oracle.compact(K, V, kept)
    for h in range(kept.shape[1]):
        kp, so = kept[0, h], src_of[0, h]
        assert sorted(so.tolist()) == kp.tolist()  # a bijection onto the kept set
        order = np.argsort(so, kind="stable")
        # sorted by old position, the rows are those of the order-preserving gather
        assert np.array_equal(Kf[0, h, :n][order].view(np.int32), Ko[0, h, :n].view(np.int32))
        assert np.array_equal(Vf[0, h, :n][order].view(np.int32), Vo[0, h, :n].view(np.int32))
        below = kp[kp < n]
        assert np.array_equal(so[below], below)  # kept rows below n never move
        assert moved[0, h] == int((kp >= n).sum())  # the least number of moves
        holes = np.setdiff1d(np.arange(n), below)
        assert np.array_equal(so[holes], kp[kp >= n])  # holes take the tail in ascending order
        assert np.array_equal(Kf[0, h, n:].view(np.int32), K[0, h, n:].view(np.int32))  # rows from n on untouched
        assert np.array_equal(Vf[0, h, n:].view(np.int32), V[0, h, n:].view(np.int32))


def test_every_subset_of_small_heads():
    for N in range(1, 8):
        K, V = _kv(1, N, 3, N)
        for n in range(0, N + 1):
            for sub in itertools.combinations(range(N), n):
                kept = np.array(sub, np.int32).reshape(1, 1, n)
                _check_properties(K, V, kept, N)


@pytest.mark.parametrize("seed", range(5))
def test_random_heads(seed):
    rng = np.random.default_rng(seed)
    P, N = 4, int(rng.integers(50, 400))
    n = int(rng.integers(1, N))
    K, V = _kv(P, N, 8, seed)
    kept = np.stack([np.sort(rng.choice(N, n, replace=False)) for _ in range(P)]).astype(np.int32)[None]
    _check_properties(K, V, kept, N)


def test_identity_moves_nothing():
    K, V = _kv(2, 20, 4, 1)
    kept = np.tile(np.arange(12, dtype=np.int32), (1, 2, 1))
    Kf, _, src_of, moved = oracle.compact_fill(K, V, kept, N=20)
    assert (moved == 0).all() and np.array_equal(src_of[0, 0], np.arange(12))
    assert np.array_equal(Kf.view(np.int32), K.view(np.int32))


def test_rejects_unsorted_or_out_of_range():
    K, V = _kv(1, 10, 2, 2)
    for bad in ([3, 2, 5], [1, 1, 4], [1, 4, 10], [-1, 2, 3]):
        with pytest.raises(RuntimeError):
            oracle.compact_fill(K, V, np.array(bad, np.int32).reshape(1, 1, 3), N=10)
