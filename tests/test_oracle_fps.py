"""Pins for the oracle's farthest point sampling (Appendix D.1, Algorithm 1),
the selection step of Continual FPS (Section 4.2, Algorithm 2), CPU only.

Expected values come from two hand-worked 2-D examples, an independent numpy
formulation (average cosine as a dot product with the mean unit vector,
vectorised nearest-pick similarities), invariants of the greedy rule, and
special cases."""
import numpy as np
import pytest
import torch

import oracle
from golden_io import load


def _numpy_fps(q, m):
    """Algorithm 1 restated with unit vectors: avg = U @ mean(U), S = U @ u_r."""
    q = np.asarray(q, np.float64)
    n = q.shape[0]
    norms = np.linalg.norm(q, axis=1)
    U = np.where(norms[:, None] > 0, q / np.where(norms > 0, norms, 1)[:, None], 0.0)
    avg = U @ U.mean(axis=0)
    picks = [int(np.argmin(avg))]  # argmin returns the lowest index on ties
    S = U @ U[picks[0]]
    picked = np.zeros(n, bool)
    picked[picks[0]] = True
    while len(picks) < min(m, n):
        r = int(np.argmin(np.where(picked, np.inf, S)))
        picks.append(r)
        picked[r] = True
        S = np.maximum(S, U @ U[r])
    return picks


def test_hand_worked_example():
    fx = load("fps_hand_worked.txt")
    q = np.array([[float(v) for v in r] for r in fx["query"]], np.float32)[None]
    picks, tie = oracle.fps(q, 4, tie_tol=1e-9)
    assert picks[0].tolist() == [int(v) for v in fx["picks"][0]]
    assert not tie.any()


def test_hand_worked_ties_go_to_lowest_index():
    fx = load("fps_hand_worked.txt")
    q = np.array([[float(v) for v in r] for r in fx["tie_query"]], np.float32)[None]
    picks, tie = oracle.fps(q, 4, tie_tol=1e-9)
    assert picks[0].tolist() == [int(v) for v in fx["tie_picks"][0]]
    assert tie[0].astype(int).tolist() == [int(v) for v in fx["tie_steps"][0]]


@pytest.mark.parametrize("n,D,m", [(7, 2, 7), (40, 16, 12), (100, 64, 16), (33, 128, 33)])
def test_matches_independent_numpy_formulation(n, D, m):
    rng = np.random.default_rng(n * 1000 + D)
    q = rng.standard_normal((3, n, D)).astype(np.float32)
    picks, _ = oracle.fps(q, m)
    for h in range(3):
        assert picks[h].tolist() == _numpy_fps(q[h], m)


def test_prefix_property_and_distinct_picks():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((2, 50, 32)).astype(np.float32)
    full, _ = oracle.fps(q, 50)
    for m in (1, 5, 17, 49):
        part, _ = oracle.fps(q, m)
        assert np.array_equal(part, full[:, :m])
    for h in range(2):
        assert sorted(full[h].tolist()) == list(range(50))


def test_scale_invariance():
    rng = np.random.default_rng(6)
    q = rng.standard_normal((1, 30, 16)).astype(np.float32)
    s = rng.uniform(0.25, 4.0, size=(1, 30, 1)).astype(np.float32)
    s = 2.0 ** np.round(np.log2(s))  # powers of two: exact in fp32
    a, _ = oracle.fps(q, 12)
    b, _ = oracle.fps(q * s, 12)
    assert np.array_equal(a, b)


def test_greedy_rule_each_pick_is_the_farthest():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((1, 25, 8)).astype(np.float64)
    picks, _ = oracle.fps(q.astype(np.float32), 10)
    U = q[0] / np.linalg.norm(q[0], axis=1, keepdims=True)
    C = U @ U.T
    assert picks[0][0] == int(np.argmin(C.mean(axis=1)))
    for k in range(1, 10):
        chosen = picks[0][:k]
        S = C[:, chosen].max(axis=1)
        rest = [j for j in range(25) if j not in chosen]
        assert S[picks[0][k]] == pytest.approx(min(S[j] for j in rest), abs=1e-6)


def test_more_picks_than_queries_and_tiny_sets():
    q = np.array([[[1, 2, 3, 4]]], np.float32)
    assert oracle.fps(q, 5)[0].tolist() == [[0]]
    rng = np.random.default_rng(8)
    q = rng.standard_normal((1, 6, 4)).astype(np.float32)
    picks, _ = oracle.fps(q, 10)
    assert picks.shape == (1, 6) and sorted(picks[0].tolist()) == list(range(6))
    assert oracle.fps(q, 0)[0].shape == (1, 0)


def test_zero_vectors_have_cosine_zero():
    # a zero query is at cosine 0 from everything: with two opposite unit
    # vectors (average cosine 0 each) and a zero vector (average 0), the
    # first pick is query 0 on the tie; S = (., -1, 0) then picks query 1
    q = np.array([[[1, 0], [-1, 0], [0, 0]]], np.float32)
    picks, tie = oracle.fps(q, 3, tie_tol=1e-9)
    assert picks[0].tolist() == [0, 1, 2]
    assert tie[0].tolist() == [True, False, False]


def test_forced_picks_are_checked_against_the_minimum():
    fx = load("fps_hand_worked.txt")
    q = np.array([[float(v) for v in r] for r in fx["tie_query"]], np.float32)[None]
    # the other side of each tie is accepted ...
    picks, _ = oracle.fps(q, 4, forced=[[1, 3, 0, 2]], tie_tol=1e-6)
    assert picks[0].tolist() == [1, 3, 0, 2]
    # ... a pick that is not (near-)minimal is not
    with pytest.raises(ValueError):
        oracle.fps(q, 4, forced=[[0, 1, 2, 3]], tie_tol=1e-6)


def test_bf16_input_widens_exactly():
    rng = np.random.default_rng(9)
    q = torch.from_numpy(rng.standard_normal((2, 20, 16)).astype(np.float32)).to(torch.bfloat16)
    a, _ = oracle.fps(q, 8)
    b, _ = oracle.fps(q.float().numpy(), 8)
    assert np.array_equal(a, b)


def test_average_includes_each_query_itself():
    # avg_i sums over every j, i included (cos(q_i, q_i) = 1 for a non-zero
    # query, 0 for a zero one): for (1, 0) and (0, 0) the averages are 1/2
    # and 0, so the zero query is picked first
    q = np.array([[[1, 0], [0, 0]]], np.float32)
    picks, tie = oracle.fps(q, 2, tie_tol=1e-9)
    assert picks[0].tolist() == [1, 0]
    assert not tie[0][0]
