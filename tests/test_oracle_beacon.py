"""Pins for the oracle's beacon update (a1), CPU only.

What fixes the expected values here is not the oracle itself: two streams
worked by hand (tests/golden/), numpy's mean for the single-slot case, the
member-mean and count invariants recomputed from the assignment log, and the
GQA head grouping checked against numpy on the raw queries.
"""
import numpy as np
import pytest

import oracle
from golden_io import load, scalar


def _stream_from_fixture(fx):
    D, G, T = int(scalar(fx, "D")), int(scalar(fx, "G")), int(scalar(fx, "T"))
    arrivals = np.array([[float(v) for v in row] for row in fx["query"]], np.float32)
    # arrival order is t-major then g; the tensor layout is [B, Hq, T, D]
    q = np.zeros((1, G, T, D), np.float32)
    i = 0
    for t in range(T):
        for g in range(G):
            q[0, g, t] = arrivals[i]
            i += 1
    return q, D, G, T


@pytest.mark.parametrize("name", ["beacon_two_cluster.txt", "beacon_gqa_order.txt"])
def test_hand_worked_streams(name):
    fx = load(name)
    q, D, G, T = _stream_from_fixture(fx)
    C = int(scalar(fx, "C"))
    beacons = np.zeros((1, 1, C, D), np.float32)
    counts = np.zeros((1, 1, C), np.int32)
    out = oracle.beacon_update(q, beacons, counts, Hkv=1)
    assert out["assign"][0, 0].tolist() == [int(v) for v in fx["assign"][0]]
    assert out["near_tie"][0, 0].astype(int).tolist() == [int(v) for v in fx["near_tie"][0]]
    assert out["counts"][0, 0].tolist() == [int(v) for v in fx["counts"][0]]
    want = np.array([[float(v) for v in row] for row in fx["beacon"]], np.float32)
    np.testing.assert_allclose(out["beacons"][0, 0], want, rtol=1e-6, atol=1e-7)


def test_single_slot_is_the_running_mean():
    rng = np.random.default_rng(1)
    G, T, D = 3, 7, 5
    q = rng.normal(size=(1, G, T, D)).astype(np.float32)
    out = oracle.beacon_update(q, np.zeros((1, 1, 1, D), np.float32), np.zeros((1, 1, 1), np.int32), Hkv=1)
    assert out["counts"][0, 0, 0] == G * T
    np.testing.assert_allclose(out["beacons"][0, 0, 0], q[0].reshape(-1, D).mean(axis=0), rtol=1e-5, atol=1e-6)


def _clustered_stream(rng, B, Hq, T, D, k, sigma=0.2):
    cent = rng.normal(size=(k, D))
    cent /= np.linalg.norm(cent, axis=1, keepdims=True)
    lab = rng.integers(0, k, size=(B, Hq, T))
    return (cent[lab] + sigma * rng.normal(size=(B, Hq, T, D))).astype(np.float32)


def test_counts_sum_and_members_mean():
    rng = np.random.default_rng(2)
    B, Hkv, G, T, D, C = 2, 2, 3, 40, 8, 4
    q = _clustered_stream(rng, B, Hkv * G, T, D, k=4)
    out = oracle.beacon_update(q, np.zeros((B, Hkv, C, D), np.float32), np.zeros((B, Hkv, C), np.int32), Hkv=Hkv)
    assert (out["counts"].sum(axis=2) == T * G).all()
    for b in range(B):
        for h in range(Hkv):
            # arrival order t-major then g over the group's query heads
            arr = q[b, h * G:(h + 1) * G].transpose(1, 0, 2).reshape(-1, D)
            lab = out["assign"][b, h]
            for c in range(C):
                members = arr[lab == c]
                assert len(members) == out["counts"][b, h, c]
                if len(members):
                    np.testing.assert_allclose(out["beacons"][b, h, c], members.mean(axis=0),
                                               rtol=2e-5, atol=2e-5)


def test_assignment_is_most_cosine_similar():
    # every non-seeding query joined the slot with the largest cosine to the
    # beacons as they stood when it arrived (checked by replaying the log)
    rng = np.random.default_rng(3)
    G, T, D, C = 2, 30, 6, 3
    q = _clustered_stream(rng, 1, G, T, D, k=3, sigma=0.4)
    out = oracle.beacon_update(q, np.zeros((1, 1, C, D), np.float32), np.zeros((1, 1, C), np.int32), Hkv=1)
    arr = q[0].transpose(1, 0, 2).reshape(-1, D).astype(np.float64)
    lab = out["assign"][0, 0]
    members = [[] for _ in range(C)]
    for i, x in enumerate(arr):
        if i < C:
            assert lab[i] == i  # empty slots seed in order
        else:
            means = np.array([np.mean(m, axis=0) for m in members])
            cos = means @ x / (np.linalg.norm(means, axis=1) * np.linalg.norm(x))
            assert lab[i] == int(np.argmax(cos))
        members[lab[i]].append(x)


def test_gqa_grouping_of_query_heads():
    # kv-head h owns query heads h*G .. h*G+G-1: with one slot each beacon is
    # the mean of exactly those heads' queries
    rng = np.random.default_rng(4)
    B, Hkv, G, T, D = 1, 3, 2, 5, 4
    q = rng.normal(size=(B, Hkv * G, T, D)).astype(np.float32)
    out = oracle.beacon_update(q, np.zeros((B, Hkv, 1, D), np.float32), np.zeros((B, Hkv, 1), np.int32), Hkv=Hkv)
    for h in range(Hkv):
        want = q[0, h * G:(h + 1) * G].reshape(-1, D).mean(axis=0)
        np.testing.assert_allclose(out["beacons"][0, h, 0], want, rtol=1e-5, atol=1e-6)


def test_zero_query_joins_lowest_slot():
    D = 3
    beacons = np.array([[[[0, 1, 0], [1, 0, 0]]]], np.float32)
    counts = np.array([[[1, 1]]], np.int32)
    q = np.zeros((1, 1, 1, D), np.float32)
    out = oracle.beacon_update(q, beacons, counts, Hkv=1)
    assert out["assign"][0, 0, 0] == 0 and bool(out["near_tie"][0, 0, 0])
    np.testing.assert_array_equal(out["beacons"][0, 0, 0], [0, 0.5, 0])
    assert out["counts"][0, 0].tolist() == [2, 1]


def test_slot_permutation_equivariance():
    rng = np.random.default_rng(5)
    G, T, D, C = 2, 20, 8, 5
    q = rng.normal(size=(1, G, T, D)).astype(np.float32)
    b0 = rng.normal(size=(1, 1, C, D)).astype(np.float32)
    c0 = rng.integers(1, 9, size=(1, 1, C)).astype(np.int32)
    perm = rng.permutation(C)
    a = oracle.beacon_update(q, b0, c0, Hkv=1)
    p = oracle.beacon_update(q, b0[:, :, perm], c0[:, :, perm], Hkv=1)
    np.testing.assert_array_equal(p["beacons"][0, 0], a["beacons"][0, 0][perm])
    np.testing.assert_array_equal(p["counts"][0, 0], a["counts"][0, 0][perm])
    # new slot i holds old slot perm[i]
    np.testing.assert_array_equal(perm[p["assign"][0, 0]], a["assign"][0, 0])


def test_bf16_queries_widen_exactly():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(6)
    q = torch.from_numpy(rng.normal(size=(1, 2, 6, 4)).astype(np.float32)).to(torch.bfloat16)
    z = lambda: (np.zeros((1, 1, 2, 4), np.float32), np.zeros((1, 1, 2), np.int32))
    a = oracle.beacon_update(q, *z(), Hkv=1)
    b = oracle.beacon_update(q.float().numpy(), *z(), Hkv=1)
    np.testing.assert_array_equal(a["beacons"], b["beacons"])
    np.testing.assert_array_equal(a["assign"], b["assign"])
