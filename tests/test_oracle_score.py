"""Pins for the oracle's observation rows (a2) and scores (a3), CPU only.

Expected values come from a closed form worked by hand, library routines
(scipy's softmax / log_softmax, complex multiplication for the rotation,
torch's bf16 rounding), a float64 brute force of the full attention matrix,
and invariants (rows normalise to 1, permuting or repeating rows changes
nothing, identical keys give -ln N).
"""
import math

import numpy as np
import pytest
from scipy.special import log_softmax, softmax

import oracle
from golden_io import load, scalar

torch = pytest.importorskip("torch")


def test_closed_form_example():
    fx = load("score_closed_form.txt")
    D = int(scalar(fx, "D"))
    keys = np.array([[float(v) for v in r] for r in fx["key"]], np.float32)
    bln = [float(v) for v in fx["beacon_sqrt2_ln"][0]]
    rln = [float(v) for v in fx["recent_sqrt2_ln"][0]]
    beacon = np.array([math.sqrt(2) * math.log(v) if v else 0.0 for v in bln], np.float32)
    recent = np.array([math.sqrt(2) * math.log(v) if v else 0.0 for v in rln], np.float32)
    N = keys.shape[0]
    K = keys.reshape(1, 1, N, D)
    s, lse = oracle.score(K, recent.reshape(1, 1, 1, D), beacon.reshape(1, 1, 1, D),
                          np.ones((1, 1, 1), np.int32), N=N)
    want = np.log([float(v) for v in fx["prob"][0]])
    np.testing.assert_allclose(s[0, 0], want, atol=2e-6)
    np.testing.assert_allclose(lse[0, 0], [math.log(float(scalar(fx, "lse_beacon_exp"))),
                                           math.log(float(scalar(fx, "lse_recent_exp")))], atol=2e-6)


def test_single_row_is_log_softmax():
    rng = np.random.default_rng(0)
    D, N = 16, 37
    Y = rng.normal(size=(1, D))
    K = rng.normal(size=(N, D)).astype(np.float32)
    scale = 0.25
    lse, s = oracle.score_rows(Y, K, scale)
    np.testing.assert_allclose(s, log_softmax(scale * (Y @ K.astype(np.float64).T))[0], rtol=0, atol=1e-12)


def test_identical_keys_give_minus_log_n():
    rng = np.random.default_rng(1)
    D, N = 8, 50
    K = np.tile(rng.normal(size=(1, D)).astype(np.float32), (N, 1))
    _, s = oracle.score_rows(rng.normal(size=(5, D)), K, 0.3)
    np.testing.assert_allclose(s, -math.log(N), atol=1e-12)


def _brute(Y, K, scale):
    P = softmax(scale * (Y @ K.T), axis=1)
    return np.log(P.max(axis=0))


@pytest.mark.parametrize("G", [1, 2, 3, 7])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_brute_force_full_attention(G, dtype):
    # No RoPE table: beacon rows are the beacons rounded to the cache dtype
    # (torch's round-to-nearest-even); recent rows are the given queries.
    rng = np.random.default_rng(10 + G)
    B, Hkv, N, D, W, C = 2, 2, 23, 8, 3, 4
    Hq = Hkv * G
    K = torch.from_numpy(rng.normal(size=(B, Hkv, N + 5, D)).astype(np.float32)).to(dtype)
    qw = torch.from_numpy((2 * rng.normal(size=(B, Hq, W, D))).astype(np.float32)).to(dtype)
    bc = (2 * rng.normal(size=(B, Hkv, C, D))).astype(np.float32)
    cn = rng.integers(0, 3, size=(B, Hkv, C)).astype(np.int32)
    cn[0, 0] = 0  # one head with no occupied beacon slot
    bc[cn == 0] = np.nan  # empty slots must not be read
    s, lse = oracle.score(K, qw, bc, cn, N=N)
    scale = float(np.float32(1 / math.sqrt(D)))
    for b in range(B):
        for h in range(Hkv):
            act = np.flatnonzero(cn[b, h] > 0)
            rows_b = torch.from_numpy(bc[b, h, act]).to(dtype).double().numpy()
            rows_w = qw[b, h * G:(h + 1) * G].double().reshape(-1, D).numpy()
            Y = np.concatenate([rows_b, rows_w])
            Kd = K[b, h, :N].double().numpy()
            np.testing.assert_allclose(s[b, h], _brute(Y, Kd, scale), rtol=0, atol=1e-11)
            L = scale * Y @ Kd.T
            want_lse = np.log(np.exp(L).sum(axis=1))
            got = np.concatenate([lse[b, h, act], lse[b, h, C:]])
            np.testing.assert_allclose(got, want_lse, atol=1e-11)
            assert np.all(np.isneginf(lse[b, h, :C][cn[b, h] == 0]))


def test_rows_normalise_and_score_is_row_max():
    rng = np.random.default_rng(2)
    R, N, D = 6, 31, 8
    Y = 3 * rng.normal(size=(R, D))
    K = rng.normal(size=(N, D)).astype(np.float32)
    scale = 0.2
    lse, s = oracle.score_rows(Y, K, scale)
    L = scale * Y @ K.astype(np.float64).T
    np.testing.assert_allclose(np.exp(L - lse[:, None]).sum(axis=1), 1.0, atol=1e-12)
    D_ = L - lse[:, None]
    assert np.all(s[None, :] >= D_ - 1e-12)
    np.testing.assert_allclose(s, D_.max(axis=0), atol=1e-12)


def test_row_permutation_and_duplication_invariance():
    rng = np.random.default_rng(3)
    R, N, D = 5, 20, 8
    Y = 2 * rng.normal(size=(R, D))
    K = rng.normal(size=(N, D)).astype(np.float32)
    _, s = oracle.score_rows(Y, K, 0.3)
    _, sp = oracle.score_rows(Y[rng.permutation(R)], K, 0.3)
    _, sd = oracle.score_rows(np.concatenate([Y, Y[:2], Y[:2]]), K, 0.3)
    np.testing.assert_allclose(sp, s, atol=1e-13)
    np.testing.assert_allclose(sd, s, atol=1e-13)


def test_no_rows_scores_minus_inf():
    K = np.ones((1, 1, 4, 2), np.float32)
    s, lse = oracle.score(K, np.zeros((1, 1, 0, 2), np.float32), np.zeros((1, 1, 2, 2), np.float32),
                          np.zeros((1, 1, 2), np.int32), N=4)
    assert np.all(np.isneginf(s)) and np.all(np.isneginf(lse))


def test_query_head_grouping():
    # q-head 2 of Hq=4, Hkv=2 (G=2) belongs to kv-head 1 (hq // G), not to
    # kv-head 0 (hq % Hkv).  Only that query is sharp; it points at key 5.
    rng = np.random.default_rng(4)
    B, Hkv, G, N, D, W = 1, 2, 2, 12, 8, 1
    K = rng.normal(size=(B, Hkv, N, D)).astype(np.float32)
    qw = 1e-3 * rng.normal(size=(B, Hkv * G, W, D)).astype(np.float32)
    qw[0, 2, 0] = 40 * K[0, 1, 5] / np.linalg.norm(K[0, 1, 5])
    s, _ = oracle.score(K, qw, np.zeros((B, Hkv, 1, D), np.float32), np.zeros((B, Hkv, 1), np.int32), N=N)
    assert np.argmax(s[0, 1]) == 5 and s[0, 1, 5] > -0.1
    assert s[0, 0].max() < -1.0


def test_rope_rotate_half_against_complex_multiplication():
    rng = np.random.default_rng(5)
    D = 16
    beta = rng.normal(size=D).astype(np.float32)
    ang = rng.uniform(-3, 3, size=D // 2)
    c, s = np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)
    out = oracle.rope_row(beta, c, s)
    z = (beta[:D // 2].astype(np.float64) + 1j * beta[D // 2:]) * (c.astype(np.float64) + 1j * s)
    np.testing.assert_allclose(out, np.concatenate([z.real, z.imag]), rtol=0, atol=1e-6)
    # exact special cases: no turn, and a quarter turn (x, y) -> (-y, x)
    one, zero = np.ones(D // 2, np.float32), np.zeros(D // 2, np.float32)
    np.testing.assert_array_equal(oracle.rope_row(beta, one, zero), beta)
    np.testing.assert_array_equal(oracle.rope_row(beta, zero, one),
                                  np.concatenate([-beta[D // 2:], beta[:D // 2]]))
    np.testing.assert_array_equal(oracle.rope_row(beta), beta)


def test_rope_products_rounded_separately_then_bf16():
    rng = np.random.default_rng(6)
    D = 64
    beta = (5 * rng.normal(size=D)).astype(np.float32)
    ang = rng.uniform(-3, 3, size=D // 2)
    c, s = np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)
    h = D // 2
    f32 = np.float32
    lo = (beta[:h] * c).astype(f32) - (beta[h:] * s).astype(f32)
    hi = (beta[h:] * c).astype(f32) + (beta[:h] * s).astype(f32)
    want = np.concatenate([lo, hi]).astype(f32)
    np.testing.assert_array_equal(oracle.rope_row(beta, c, s), want)
    want_bf = torch.from_numpy(want).to(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(oracle.rope_row(beta, c, s, to_bf16=True), want_bf)


def test_beacon_rows_are_rotated_to_the_step():
    # a beacon and the same vector given as a recent query differ only by
    # the rotation the beacon receives
    rng = np.random.default_rng(7)
    N, D = 9, 8
    K = rng.normal(size=(1, 1, N, D)).astype(np.float32)
    beta = rng.normal(size=(1, 1, 1, D)).astype(np.float32)
    ang = rng.uniform(-3, 3, size=D // 2)
    c, s = np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)
    sb, _ = oracle.score(K, np.zeros((1, 1, 0, D), np.float32), beta, np.ones((1, 1, 1), np.int32),
                         N=N, rope_cos=c, rope_sin=s)
    rot = oracle.rope_row(beta[0, 0, 0], c, s).reshape(1, 1, 1, D)
    sr, _ = oracle.score(K, rot, np.zeros((1, 1, 1, D), np.float32), np.zeros((1, 1, 1), np.int32), N=N)
    np.testing.assert_array_equal(sb, sr)
    su, _ = oracle.score(K, beta, np.zeros((1, 1, 1, D), np.float32), np.zeros((1, 1, 1), np.int32), N=N)
    assert np.abs(su - sb).max() > 1e-3
