"""GPU parity of Continual FPS (bkv_fps, bkv_fps_gather) against the oracle.

Comparison rule.  FPS turns floating point into indices (Appendix D.1,
Algorithm 1: argmins of average and running-maximum cosines).  The kernels
form every cosine, and every summed average, from at most K = n + D + 8 fp32
operations on exact inputs, so each value is within gamma_K = K u / (1 - K u)
(u = 2^-24, relative to a quantity of magnitude <= 1) of its exact value, and
two of them can swap order only when they lie within 2 gamma_K of each
other.  Hence, with tol = 2 gamma_K:
  * every GPU pick must be within tol of the oracle's minimum at that step,
    given the GPU's earlier picks (the oracle's forced mode checks this);
  * GPU and oracle picks agree exactly up to the first step at which the
    oracle sees a second candidate within tol of its minimum;
  * gathered rows are bit-exact copies (or exact fp32 widenings) of the
    picked rows; the rows after them are untouched.
At sizes where the oracle's O(n^2 D) average is too slow the same greedy rule
is checked in fp64 numpy (the average regrouped as q_i/|q_i| . mean_j
q_j/|q_j|), and a repeated-axes input whose answer is known in closed form
pins the exact picks.
"""

import numpy as np
import pytest
import torch

import oracle
from golden_io import load
from gpu_util import host, say
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def fps_tol(n, D):
    K = n + D + 8
    return 2.0 * K * U / (1.0 - K * U)


def queries(H, n, D, dtype="bf16", seed=0, device="cuda", B=1):
    """[B, H, n, D] pre-RoPE queries around per-head centroids (the synthetic
    query recipe of the eviction workloads)."""
    w = synth.Workload("fps", B=B, Hq=H, Hkv=H, D=D, N=n, W=0, C=0, budget=1, dtype=dtype, n_centroids=8,
                       sigma=0.35)
    return synth.query_stream(w, n, seed=seed, device=device)


def check_against_oracle(q, picks, m, threads=8):
    """q [..., n, D] (host), picks [..., k] (host) for every head."""
    n, D = q.shape[-2], q.shape[-1]
    q3 = q.reshape(-1, n, D)
    g = picks.reshape(q3.shape[0], -1).numpy().astype(np.int32)
    k = min(m, n)
    assert g.shape[1] == k
    for h in range(g.shape[0]):
        assert len(set(g[h].tolist())) == k and g[h].min() >= 0 and g[h].max() < n
    tol = fps_tol(n, D)
    ref, tie = oracle.fps(q3, m, tie_tol=tol, threads=threads)
    exact_steps = 0
    for h in range(g.shape[0]):
        s = int(np.argmax(tie[h])) if tie[h].any() else k
        assert np.array_equal(g[h, :s], ref[h, :s]), f"head {h}: differs before the first near tie (step {s})"
        exact_steps += s
    oracle.fps(q3, m, forced=g, tie_tol=tol, threads=threads)  # ValueError if a pick leaves the band
    return exact_steps, g.size


def check_greedy_rule(q, picks, m):
    """The FPS rule in fp64 numpy for large sets, given the GPU's picks."""
    n, D = q.shape[-2], q.shape[-1]
    q3 = q.reshape(-1, n, D).float().double().numpy()
    g = picks.reshape(q3.shape[0], -1).numpy()
    tol = fps_tol(n, D)
    for h in range(q3.shape[0]):
        x = q3[h]
        nrm = np.linalg.norm(x, axis=1)
        u = np.divide(x, nrm[:, None], out=np.zeros_like(x), where=nrm[:, None] > 0)
        val = u @ u.mean(axis=0)
        picked = np.zeros(n, bool)
        for k in range(min(m, n)):
            r = int(g[h, k])
            assert 0 <= r < n and not picked[r]
            assert val[r] <= val[~picked].min() + tol, f"head {h} step {k}"
            picked[r] = True
            c = u @ u[r]
            val = c if k == 0 else np.maximum(val, c)


# ---- worked examples -------------------------------------------------------------
def _golden(key, D):
    fx = load("fps_hand_worked.txt")
    rows = np.array([[float(v) for v in r] for r in fx[key]], np.float32)
    q = np.zeros((1, rows.shape[0], D), np.float32)
    q[0, :, :2] = rows  # zero padding changes no cosine
    return q, fx


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_fps_hand_worked_example(dtype):
    tdt = torch.float32 if dtype == "fp32" else torch.bfloat16
    q, fx = _golden("query", 64)
    picks = bkv.fps(torch.from_numpy(q).to(tdt).cuda(), 4)
    assert host(picks)[0].tolist() == [int(v) for v in fx["picks"][0]]
    q, fx = _golden("tie_query", 128)
    picks = bkv.fps(torch.from_numpy(q).to(tdt).cuda(), 4)
    assert host(picks)[0].tolist() == [int(v) for v in fx["tie_picks"][0]]


@pytest.mark.parametrize("reps", [1, 17, 64, 256, 300, 8192])
def test_fps_repeated_axes_closed_form(reps):
    # rows 4i..4i+3 = e0, e1, -e0, -e1: every average cosine is exactly 0,
    # so the picks are 0 (lowest index), 2 (cos -1), 1 and 3 (S = 0, lowest
    # first), then the remaining rows in index order (all at S = 1).  This
    # runs every kernel: the Gram kernel (n <= 64), the register-resident
    # one (bf16, n <= 1024) and the streaming one, up to n = 32768.
    q, _ = _golden("tie_query", 128)
    n = 4 * reps
    x = torch.from_numpy(np.tile(q[0], (reps, 1))[None]).to(torch.bfloat16).cuda()
    m = min(n, 40)
    picks = host(bkv.fps(x, m))[0].tolist()
    expect = ([0, 2, 1, 3] + list(range(4, n)))[:m] if n > 4 else [0, 2, 1, 3]
    assert picks == expect


# ---- random sets against the oracle ---------------------------------------------
GRAM_CASES = [("bf16", 128, 32, 16, 37), ("bf16", 128, 64, 64, 8), ("bf16", 64, 17, 40, 9), ("fp32", 128, 48, 16, 5),
              ("fp32", 64, 1, 1, 3), ("bf16", 128, 5, 3, 4), ("fp32", 128, 33, 20, 6), ("bf16", 64, 16, 16, 2)]


@pytest.mark.parametrize("dtype,D,n,m,H", GRAM_CASES)
def test_fps_small_sets(dtype, D, n, m, H):
    q = queries(H, n, D, dtype, seed=n * 131 + D)
    picks = bkv.fps(q, m)
    torch.cuda.synchronize()
    ex, tot = check_against_oracle(host(q), host(picks), m)
    say(f"fps {dtype} D={D} n={n} m={m} H={H}: {ex}/{tot} picks exact before the first near tie")


# bf16 sets of 65 to 1024 rows run the register-resident kernel (16-row
# blocks, 1, 2, 4 or 8 per wave); fp32 sets and larger ones stream.
STREAM_CASES = [("bf16", 128, 65, 16, 6), ("bf16", 128, 200, 100, 3), ("fp32", 64, 1000, 16, 3),
                ("bf16", 128, 2500, 32, 2), ("bf16", 64, 4600, 16, 1), ("bf16", 128, 1024, 16, 4),
                ("bf16", 64, 777, 40, 3), ("bf16", 128, 513, 64, 2), ("bf16", 128, 129, 129, 2),
                ("bf16", 64, 400, 16, 3), ("fp32", 128, 1024, 16, 2)]


@pytest.mark.parametrize("dtype,D,n,m,H", STREAM_CASES)
def test_fps_large_sets(dtype, D, n, m, H):
    q = queries(H, n, D, dtype, seed=n * 7 + D)
    picks = bkv.fps(q, m)
    torch.cuda.synchronize()
    ex, tot = check_against_oracle(host(q), host(picks), m)
    say(f"fps {dtype} D={D} n={n} m={m} H={H}: {ex}/{tot} picks exact before the first near tie")


@pytest.mark.parametrize("n", [20000, 32768])
def test_fps_largest_sets_greedy_rule(n):
    q = queries(2, n, 128, "bf16", seed=n)
    picks = bkv.fps(q, 16)
    torch.cuda.synchronize()
    check_greedy_rule(host(q), host(picks), 16)


@pytest.mark.parametrize("n", [40, 300, 1000])
def test_fps_zero_and_duplicate_rows(n):
    q = queries(4, n, 128, "bf16", seed=5)
    g = torch.Generator(device="cpu").manual_seed(n)
    zero = torch.randperm(n, generator=g)[: n // 8]
    q[:, :, zero.cuda()] = 0
    src = torch.randperm(n, generator=g)[: n // 5]
    dst = torch.randperm(n, generator=g)[: n // 5]
    q[:, :, dst.cuda()] = q[:, :, src.cuda()]
    picks = bkv.fps(q, n // 2)
    torch.cuda.synchronize()
    check_against_oracle(host(q), host(picks), n // 2)


def test_fps_prefix_of_a_head_buffer():
    # only the first n of q_rows rows take part; rows past n are never read
    # for selection
    q = queries(5, 48, 128, "bf16", seed=11)
    qs = q.clone()
    qs[:, :, 30:] = float("nan")
    picks = bkv.fps(qs, 12, n=30)
    torch.cuda.synchronize()
    check_against_oracle(host(q[:, :, :30]).contiguous(), host(picks), 12)


def test_fps_empty_calls_leave_outputs():
    q = queries(3, 20, 64, "bf16")
    before = q.clone()
    dst = torch.full((1, 3, 8, 64), 2.0, device="cuda")
    counts = torch.full((1, 3, 8), 7, dtype=torch.int32, device="cuda")
    assert bkv.fps(q, 0).shape == (1, 3, 0)
    assert bkv.fps(q, 5, n=0).shape == (1, 3, 0)
    bkv.fps_gather(q, 0)
    bkv.fps_gather(q, 5, n=0, dst=dst, counts=counts)
    torch.cuda.synchronize()
    assert torch.equal(q, before)
    assert (host(dst) == 2.0).all() and (host(counts) == 7).all()


# ---- gather -------------------------------------------------------------------------
@pytest.mark.parametrize("n,m,D,dtype", [(32, 16, 128, "bf16"), (64, 64, 64, "fp32"), (300, 128, 128, "bf16"),
                                         (1000, 100, 64, "fp32"), (1024, 128, 128, "bf16"), (700, 33, 64, "bf16")])
def test_fps_gather_in_place(n, m, D, dtype):
    q = queries(24, n, D, dtype, seed=n + m)
    orig = host(q).clone()
    picks = torch.empty(1, 24, min(m, n), dtype=torch.int32, device="cuda")
    bkv.fps_gather(q, m, picks=picks)
    torch.cuda.synchronize()
    p = host(picks)
    check_against_oracle(orig, p, m)
    after = host(q)
    k = p.shape[-1]
    want = torch.gather(orig, 2, p.long().unsqueeze(-1).expand(-1, -1, -1, D))
    assert torch.equal(after[:, :, :k].view(torch.int16 if dtype == "bf16" else torch.int32),
                       want.view(torch.int16 if dtype == "bf16" else torch.int32))
    assert torch.equal(after[:, :, k:], orig[:, :, k:])


@pytest.mark.parametrize("n", [32, 150, 600])
def test_fps_gather_into_beacon_layout_feeds_scoring(n):
    # per-query-head FPS of a bf16 buffer [B, Hq, n, D], widened to fp32 into
    # [B, Hq, n_beacon, D] == [B, Hkv, G * n_beacon, D]: the group-level union
    # of beacon sets, with counts marking every slot occupied (n = 32 runs
    # the Gram kernel, 150 and 600 the register-resident one)
    B, Hq, Hkv, D, nb = 2, 8, 2, 128, 16
    G = Hq // Hkv
    buf = queries(Hq, n, D, "bf16", seed=3, B=B)
    beacons = torch.full((B, Hkv, G * nb, D), 5.0, device="cuda")
    counts = torch.full((B, Hkv, G * nb), -1, dtype=torch.int32, device="cuda")
    picks = torch.empty(B, Hq, nb, dtype=torch.int32, device="cuda")
    bkv.fps_gather(buf, nb, dst=beacons.view(B, Hq, nb, D), picks=picks, counts=counts.view(B, Hq, nb))
    torch.cuda.synchronize()
    p = host(picks)
    check_against_oracle(host(buf), p, nb)
    want = torch.gather(host(buf).float(), 2, p.long().unsqueeze(-1).expand(-1, -1, -1, D))
    assert torch.equal(host(beacons).view(B, Hq, nb, D), want)
    assert (host(counts) == 1).all()
    # the same beacons, built on the host, score identically
    w = synth.QWEN3_4B_4K.with_(B=B, Hq=Hq, Hkv=Hkv, N=1024, W=4, C=G * nb, budget=512)
    d = bkv.dims(B=B, Hq=Hq, Hkv=Hkv, D=D, N=1024, W=4, C=G * nb, budget=512)
    x = synth.make_layer(w, seed=9, device="cuda")
    ws = bkv.workspace(d, bkv.OP_SCORE)
    s1 = torch.empty(B, Hkv, 1024, device="cuda")
    s2 = torch.empty_like(s1)
    bkv.score(d, x["K"], x["q_win"], beacons, counts, s1, ws, rope_cos=x["rope_cos"], rope_sin=x["rope_sin"])
    bkv.score(d, x["K"], x["q_win"], want.view(B, Hkv, G * nb, D).cuda().contiguous(),
              torch.ones_like(counts), s2, ws, rope_cos=x["rope_cos"], rope_sin=x["rope_sin"])
    torch.cuda.synchronize()
    assert torch.equal(host(s1), host(s2))


def test_fps_gather_counts_partial():
    # fewer rows than slots: counts mark the first k, the rest stay untouched
    q = queries(6, 10, 64, "bf16", seed=2)
    dst = torch.full((1, 6, 16, 64), 3.0, device="cuda")
    counts = torch.full((1, 6, 16), 9, dtype=torch.int32, device="cuda")
    picks = torch.empty(1, 6, 10, dtype=torch.int32, device="cuda")
    bkv.fps_gather(q, 16, dst=dst, picks=picks, counts=counts)
    torch.cuda.synchronize()
    c = host(counts)
    assert (c[..., :10] == 1).all() and (c[..., 10:] == 0).all()
    assert (host(dst)[:, :, 10:] == 3.0).all()
    assert sorted(host(picks)[0, 0].tolist()) == list(range(10))


# ---- the workloads' own sizes ----------------------------------------------------------
def test_fps_continual_compress_full_size():
    # Qwen3-4B, 36 layers x 16 sequences x 32 query heads: every buffer of
    # B_Q^max = 32 pre-RoPE queries compressed to B_Q^min = 16 in one call
    H_b, layers = 16, 36
    w = synth.QWEN3_4B_32K
    buf = queries(w.Hq, 32, w.D, "bf16", seed=1, B=H_b * layers)
    orig = buf.clone()
    picks = torch.empty(H_b * layers, w.Hq, 16, dtype=torch.int32, device="cuda")
    say(f"continual compress: {H_b * layers * w.Hq} heads")
    bkv.fps_gather(buf, 16, picks=picks)
    torch.cuda.synchronize()
    want = torch.gather(orig, 2, picks.long().unsqueeze(-1).expand(-1, -1, -1, w.D))
    assert torch.equal(buf[:, :, :16].view(torch.int16), want.view(torch.int16))
    assert torch.equal(buf[:, :, 16:], orig[:, :, 16:])
    sample = torch.randperm(H_b * layers * w.Hq, generator=torch.Generator().manual_seed(0))[:96]
    qh = host(orig).reshape(-1, 32, w.D)[sample]
    ph = host(picks).reshape(-1, 16)[sample]
    ex, tot = check_against_oracle(qh, ph, 16)
    say(f"continual compress: {ex}/{tot} sampled picks exact before the first near tie")


@pytest.mark.parametrize("T", [1024, 4096])
def test_fps_prefill_initialisation_full_size(T):
    # prefill: FPS over a T-token prompt's pre-RoPE queries per query head
    # (B=16, Hq=32), the selection written into the heads' 32-row buffers
    # (1024 rows run the register-resident kernel, 4096 the streaming one)
    w = synth.QWEN3_4B_32K
    q = queries(w.Hq, T, w.D, "bf16", seed=2, B=16)
    obs = torch.zeros(16, w.Hq, 32, w.D, dtype=torch.bfloat16, device="cuda")
    picks = torch.empty(16, w.Hq, 16, dtype=torch.int32, device="cuda")
    bkv.fps_gather(q, 16, dst=obs, picks=picks)
    torch.cuda.synchronize()
    want = torch.gather(q, 2, picks.long().unsqueeze(-1).expand(-1, -1, -1, w.D))
    assert torch.equal(obs[:, :, :16].view(torch.int16), want.view(torch.int16))
    assert not obs[:, :, 16:].any()
    heads = [0, 511]
    qh = host(q).reshape(-1, T, w.D)[heads]
    ph = host(picks).reshape(-1, 16)[heads]
    ex, tot = check_against_oracle(qh, ph, 16, threads=2)
    say(f"prefill init: {ex}/{tot} sampled picks exact before the first near tie")
