"""GPU parity of bkv_score (observation rows + scores) against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_scores_close, dims_of, host, say, to_dev
from paper_2609_04971_amd import synth

pytestmark = pytest.mark.gpu

W = synth.Workload
CASES = {
    # the tiny fp32 configuration, in full
    "tiny-fp32": synth.TINY_FP32,
    # bf16, D=128, several chunks and a ragged tail, one empty beacon slot
    "bf16-d128-ragged": W("c1", B=2, Hq=8, Hkv=2, D=128, N=1000, W=8, C=4, budget=256, revisit_frac=0.1),
    # D=64, odd group size G=7, N not a multiple of 16
    "bf16-d64-g7": W("c2", B=1, Hq=14, Hkv=2, D=64, N=777, W=5, C=3, budget=200, n_centroids=3),
    # rows spill over one LDS row group (R = 16 + 7*24 = 184 > 160)
    "bf16-two-row-groups": W("c3", B=1, Hq=14, Hkv=2, D=128, N=600, W=24, C=16, budget=300, n_centroids=16),
    # fp32 with R = 8 + 4*20 = 88 > 80 rows per group, D=128
    "fp32-two-row-groups": W("c4", B=1, Hq=8, Hkv=2, D=128, N=300, W=20, C=8, budget=100, dtype="fp32"),
    # beacons only (W = 0) and recent only (C = 0)
    "beacons-only": W("c5", B=2, Hq=4, Hkv=2, D=128, N=513, W=0, C=8, budget=64),
    "recent-only": W("c6", B=2, Hq=4, Hkv=2, D=128, N=513, W=16, C=0, budget=64),
    # a single cached token
    "one-token": W("c7", B=1, Hq=4, Hkv=1, D=128, N=1, W=4, C=2, budget=8),
    # many heads: the 1024-key work items (P * N/1024 >= 2048)
    "big-chunks": W("c8", B=16, Hq=32, Hkv=8, D=128, N=16384, W=32, C=8, budget=2048, revisit_frac=0.05),
}


def _run(w, x, d, rope=True, scale=0.0):
    import paper_2609_04971_amd as bkv
    ws = bkv.workspace(d, bkv.OP_SCORE)
    scores = torch.full((d.B, d.Hkv, d.N), float("nan"), device="cuda")
    lse = torch.full((d.B, d.Hkv, d.C + d.G * d.W), float("nan"), device="cuda")
    bkv.score(d, x["K"], x["q_win"], x["beacons"], x["counts"], scores, ws, row_lse=lse,
              rope_cos=x["rope_cos"] if rope else None, rope_sin=x["rope_sin"] if rope else None, scale=scale)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    return host(scores).numpy(), host(lse).numpy()


@pytest.mark.parametrize("name", list(CASES))
def test_score_parity(name):
    w = CASES[name]
    big = w.P * w.N > 1 << 20
    x = synth.make_layer(w, seed=11, device="cuda" if big else "cpu")
    if big:
        x = {k: host(v) for k, v in x.items()}
    if name == "bf16-d128-ragged":
        x["counts"][0, 1, 2] = 0          # an empty slot ...
        x["beacons"][0, 1, 2] = float("nan")  # ... whose vector must never be read
    d = dims_of(w)
    say(f"score {name} {d}")
    heads = None
    if w.P > 16:
        heads = [(b, h) for b in (0, w.B - 1) for h in (0, w.Hkv - 1)]
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, rope_cos=x["rope_cos"],
                                  rope_sin=x["rope_sin"], heads=heads, threads=8)
    s_gpu, lse_gpu = _run(w, to_dev(x), d)
    sel = (slice(None),) if heads is None else tuple(np.array(heads).T)
    assert_scores_close(s_gpu[sel], s_ref[sel])
    assert_scores_close(lse_gpu[sel], lse_ref[sel], "row_lse")
    assert np.all(s_gpu <= 1e-4)  # log of a probability


def test_score_no_rope_and_explicit_scale():
    w = CASES["bf16-d128-ragged"]
    x = synth.make_layer(w, seed=12)
    d = dims_of(w)
    say("score no-rope scale=0.05")
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, scale=0.05)
    s_gpu, lse_gpu = _run(w, to_dev(x), d, rope=False, scale=0.05)
    assert_scores_close(s_gpu, s_ref)
    assert_scores_close(lse_gpu, lse_ref, "row_lse")


def test_score_no_rows_gives_minus_inf():
    w = W("c9", B=1, Hq=2, Hkv=1, D=64, N=100, W=0, C=2, budget=10)
    x = synth.make_layer(w, seed=13)
    x["counts"].zero_()
    d = dims_of(w)
    say("score all slots empty, W=0")
    s_gpu, lse_gpu = _run(w, to_dev(x), d)
    assert np.all(np.isneginf(s_gpu)) and np.all(np.isneginf(lse_gpu))


def test_score_cache_stride_larger_than_n():
    w = CASES["bf16-d64-g7"]
    x = synth.make_layer(w, seed=14, N_cap=w.N + 333)
    d = dims_of(w, N_cap=w.N + 333)
    say(f"score N_cap>N {d}")
    s_ref, _ = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, rope_cos=x["rope_cos"],
                            rope_sin=x["rope_sin"])
    s_gpu, _ = _run(w, to_dev(x), d)
    assert_scores_close(s_gpu, s_ref)


def test_score_workspace_reused_across_lengths():
    # one initialised workspace serves calls with different N (same B*Hkv, budget)
    import paper_2609_04971_amd as bkv
    w = CASES["bf16-d128-ragged"]
    x = to_dev(synth.make_layer(w, seed=15))
    d_big = dims_of(w)
    ws = bkv.workspace(d_big, bkv.OP_SCORE)
    for N in (1000, 700, 1000, 65):
        d = dims_of(w, N=N, N_cap=w.N)
        say(f"score reuse N={N}")
        sc = torch.empty(d.B, d.Hkv, N, device="cuda")
        bkv.score(d, x["K"], x["q_win"], x["beacons"], x["counts"], sc, ws, rope_cos=x["rope_cos"],
                  rope_sin=x["rope_sin"])
        s_ref, _ = oracle.score(host(x["K"]), host(x["q_win"]), host(x["beacons"]), host(x["counts"]), N=N,
                                rope_cos=host(x["rope_cos"]), rope_sin=host(x["rope_sin"]))
        assert_scores_close(host(sc).numpy(), s_ref)
    assert bkv.device_status(ws) == bkv.OK


def test_score_deterministic():
    import paper_2609_04971_amd as bkv
    w = CASES["big-chunks"].with_(B=4)
    x = to_dev(synth.make_layer(w, seed=16))
    d = dims_of(w)
    ws = bkv.workspace(d, bkv.OP_SCORE)
    outs = []
    for _ in range(3):
        say("score determinism")
        sc = torch.empty(d.B, d.Hkv, d.N, device="cuda")
        bkv.score(d, x["K"], x["q_win"], x["beacons"], x["counts"], sc, ws, rope_cos=x["rope_cos"],
                  rope_sin=x["rope_sin"])
        outs.append(host(sc))
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[2])


@pytest.mark.parametrize("mean", [False, True])
def test_score_offsets_far_apart_between_chunks(mean):
    # one recent row sees a key of ~104 nats in the first group of one work
    # item and its largest key, ~131 nats, inside a later item whose first
    # keys are ordinary: the items' offsets lie more than 126 (log2 units)
    # apart while the later item's sum is far from overflow; merging their
    # statistics must keep the later sum
    import paper_2609_04971_amd as bkv
    w = W("c10", B=2, Hq=8, Hkv=2, D=128, N=3000, W=8, C=4, budget=500)
    x = synth.make_layer(w, seed=23, device="cpu")
    K = x["K"].float()
    for b in range(w.B):
        for h in range(w.Hkv):
            y = x["q_win"][b, h * w.G].float()[0]
            for j, nats in ((256 + 3, 104.0), (1024 + 170, 131.0)):
                K[b, h, j] = nats * np.sqrt(w.D) * y / y.norm() ** 2
    x["K"] = K.to(torch.bfloat16).contiguous()
    d = dims_of(w)
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, rope_cos=x["rope_cos"],
                                  rope_sin=x["rope_sin"], threads=4, agg="mean" if mean else "max")
    assert lse_ref[..., w.C].max() > 120.0, "the planted keys do not dominate their row"
    xd = to_dev(x)
    ws = bkv.workspace(d, bkv.OP_SCORE)
    scores = torch.full((d.B, d.Hkv, d.N), float("nan"), device="cuda")
    lse = torch.full((d.B, d.Hkv, d.C + d.G * d.W), float("nan"), device="cuda")
    say(f"score with offsets far apart between items, mean={mean}: {d}")
    bkv.score(d, xd["K"], xd["q_win"], xd["beacons"], xd["counts"], scores, ws, row_lse=lse,
              rope_cos=xd["rope_cos"], rope_sin=xd["rope_sin"], mean=mean)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    err = assert_scores_close(host(scores).numpy(), s_ref)
    assert_scores_close(host(lse).numpy(), lse_ref, "row_lse")
    say(f"  max |diff| {err:.2e}")


@pytest.mark.parametrize("mean", [False, True])
def test_score_key_far_above_its_lanes_first_keys(mean):
    # a key whose logit for a row lies ~300 nats above everything else: it is
    # not among the first keys a wave sees in its work item, so the row's
    # running sum overflows against the offset taken from those first keys
    # and the statistics are redone with a running max; scores and row
    # normalisers must still match the oracle within 1e-3
    import paper_2609_04971_amd as bkv
    w = W("c9", B=2, Hq=8, Hkv=2, D=128, N=3000, W=8, C=4, budget=500)
    x = synth.make_layer(w, seed=17, device="cpu")
    K = x["K"].float()
    for b in range(w.B):
        for h in range(w.Hkv):
            y = x["q_win"][b, h * w.G].float()[0]  # one recent row of the head
            for j in (100, 1500 + 40 * h, 2999):
                K[b, h, j] = 300.0 * np.sqrt(w.D) * y / y.norm() ** 2
    x["K"] = K.to(torch.bfloat16).contiguous()
    d = dims_of(w)
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, rope_cos=x["rope_cos"],
                                  rope_sin=x["rope_sin"], threads=4, agg="mean" if mean else "max")
    assert lse_ref[..., w.C].max() > 250.0, "the planted keys do not dominate their row"
    xd = to_dev(x)
    ws = bkv.workspace(d, bkv.OP_SCORE)
    scores = torch.full((d.B, d.Hkv, d.N), float("nan"), device="cuda")
    lse = torch.full((d.B, d.Hkv, d.C + d.G * d.W), float("nan"), device="cuda")
    say(f"score with a dominant key, mean={mean}: {d}")
    bkv.score(d, xd["K"], xd["q_win"], xd["beacons"], xd["counts"], scores, ws, row_lse=lse,
              rope_cos=xd["rope_cos"], rope_sin=xd["rope_sin"], mean=mean)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    err = assert_scores_close(host(scores).numpy(), s_ref)
    assert_scores_close(host(lse).numpy(), lse_ref, "row_lse")
    say(f"  max |diff| {err:.2e}")
