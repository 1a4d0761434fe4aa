"""GPU parity of the row-split score items: heads whose observation rows span
four register groups of 7 to 9 row tiles (R of about 430 to 576, e.g. the
Qwen2.5-7B shape with R = 16 + 7*64 = 464 and the Llama-8B shape with
R = 32 + 4*128 = 544).  There each of a work item's four waves holds one
row group and all four share one stream of the item's keys.

Every case checks scores and row normalisers against the oracle within
1e-3 (natural-log units) on every head, for the max and mean forms
(Eq. 6) with and without causal recent rows, across ragged key counts
(a last item shorter than one 128-key super-stage, fewer keys than recent
queries), D = 64 and 128; plus a key far above the first keys of its
lanes (the statistics redone with a running max), keys whose weights all
lie below the fp32 range (mean form).  The fused eviction on such heads is
covered with the other fused cases."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_scores_close, dims_of, host, say, to_dev
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth

pytestmark = pytest.mark.gpu

W = synth.Workload
# R = C + G W; tiles = ceil(R / 16) in 28..36 gives four groups of 7..9 tiles
CASES = {
    # R = 464: 29 tiles -> 4 groups of 8; three items, the last of 52 keys
    "d128-r464": W("s1", B=1, Hq=28, Hkv=4, D=128, N=2100, W=64, C=16, budget=512, n_centroids=16, zipf=1.2),
    # R = 544: 34 tiles -> 4 groups of 9 (two padding tiles)
    "d128-r544": W("s2", B=1, Hq=8, Hkv=2, D=128, N=3000, W=128, C=32, budget=800, n_centroids=32),
    # D = 64, R = 444: 28 tiles -> 4 groups of 7
    "d64-r444": W("s3", B=2, Hq=8, Hkv=2, D=64, N=1100, W=107, C=16, budget=300, n_centroids=8),
    # fewer keys than one super-stage and than the recent window
    "short": W("s4", B=1, Hq=8, Hkv=2, D=128, N=100, W=128, C=32, budget=160),
}
OPTIONS = [(False, False), (True, False), (False, True), (True, True)]  # (mean, causal)


def _score(w, x, mean=False, causal=False, rope=True):
    d = dims_of(w)
    xd = to_dev(x)
    ws = bkv.workspace(d, bkv.OP_SCORE)
    scores = torch.full((d.B, d.Hkv, d.N), float("nan"), device="cuda")
    lse = torch.full((d.B, d.Hkv, d.C + d.G * d.W), float("nan"), device="cuda")
    kw = dict(rope_cos=xd["rope_cos"], rope_sin=xd["rope_sin"]) if rope else {}
    bkv.score(d, xd["K"], xd["q_win"], xd["beacons"], xd["counts"], scores, ws, row_lse=lse, mean=mean,
              causal=causal, **kw)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    return host(scores).numpy(), host(lse).numpy()


@pytest.mark.parametrize("mean,causal", OPTIONS)
@pytest.mark.parametrize("name", list(CASES))
def test_split_score_parity(name, mean, causal):
    w = CASES[name]
    x = synth.make_layer(w, seed=61, device="cpu")
    x["counts"][0, 0, 1] = 0  # an empty beacon slot: one row fewer
    say(f"row-split score mean={mean} causal={causal} {name} {dims_of(w)}")
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, rope_cos=x["rope_cos"],
                                  rope_sin=x["rope_sin"], threads=8, agg="mean" if mean else "max",
                                  causal=causal)
    s_gpu, lse_gpu = _score(w, x, mean, causal)
    err = assert_scores_close(s_gpu, s_ref, "scores")
    assert_scores_close(lse_gpu, lse_ref, "row_lse")
    assert not np.isnan(s_gpu).any() and np.all(s_gpu <= 1e-4)
    say(f"  max |diff| {err:.2e}")


@pytest.mark.parametrize("mean", [False, True])
def test_split_key_far_above_its_lanes_first_keys(mean):
    # a key ~300 nats above every other key of one recent row, planted after
    # an item's first group: that row's offset-relative sum overflows and the
    # wave redoes its statistics with a running max
    w = CASES["d128-r544"]
    x = synth.make_layer(w, seed=17, device="cpu")
    K = x["K"].float()
    for h in range(w.Hkv):
        y = x["q_win"][0, h * w.G].float()[0]
        for j in (100, 1500 + 40 * h, 2999):
            K[0, h, j] = 300.0 * np.sqrt(w.D) * y / y.norm() ** 2
    x["K"] = K.to(torch.bfloat16).contiguous()
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, rope_cos=x["rope_cos"],
                                  rope_sin=x["rope_sin"], threads=4, agg="mean" if mean else "max")
    assert lse_ref[..., w.C].max() > 250.0, "the planted keys do not dominate their row"
    say(f"row-split score, dominant key, mean={mean}")
    s_gpu, lse_gpu = _score(w, x, mean)
    err = assert_scores_close(s_gpu, s_ref, "scores")
    assert_scores_close(lse_gpu, lse_ref, "row_lse")
    say(f"  max |diff| {err:.2e}")


@pytest.mark.parametrize("mean", [False, True])
def test_split_offsets_far_apart_between_chunks(mean):
    # one recent row sees a key of ~104 nats in the first group of one item
    # and its largest key, ~131 nats, deep inside a later item whose first
    # keys are ordinary: the first item's offset then lies more than 126
    # (log2 units) above the second's, whose sum is still far from overflow;
    # merging the two must not lose the second item's sum
    w = CASES["d128-r544"]
    x = synth.make_layer(w, seed=19, device="cpu")
    K = x["K"].float()
    for h in range(w.Hkv):
        y = x["q_win"][0, h * w.G].float()[0]
        for j, nats in ((1024 + 5, 104.0), (2048 + 700, 131.0)):
            K[0, h, j] = nats * np.sqrt(w.D) * y / y.norm() ** 2
    x["K"] = K.to(torch.bfloat16).contiguous()
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, rope_cos=x["rope_cos"],
                                  rope_sin=x["rope_sin"], threads=4, agg="mean" if mean else "max")
    assert lse_ref[..., w.C].max() > 120.0, "the planted keys do not dominate their row"
    say(f"row-split score, offsets far apart between items, mean={mean}")
    s_gpu, lse_gpu = _score(w, x, mean)
    err = assert_scores_close(s_gpu, s_ref, "scores")
    assert_scores_close(lse_gpu, lse_ref, "row_lse")
    assert np.all(s_gpu <= 1e-4)
    say(f"  max |diff| {err:.2e}")


def _away(y):
    """Unit vector whose dot product with every row of y is negative (linear
    programming: push the largest normalised dot product furthest below 0)."""
    from scipy.optimize import linprog
    yn = y / np.linalg.norm(y, axis=1, keepdims=True)
    R, D = yn.shape
    res = linprog(np.r_[np.zeros(D), 1.0], A_ub=np.c_[yn, -np.ones(R)], b_ub=np.zeros(R),
                  bounds=[(-1, 1)] * D + [(None, None)], method="highs")
    assert res.status == 0 and res.x[D] < 0, "no direction away from every row"
    return res.x[:D] / np.linalg.norm(res.x[:D])


def test_split_mean_form_far_below_fp32_range():
    # keys pointing away from every row with logits near -300: their mean
    # weights lie far below 2^-126, their log-scores stay finite and match
    w = CASES["d128-r464"]
    x = synth.make_layer(w, seed=41, device="cpu")
    K = x["K"].float()
    deep = np.r_[3:40, 1500:1530]
    for h in range(w.Hkv):
        rows = [x["q_win"][0, h * w.G + g].float() for g in range(w.G)]
        rows.append(x["beacons"][0, h][x["counts"][0, h] > 0].to(x["K"].dtype).float())
        y = torch.cat(rows).double().numpy()
        k = _away(y)
        K[0, h, deep] = torch.from_numpy(k * (300.0 * np.sqrt(w.D) / -(y @ k).max())).float()
    x["K"] = K.to(x["K"].dtype).contiguous()
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, threads=4, agg="mean")
    assert np.all(s_ref[..., deep] < -200.0), "the planted keys are not below the fp32 range"
    say("row-split score, mean form, deep keys")
    s_gpu, lse_gpu = _score(w, x, mean=True, rope=False)
    assert np.isfinite(s_gpu).all()
    err = assert_scores_close(s_gpu, s_ref, "scores")
    assert_scores_close(lse_gpu, lse_ref, "row_lse")
    say(f"  max |diff| {err:.2e}")
