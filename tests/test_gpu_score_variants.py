"""GPU parity of the scoring options (bkv_score_ex / bkv_evict_ex): Eq. (6)'s
mean form and causal recent queries, against the oracle on the same inputs.

Rules as for the max form: scores and row normalisers within 1e-3 in
natural-log units, kept indices under the tie-band rule, compacted rows
bit-exact where the kept index agrees.  The mean form is held to the same
1e-3 rule everywhere, also where every weight of a key lies far below the
fp32 range (the kernels sum weights relative to each key's largest)."""
import numpy as np
import pytest
import torch
from scipy.optimize import linprog

import oracle
from gpu_util import assert_rows_match, assert_scores_close, compare_kept, dims_of, host, say, to_dev
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth

pytestmark = pytest.mark.gpu

W = synth.Workload
CASES = {
    # fast path (bf16, R <= 144): ragged tail, an empty beacon slot
    "fast-d128": W("v1", B=2, Hq=8, Hkv=2, D=128, N=1000, W=8, C=4, budget=256, revisit_frac=0.1),
    # fast path at the benchmark's row count (R = 16 + 4*32 = 144), 1024-key items
    "fast-r144": W("v2", B=16, Hq=32, Hkv=8, D=128, N=8192, W=32, C=16, budget=1024, revisit_frac=0.05),
    # fast path, D = 64, odd group size
    "fast-d64-g7": W("v3", B=1, Hq=14, Hkv=2, D=64, N=777, W=5, C=3, budget=200, n_centroids=3),
    # generic path: fp32, and bf16 with R = 16 + 7*24 = 184 > 144 rows
    "generic-fp32": synth.TINY_FP32,
    "generic-bf16-r184": W("v4", B=1, Hq=14, Hkv=2, D=128, N=600, W=24, C=16, budget=300, n_centroids=16),
    # fewer keys than recent queries: the oldest recent rows see no key
    "fast-short": W("v5", B=1, Hq=4, Hkv=1, D=128, N=20, W=32, C=2, budget=64),
    "generic-short": W("v6", B=1, Hq=4, Hkv=1, D=64, N=20, W=32, C=2, budget=64, dtype="fp32"),
}
OPTIONS = [(True, False), (False, True), (True, True)]  # (mean, causal)


def _heads(w):
    return None if w.P <= 16 else [(b, h) for b in (0, w.B - 1) for h in (0, w.Hkv - 1)]


@pytest.mark.parametrize("mean,causal", OPTIONS)
@pytest.mark.parametrize("name", list(CASES))
def test_score_options_parity(name, mean, causal):
    w = CASES[name]
    x = synth.make_layer(w, seed=21, device="cpu")
    if name == "fast-d128":
        x["counts"][0, 1, 2] = 0
    d = dims_of(w)
    heads = _heads(w)
    say(f"score options mean={mean} causal={causal} {name} {d}")
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, rope_cos=x["rope_cos"],
                                  rope_sin=x["rope_sin"], heads=heads, threads=8, agg="mean" if mean else "max",
                                  causal=causal)
    xd = to_dev(x)
    ws = bkv.workspace(d, bkv.OP_SCORE)
    scores = torch.full((d.B, d.Hkv, d.N), float("nan"), device="cuda")
    lse = torch.full((d.B, d.Hkv, d.C + d.G * d.W), float("nan"), device="cuda")
    bkv.score(d, xd["K"], xd["q_win"], xd["beacons"], xd["counts"], scores, ws, row_lse=lse,
              rope_cos=xd["rope_cos"], rope_sin=xd["rope_sin"], mean=mean, causal=causal)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    s_gpu, lse_gpu = host(scores).numpy(), host(lse).numpy()
    sel = (slice(None),) if heads is None else tuple(np.array(heads).T)
    err = assert_scores_close(s_gpu[sel], s_ref[sel], "scores")
    assert_scores_close(lse_gpu[sel], lse_ref[sel], "row_lse")
    assert not np.isnan(s_gpu).any() and np.all(s_gpu <= 1e-4)
    say(f"  max |diff| {err:.2e}")


def test_options_differ_from_the_max_form():
    # the options change the scores where they should, and only there
    w = CASES["fast-d128"]
    x = to_dev(synth.make_layer(w, seed=5, device="cpu"))
    d = dims_of(w)
    ws = bkv.workspace(d, bkv.OP_SCORE)
    out = {}
    for key in [(False, False), (True, False), (False, True)]:
        s = torch.empty(d.B, d.Hkv, d.N, device="cuda")
        bkv.score(d, x["K"], x["q_win"], x["beacons"], x["counts"], s, ws, rope_cos=x["rope_cos"],
                  rope_sin=x["rope_sin"], mean=key[0], causal=key[1])
        out[key] = host(s).numpy()
    base = out[(False, False)]
    assert np.all(out[(True, False)] <= base + 1e-4)  # mean <= max
    R = w.C + w.G * w.W
    assert np.all(out[(True, False)] >= base - np.log(R) - 1e-3)
    # causal: keys before N - W + 1 keep their max-form scores only if no
    # recent row's normaliser changed; the normalisers of the older recent
    # rows shrink, so scores can only rise there
    assert not np.array_equal(out[(False, True)], base)


@pytest.mark.parametrize("mean,causal", OPTIONS)
def test_evict_options_parity(mean, causal):
    w = W("v7", B=2, Hq=8, Hkv=2, D=128, N=3000, W=16, C=8, budget=700, n_prefix=4, revisit_frac=0.1)
    x = synth.make_layer(w, seed=31, device="cpu")
    d = dims_of(w)
    ref = oracle.evict(x["K"], x["V"], x["q_win"], x["beacons"], x["counts"], N=w.N, budget=w.budget, W=w.W,
                       n_prefix=w.n_prefix, rope_cos=x["rope_cos"], rope_sin=x["rope_sin"], threads=4,
                       agg="mean" if mean else "max", causal=causal)
    xd = to_dev(x)
    ws = bkv.workspace(d, bkv.OP_EVICT)
    kept = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    scores = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    bkv.evict(d, xd["K"], xd["V"], xd["q_win"], xd["beacons"], xd["counts"], ws, kept=kept, scores=scores,
              rope_cos=xd["rope_cos"], rope_sin=xd["rope_sin"], mean=mean, causal=causal)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    assert_scores_close(host(scores).numpy(), ref["scores"], "scores")
    kg = host(kept).numpy()
    band, diff = compare_kept(kg, ref["kept"], ref["scores"], w.N, w.W, w.n_prefix, w.budget)
    say(f"evict mean={mean} causal={causal}: tie band {band}, {diff} in-band differences")
    assert_rows_match(xd["K"], ref["K"], kg, ref["kept"], d.n_keep, "K")
    assert_rows_match(xd["V"], ref["V"], kg, ref["kept"], d.n_keep, "V")


DEEP = {
    "fast-bf16": W("v8", B=2, Hq=8, Hkv=2, D=128, N=1500, W=8, C=4, budget=400),
    "generic-fp32": W("v9", B=1, Hq=8, Hkv=2, D=64, N=700, W=16, C=4, budget=200, dtype="fp32"),
    "fast-bf16-r184": CASES["generic-bf16-r184"],  # rows in two register groups
}


def _away(y):
    """Unit vector whose dot product with every row of y is negative: the
    k (|k_i| <= 1) that pushes the largest normalised dot product furthest
    below 0, by linear programming."""
    yn = y / np.linalg.norm(y, axis=1, keepdims=True)
    R, D = yn.shape
    res = linprog(np.r_[np.zeros(D), 1.0], A_ub=np.c_[yn, -np.ones(R)], b_ub=np.zeros(R),
                  bounds=[(-1, 1)] * D + [(None, None)], method="highs")
    assert res.status == 0 and res.x[D] < 0, "no direction away from every row"
    k = res.x[:D]
    return k / np.linalg.norm(k)


@pytest.mark.parametrize("name", list(DEEP))
def test_mean_form_far_below_fp32_range(name):
    # keys pointing away from every observation row, with logits near -300
    # for every row: all their weights lie far below 2^-126, yet the mean
    # form's log-score is finite and matches the oracle within the same 1e-3
    # (no rotation, so the rows are the beacons and window queries as given)
    w = DEEP[name]
    x = synth.make_layer(w, seed=41, device="cpu")
    K = x["K"].float()
    deep = np.r_[3:40, w.N - w.W - 6:w.N - w.W]
    for b in range(w.B):
        for h in range(w.Hkv):
            rows = [x["q_win"][b, h * w.G + g].float() for g in range(w.G)]
            rows.append(x["beacons"][b, h][x["counts"][b, h] > 0].to(x["K"].dtype).float())
            y = torch.cat(rows).double().numpy()
            k = _away(y)
            K[b, h, deep] = torch.from_numpy(k * (300.0 * np.sqrt(w.D) / -(y @ k).max())).float()
    x["K"] = K.to(x["K"].dtype).contiguous()
    d = dims_of(w)
    s_ref, lse_ref = oracle.score(x["K"], x["q_win"], x["beacons"], x["counts"], N=w.N, threads=4, agg="mean")
    assert np.all(s_ref[..., deep] < -200.0), "the planted keys are not below the fp32 range"
    xd = to_dev(x)
    ws = bkv.workspace(d, bkv.OP_SCORE)
    scores = torch.full((d.B, d.Hkv, d.N), float("nan"), device="cuda")
    lse = torch.full((d.B, d.Hkv, d.C + d.G * d.W), float("nan"), device="cuda")
    say(f"mean form, deep keys, {name} {d}")
    bkv.score(d, xd["K"], xd["q_win"], xd["beacons"], xd["counts"], scores, ws, row_lse=lse, mean=True)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    s_gpu = host(scores).numpy()
    assert np.isfinite(s_gpu).all()
    err = assert_scores_close(s_gpu, s_ref, "scores")
    assert_scores_close(host(lse).numpy(), lse_ref, "row_lse")
    say(f"  max |diff| {err:.2e}, deepest {s_ref[..., deep].min():.1f}")
