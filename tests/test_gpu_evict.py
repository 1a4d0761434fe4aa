"""End-to-end GPU parity of bkv_evict (score -> select -> compact) against the
oracle, on the tiny and Qwen3-4B-shaped configurations and edge cases."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_rows_match, assert_scores_close, compare_kept, dims_of, host, say, to_dev
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth

pytestmark = pytest.mark.gpu

W = synth.Workload
CASES = {
    "tiny-fp32": (synth.TINY_FP32, 0),
    "qwen3-4b-layer-4k": (synth.QWEN3_4B_4K, 0),
    "prefix-kept": (W("e1", B=2, Hq=8, Hkv=2, D=128, N=1500, W=16, C=6, budget=400, revisit_frac=0.1), 7),
    "gqa7-d64": (W("e2", B=1, Hq=28, Hkv=4, D=64, N=2100, W=9, C=16, budget=512, n_centroids=16, zipf=1.2), 0),
    "n-below-budget": (W("e3", B=1, Hq=4, Hkv=2, D=128, N=90, W=8, C=4, budget=100), 0),
    "only-forced": (W("e4", B=1, Hq=4, Hkv=2, D=128, N=900, W=60, C=4, budget=64), 4),
    # chained calls with the selection split over several workgroups per head:
    # an fp32 layer (generic score path) and a bf16 head past 32K tokens
    "split-select-fp32": (W("e5", B=1, Hq=8, Hkv=2, D=64, N=12000, W=16, C=4, budget=1500, dtype="fp32"), 2),
    "split-select-40k": (W("e6", B=1, Hq=8, Hkv=2, D=128, N=40000, W=32, C=8, budget=5000, revisit_frac=0.05), 0),
}


def _evict(w, x, d, with_outputs=True):
    ws = bkv.workspace(d, bkv.OP_EVICT)
    kept = torch.full((d.B, d.Hkv, d.n_keep), -1, dtype=torch.int32, device="cuda") if with_outputs else None
    scores = torch.empty(d.B, d.Hkv, d.N, device="cuda") if with_outputs else None
    lse = torch.empty(d.B, d.Hkv, d.C + d.G * d.W, device="cuda") if with_outputs else None
    bkv.evict(d, x["K"], x["V"], x["q_win"], x["beacons"], x["counts"], ws, kept=kept, scores=scores, row_lse=lse,
              rope_cos=x["rope_cos"], rope_sin=x["rope_sin"])
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    return kept, scores, lse


@pytest.mark.parametrize("name", list(CASES))
def test_evict_parity(name):
    w, n_prefix = CASES[name]
    w = w.with_(n_prefix=n_prefix)
    x = synth.make_layer(w, seed=21)
    d = dims_of(w)
    say(f"evict {name} {d}")
    ref = oracle.evict(x["K"], x["V"], x["q_win"], x["beacons"], x["counts"], N=w.N, budget=w.budget, W=w.W,
                       n_prefix=n_prefix, rope_cos=x["rope_cos"], rope_sin=x["rope_sin"], threads=8)
    xd = to_dev(x)
    kept, scores, lse = _evict(w, xd, d)
    assert_scores_close(host(scores).numpy(), ref["scores"])
    assert_scores_close(host(lse).numpy(), ref["row_lse"], "row_lse")
    kg = host(kept).numpy()
    band, diff = compare_kept(kg, ref["kept"], ref["scores"], w.N, w.W, n_prefix, w.budget)
    say(f"evict {name}: tie band {band} candidates, {diff} in-band differences")
    assert_rows_match(xd["K"], ref["K"], kg, ref["kept"], d.n_keep, "K")
    assert_rows_match(xd["V"], ref["V"], kg, ref["kept"], d.n_keep, "V")
    # rows past the kept prefix are untouched
    assert torch.equal(host(xd["K"])[..., d.n_keep:, :], x["K"][..., d.n_keep:, :])


def test_evict_equals_chained_ops_and_optional_outputs():
    w = CASES["prefix-kept"][0].with_(n_prefix=3)
    x = synth.make_layer(w, seed=22)
    d = dims_of(w)
    a, b = to_dev(x), to_dev(x)
    say("evict without optional outputs")
    _evict(w, a, d, with_outputs=False)
    say("score + topk + compact chained")
    ws = bkv.workspace(d, bkv.OP_EVICT)
    sc = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    kept = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    bkv.score(d, b["K"], b["q_win"], b["beacons"], b["counts"], sc, ws, rope_cos=b["rope_cos"],
              rope_sin=b["rope_sin"])
    bkv.topk(d, sc, kept)
    bkv.compact(d, b["K"], b["V"], kept, ws)
    torch.cuda.synchronize()
    assert torch.equal(a["K"].view(torch.int16), b["K"].view(torch.int16))
    assert torch.equal(a["V"].view(torch.int16), b["V"].view(torch.int16))


def test_evict_invariants_repeated_calls():
    # steady-state use: evict, append tokens, evict again on the same buffers
    w = W("e5", B=2, Hq=8, Hkv=2, D=128, N=1200, W=16, C=8, budget=1024, revisit_frac=0.05)
    d0 = dims_of(w, N_cap=1200)
    x = to_dev(synth.make_layer(w, seed=23))
    ws = bkv.workspace(d0, bkv.OP_EVICT)
    N = 1200
    for it in range(4):
        d = dims_of(w, N=N, N_cap=1200)
        kept = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
        say(f"evict repeated it={it} N={N}")
        bkv.evict(d, x["K"], x["V"], x["q_win"], x["beacons"], x["counts"], ws, kept=kept,
                  rope_cos=x["rope_cos"], rope_sin=x["rope_sin"])
        k = host(kept).numpy()
        assert k.shape[-1] == min(w.budget, N)
        assert np.all(np.diff(k, axis=-1) > 0)
        assert np.all(k[..., -w.W:] == np.arange(N - w.W, N))  # recent window retained
        N = min(w.budget, N) + 176  # append 176 new tokens (they are already in the buffer)
    assert bkv.device_status(ws) == bkv.OK


def test_workspace_stamp_mismatch_is_reported_not_run():
    w = CASES["prefix-kept"][0]
    x = to_dev(synth.make_layer(w, seed=24))
    d = dims_of(w)
    ws = bkv.workspace(d, bkv.OP_EVICT)
    other = d.replace(budget=d.budget - 1)  # control block stamped for a different budget
    K0 = x["K"].clone()
    say("evict with a workspace stamped for other dims")
    bkv.evict(other, x["K"], x["V"], x["q_win"], x["beacons"], x["counts"], ws, rope_cos=x["rope_cos"],
              rope_sin=x["rope_sin"])
    assert bkv.device_status(ws) == bkv.ERR_DEVICE
    assert torch.equal(x["K"].view(torch.int16), K0.view(torch.int16))  # nothing was compacted
    bkv.workspace_init(d, ws)
    assert bkv.device_status(ws) == bkv.OK
