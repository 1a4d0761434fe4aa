"""GPU test of bkv_evict_noalloc, the eviction that allocates nothing: its
workspace is the library's fixed device array.  Checked against
bkv_evict_ex (the same eviction with a caller workspace) on the same inputs:
kept indices and compacted K/V bit-exact, scores within 1e-3 (the same
kernels run, so they agree exactly in practice).  Two calls in a row, the
second with a smaller input, so that the second finds the first's contents
in the array."""
import numpy as np
import pytest
import torch

from gpu_util import assert_scores_close, dims_of, raw_bits, say
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth

pytestmark = pytest.mark.gpu

W = synth.Workload
BIG = W("na-big", B=4, Hq=32, Hkv=8, D=128, N=8192, W=32, C=16, budget=1024, revisit_frac=0.05)
SMALL = W("na-small", B=2, Hq=8, Hkv=2, D=128, N=3000, W=16, C=8, budget=700, n_prefix=4, revisit_frac=0.1)


def _both(w, seed, mean=False, causal=False, outputs=True):
    d = dims_of(w)
    x = synth.make_layer(w, seed=seed, device="cuda")
    rope = dict(rope_cos=x["rope_cos"], rope_sin=x["rope_sin"], mean=mean, causal=causal)
    # the existing entry point, with a workspace of its own
    Kr, Vr = x["K"].clone(), x["V"].clone()
    ws = bkv.workspace(d, bkv.OP_EVICT)
    kept_r = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    scores_r = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    bkv.evict(d, Kr, Vr, x["q_win"], x["beacons"], x["counts"], ws, kept=kept_r, scores=scores_r, **rope)
    assert bkv.device_status(ws) == bkv.OK
    # the no-allocation entry point on a copy of the same inputs
    K, V = x["K"], x["V"]
    kept = torch.full((d.B, d.Hkv, d.n_keep), -1, dtype=torch.int32, device="cuda") if outputs else None
    scores = torch.full((d.B, d.Hkv, d.N), float("nan"), device="cuda") if outputs else None
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    say(f"no-alloc evict {w.name} mean={mean} causal={causal} outputs={outputs}: {d}")
    bkv.evict_noalloc(d, K, V, x["q_win"], x["beacons"], x["counts"], kept=kept, scores=scores, status=status,
                      **rope)
    torch.cuda.synchronize()
    assert int(status.item()) == bkv.OK
    if outputs:
        err = assert_scores_close(scores.cpu().numpy(), scores_r.cpu().numpy())
        np.testing.assert_array_equal(kept.cpu().numpy(), kept_r.cpu().numpy())
        say(f"  max |score diff| {err:.2e}")
    n = d.n_keep
    assert np.array_equal(raw_bits(K)[..., :n, :], raw_bits(Kr)[..., :n, :])
    assert np.array_equal(raw_bits(V)[..., :n, :], raw_bits(Vr)[..., :n, :])


def test_noalloc_two_calls_second_smaller():
    _both(BIG, seed=61)
    _both(SMALL, seed=62)


def test_noalloc_options_and_internal_outputs():
    # scoring options, and scores / kept left to the array
    _both(SMALL, seed=63, mean=True, causal=True)
    _both(BIG, seed=64, outputs=False)
    _both(SMALL, seed=65, outputs=False)


# its use case: callers that cannot allocate, such as code under HIP graph
# capture.  The call is captured once and replayed several times, with the
# program's own eager work and synchronisations between replays; every replay
# is checked bit for bit against an eager call on the same inputs (one
# layer on the chained calls, one on the fused launch).
@pytest.mark.parametrize("w", [
    W("na-graph", B=2, Hq=8, Hkv=2, D=128, N=3000, W=16, C=8, budget=700, n_prefix=4, revisit_frac=0.1),
    W("na-graph-fused", B=2, Hq=8, Hkv=2, D=128, N=16384, W=16, C=8, budget=2048, revisit_frac=0.05),
], ids=lambda w: w.name)
def test_noalloc_graph_replays(w):
    d = dims_of(w)
    x = synth.make_layer(w, seed=71, device="cuda")
    K0, V0 = x["K"].clone(), x["V"].clone()
    args = (x["q_win"], x["beacons"], x["counts"])
    rope = dict(rope_cos=x["rope_cos"], rope_sin=x["rope_sin"])
    # eager reference
    Kr, Vr = K0.clone(), V0.clone()
    kept_r = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    scores_r = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    bkv.evict_noalloc(d, Kr, Vr, *args, kept=kept_r, scores=scores_r, status=status, **rope)
    torch.cuda.synchronize()
    assert int(status.item()) == bkv.OK
    # captured call on static buffers
    K, V = K0.clone(), V0.clone()
    kept = torch.full_like(kept_r, -1)
    scores = torch.full_like(scores_r, float("nan"))
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    say(f"capture bkv_evict_noalloc {w.name}: {d}")
    with torch.cuda.graph(g):
        bkv.evict_noalloc(d, K, V, *args, kept=kept, scores=scores, status=status, **rope)
    torch.cuda.synchronize()
    for r in range(4):
        # the program's own eager work between replays: fresh inputs, cleared outputs
        K.copy_(K0)
        V.copy_(V0)
        kept.fill_(-1)
        scores.fill_(float("nan"))
        status.fill_(-1)
        torch.cuda.synchronize()
        say(f"  replay {r}")
        g.replay()
        torch.cuda.synchronize()
        assert int(status.item()) == bkv.OK
        np.testing.assert_array_equal(kept.cpu().numpy(), kept_r.cpu().numpy())
        assert torch.equal(scores, scores_r)
        n = d.n_keep
        assert np.array_equal(raw_bits(K)[..., :n, :], raw_bits(Kr)[..., :n, :])
        assert np.array_equal(raw_bits(V)[..., :n, :], raw_bits(Vr)[..., :n, :])
