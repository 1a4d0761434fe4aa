"""GPU parity at the benchmark's full size: whole Qwen3-4B-shaped layers at
32K tokens (B=16, Hkv=8, D=128, N=32768, R=144, budget 4096), evicted by the
same calls bench.py times (score -> top-k -> compact on one workspace).
Every head of one layer is checked against the oracle (scores, kept set,
and the selection and compaction in isolation, bit for bit); a second layer
through the same workspace is checked on sampled heads; properties that hold
at any size are checked on every head.  The decode trace's evictions (12
Qwen3-4B layers stacked into one call at the steady state 4224 -> 4096, with
the fused launch and with the hole-filling compaction) and the wide-group
layers are checked on sampled heads, with every head's selection in
isolation."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_rows_match, assert_scores_close, compare_kept, dims_of, host, raw_bits, say
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth

pytestmark = pytest.mark.gpu

BATCHES = [0, 7, 15]                           # batches copied to the host
HEADS = [(0, 0), (0, 7), (1, 3), (2, 0), (2, 7)]  # (index into BATCHES, kv-head)


def _host_batches(x):
    per_batch = ("K", "V", "q_win", "beacons", "counts")
    return {k: host(v[BATCHES]) if k in per_batch else host(v) for k, v in x.items()}


def test_benchmark_layer_all_heads():
    # layer 0 of the benchmark: all 128 heads against the oracle
    #  * scores element by element within 1e-3, kept under the tie-band rule;
    #  * isolation, zero tolerance: the oracle's selection fed the GPU's own
    #    scores reproduces the GPU's kept indices, and the oracle's compaction
    #    fed the GPU's own kept indices reproduces the GPU's K and V
    w = synth.QWEN3_4B_32K
    d = dims_of(w)
    ws = bkv.workspace(d, bkv.OP_EVICT)
    scores = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    kept = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    x = synth.make_layer(w, seed=100, device="cuda")
    xh = {k: host(v) for k, v in x.items()}  # 2 GB of K and V before the eviction
    say(f"benchmark layer 0, all heads: {d}")
    bkv.score(d, x["K"], x["q_win"], x["beacons"], x["counts"], scores, ws, rope_cos=x["rope_cos"],
              rope_sin=x["rope_sin"])
    bkv.topk(d, scores, kept)
    bkv.compact(d, x["K"], x["V"], kept, ws)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    s_all, k_all = host(scores).numpy(), host(kept).numpy()
    assert not np.isnan(s_all).any() and np.all(s_all <= 1e-4)

    say("  isolation: oracle top-k on the GPU's scores, all heads")
    np.testing.assert_array_equal(oracle.topk(s_all.astype(np.float64), w.budget, w.W, 0), k_all)
    say("  isolation: oracle compaction on the GPU's kept indices, all heads")
    Kr, Vr = oracle.compact(xh["K"], xh["V"], k_all)
    n = d.n_keep
    assert np.array_equal(raw_bits(x["K"])[..., :n, :], Kr[..., :n, :].view(np.uint16)), "K differs"
    assert np.array_equal(raw_bits(x["V"])[..., :n, :], Vr[..., :n, :].view(np.uint16)), "V differs"
    del Kr, Vr

    say("  oracle scores on all 128 heads")
    s_ref, _ = oracle.score(xh["K"], xh["q_win"], xh["beacons"], xh["counts"], N=w.N, rope_cos=xh["rope_cos"],
                            rope_sin=xh["rope_sin"], threads=16)
    err = assert_scores_close(s_all, s_ref)
    k_ref = oracle.topk(s_ref, w.budget, w.W, 0)
    band, diff = compare_kept(k_all, k_ref, s_ref, w.N, w.W, 0, w.budget)
    exact = int(np.all(k_all == k_ref, axis=-1).sum())
    say(f"  max |score diff| {err:.2e}; tie band {band} keys, {diff} in-band differences; "
        f"{exact}/{d.P} heads keep exactly the oracle's set")


def test_benchmark_second_layer_sampled_heads():
    # a second layer through the same workspace, as the benchmark runs it
    w = synth.QWEN3_4B_32K
    d = dims_of(w)
    ws = bkv.workspace(d, bkv.OP_EVICT)
    scores = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    kept = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    for layer in (0, 1):
        x = synth.make_layer(w, seed=100 + layer, device="cuda")
        xh = _host_batches(x)
        say(f"benchmark layer {layer}: {d}")
        bkv.score(d, x["K"], x["q_win"], x["beacons"], x["counts"], scores, ws, rope_cos=x["rope_cos"],
                  rope_sin=x["rope_sin"])
        bkv.topk(d, scores, kept)
        bkv.compact(d, x["K"], x["V"], kept, ws)
        torch.cuda.synchronize()
        assert bkv.device_status(ws) == bkv.OK

        # every head: scores are log-probabilities, kept is ascending and
        # holds the recent window
        s_all = host(scores).numpy()
        k_all = host(kept).numpy()
        assert not np.isnan(s_all).any() and np.all(s_all <= 1e-4)
        assert np.all(np.diff(k_all, axis=-1) > 0)
        assert np.array_equal(k_all[..., -w.W:], np.broadcast_to(np.arange(w.N - w.W, w.N), k_all[..., -w.W:].shape))
        if layer == 0:
            continue  # all of layer 0 is checked above

        say(f"benchmark layer {layer}: oracle on {len(HEADS)} heads")
        ref = oracle.evict(xh["K"], xh["V"], xh["q_win"], xh["beacons"], xh["counts"], N=w.N, budget=w.budget,
                           W=w.W, rope_cos=xh["rope_cos"], rope_sin=xh["rope_sin"], heads=HEADS,
                           threads=len(HEADS))
        bi = np.array([BATCHES[b] for b, _ in HEADS])
        hi = np.array([h for _, h in HEADS])
        li = np.array([b for b, _ in HEADS])
        assert_scores_close(s_all[bi, hi], ref["scores"][li, hi])
        kg, kr = k_all[bi, hi], ref["kept"][li, hi]
        band, diff = compare_kept(kg, kr, ref["scores"][li, hi], w.N, w.W, 0, w.budget)
        say(f"benchmark layer {layer}: tie band {band}, {diff} in-band differences")
        K_gpu = host(x["K"][torch.as_tensor(bi), torch.as_tensor(hi)])
        V_gpu = host(x["V"][torch.as_tensor(bi), torch.as_tensor(hi)])
        assert_rows_match(K_gpu, ref["K"][li, hi], kg, kr, d.n_keep, "K")
        assert_rows_match(V_gpu, ref["V"][li, hi], kg, kr, d.n_keep, "V")
        # every compacted row is the original row at the GPU's own index
        for j, (b, h) in enumerate(HEADS):
            src = raw_bits(xh["K"][b, h])[kg[j]]
            assert np.array_equal(raw_bits(K_gpu[j])[: d.n_keep], src)
        del x
        torch.cuda.empty_cache()


@pytest.mark.parametrize("w", [synth.QWEN25_7B_16K, synth.LLAMA8B_64K], ids=lambda w: w.name)
def test_wide_group_layers_sampled_heads(w):
    # the shapes whose observation rows (R = 464, 544) span several row groups
    d = dims_of(w)
    ws = bkv.workspace(d, bkv.OP_EVICT)
    scores = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    kept = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    x = synth.make_layer(w, seed=200, device="cuda")
    heads = [(0, 0), (w.B - 1, w.Hkv - 1)]
    bsel = sorted({b for b, _ in heads})
    xh = {k: (host(v[bsel]) if k in ("K", "V", "q_win", "beacons", "counts") else host(v)) for k, v in x.items()}
    say(f"wide layer {w.name}: {d}")
    bkv.score(d, x["K"], x["q_win"], x["beacons"], x["counts"], scores, ws, rope_cos=x["rope_cos"],
              rope_sin=x["rope_sin"])
    bkv.topk(d, scores, kept)
    bkv.compact(d, x["K"], x["V"], kept, ws)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    s_all = host(scores).numpy()
    assert not np.isnan(s_all).any() and np.all(s_all <= 1e-4)
    hl = [(bsel.index(b), h) for b, h in heads]
    say(f"wide layer {w.name}: oracle on {len(hl)} heads")
    ref = oracle.evict(xh["K"], xh["V"], xh["q_win"], xh["beacons"], xh["counts"], N=w.N, budget=w.budget, W=w.W,
                       rope_cos=xh["rope_cos"], rope_sin=xh["rope_sin"], heads=hl, threads=len(hl))
    for (b, h), (lb, _) in zip(heads, hl):
        assert_scores_close(s_all[b, h], ref["scores"][lb, h])
        kg, kr = host(kept)[b, h].numpy(), ref["kept"][lb, h]
        band, diff = compare_kept(kg[None], kr[None], ref["scores"][lb, h][None], w.N, w.W, 0, w.budget)
        say(f"  head ({b}, {h}): tie band {band}, {diff} in-band differences")
        assert_rows_match(host(x["K"][b, h])[None], ref["K"][lb, h][None], kg[None], kr[None], d.n_keep, "K")


def test_stacked_layers_steady_state_sampled_heads():
    # the decode trace's eviction: several layers stacked into the batch of
    # one call (here 12 layers of the Qwen3-4B shape, B = 192, 1536 heads),
    # at the steady state 4224 -> 4096 tokens; every head's properties, and
    # sampled heads (first, last, and layer boundaries) against the oracle
    w = synth.QWEN3_4B_32K.with_(B=16 * 12, N=4224)
    d = dims_of(w)
    ws = bkv.workspace(d, bkv.OP_EVICT)
    kept = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    scores = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    x = synth.make_layer(w, seed=300, device="cuda")
    heads = [(0, 0), (15, 7), (16, 0), (100, 3), (191, 7)]
    bsel = sorted({b for b, _ in heads})
    xh = {k: (host(v[bsel]) if k in ("K", "V", "q_win", "beacons", "counts") else host(v)) for k, v in x.items()}
    say(f"stacked layers: {d}")
    bkv.evict(d, x["K"], x["V"], x["q_win"], x["beacons"], x["counts"], ws, kept=kept, scores=scores,
              rope_cos=x["rope_cos"], rope_sin=x["rope_sin"])
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    s_all, k_all = host(scores).numpy(), host(kept).numpy()
    assert not np.isnan(s_all).any() and np.all(s_all <= 1e-4)
    assert np.all(np.diff(k_all, axis=-1) > 0)
    assert np.array_equal(k_all[..., -w.W:], np.broadcast_to(np.arange(w.N - w.W, w.N), k_all[..., -w.W:].shape))
    say(f"  isolation: oracle top-k on the GPU's scores, all {d.P} heads")
    np.testing.assert_array_equal(oracle.topk(s_all.astype(np.float64), w.budget, w.W, 0), k_all)
    hl = [(bsel.index(b), h) for b, h in heads]
    say(f"  oracle on {len(hl)} heads")
    ref = oracle.evict(xh["K"], xh["V"], xh["q_win"], xh["beacons"], xh["counts"], N=w.N, budget=w.budget, W=w.W,
                       rope_cos=xh["rope_cos"], rope_sin=xh["rope_sin"], heads=hl, threads=len(hl))
    for (b, h), (lb, _) in zip(heads, hl):
        assert_scores_close(s_all[b, h], ref["scores"][lb, h])
        kg, kr = k_all[b, h], ref["kept"][lb, h]
        band, diff = compare_kept(kg[None], kr[None], ref["scores"][lb, h][None], w.N, w.W, 0, w.budget)
        say(f"  head ({b}, {h}): tie band {band}, {diff} in-band differences")
        K_gpu = host(x["K"][b, h])
        assert_rows_match(K_gpu[None], ref["K"][lb, h][None], kg[None], kr[None], d.n_keep, "K")
        assert np.array_equal(raw_bits(K_gpu)[: d.n_keep], raw_bits(xh["K"][lb, h])[kg])


def test_stacked_layers_steady_state_hole_filling():
    # the decode trace's eviction with the hole-filling compaction, as timed:
    # bkv_score, bkv_topk and bkv_compact_fill over 12 stacked layers of the
    # Qwen3-4B shape (B = 192, 1536 heads) at the steady state 4224 -> 4096.
    #  * every head: the oracle's selection on the GPU's own scores gives the
    #    GPU's kept set bit for bit; src_of holds that set, and each row below
    #    4096 of K and V is, bit for bit, the old row src_of names;
    #  * sampled heads: scores against the oracle, and the oracle's
    #    hole-filling compaction of the GPU's kept set gives the GPU's K, V
    #    (all 4224 rows) and src_of bit for bit
    w = synth.QWEN3_4B_32K.with_(B=16 * 12, N=4224)
    d = dims_of(w)
    ws = bkv.workspace(d, bkv.OP_EVICT)
    sel = torch.empty(d.B, d.Hkv, d.n_keep, dtype=torch.int32, device="cuda")
    src_of = torch.empty_like(sel)
    scores = torch.empty(d.B, d.Hkv, d.N, device="cuda")
    x = synth.make_layer(w, seed=301, device="cuda")
    heads = [(0, 0), (15, 7), (16, 0), (100, 3), (191, 7)]
    bsel = sorted({b for b, _ in heads})
    xh = {k: (host(v[bsel]) if k in ("K", "V", "q_win", "beacons", "counts") else host(v)) for k, v in x.items()}
    K0, V0 = x["K"].clone(), x["V"].clone()
    say(f"stacked layers, hole filling: {d}")
    bkv.score(d, x["K"], x["q_win"], x["beacons"], x["counts"], scores, ws, rope_cos=x["rope_cos"],
              rope_sin=x["rope_sin"])
    bkv.topk(d, scores, sel, ws)
    bkv.compact_fill(d, x["K"], x["V"], sel, src_of, ws)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    s_all, k_all, so_all = host(scores).numpy(), host(sel).numpy(), host(src_of).numpy()
    assert not np.isnan(s_all).any() and np.all(s_all <= 1e-4)
    say(f"  isolation: oracle top-k on the GPU's scores, all {d.P} heads")
    np.testing.assert_array_equal(oracle.topk(s_all.astype(np.float64), w.budget, w.W, 0), k_all)
    assert np.array_equal(np.sort(so_all, axis=-1), k_all)
    say("  every head's rows below 4096 against src_of")
    for l in range(12):  # one layer (16 batches) at a time: the index tensor stays small
        b0, b1 = 16 * l, 16 * (l + 1)
        idx = src_of[b0:b1].long()[..., None].expand(-1, -1, -1, d.D)
        for new, old in ((x["K"], K0), (x["V"], V0)):
            assert torch.equal(new[b0:b1, :, : d.n_keep].view(torch.int16), old[b0:b1].gather(2, idx).view(torch.int16))
    del K0, V0
    hl = [(bsel.index(b), h) for b, h in heads]
    say(f"  oracle on {len(hl)} heads")
    ref = oracle.evict(xh["K"], xh["V"], xh["q_win"], xh["beacons"], xh["counts"], N=w.N, budget=w.budget, W=w.W,
                       rope_cos=xh["rope_cos"], rope_sin=xh["rope_sin"], heads=hl, threads=len(hl))
    for (b, h), (lb, _) in zip(heads, hl):
        assert_scores_close(s_all[b, h], ref["scores"][lb, h])
        kg = k_all[b, h]
        band, diff = compare_kept(kg[None], ref["kept"][lb, h][None], ref["scores"][lb, h][None], w.N, w.W, 0,
                                  w.budget)
        say(f"  head ({b}, {h}): tie band {band}, {diff} in-band differences")
        kf, vf, so, moved = oracle.compact_fill(xh["K"][lb:lb + 1, h:h + 1], xh["V"][lb:lb + 1, h:h + 1],
                                                kg[None, None], w.N)
        assert np.array_equal(raw_bits(x["K"][b, h]), kf[0, 0])
        assert np.array_equal(raw_bits(x["V"][b, h]), vf[0, 0])
        assert np.array_equal(so_all[b, h], so[0, 0])
        say(f"  head ({b}, {h}): {int(moved[0, 0])} rows moved")
