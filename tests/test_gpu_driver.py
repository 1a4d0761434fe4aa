"""GPU check of the periodic eviction driver (Algorithm 2's phase machine on
the library's kernels) in lockstep with the oracle.

A short synthetic decode (2 layers, B_max = 64, B_min = 56, 4 beacon and 4
recent queries per head) runs through three evictions.  Every call the
driver makes is recorded with its inputs, and the test checks:
  * the order of the calls: prefill FPS, a fill-compress whenever the buffer
    holds n_beacon + n_recent queries, the freeze at L = B_max - n_recent,
    the eviction at L = B_max, the merge after it;
  * the data each call saw: a buffer made of the previous selection and the
    steps' pre-RoPE queries; recent rows equal to those steps' post-RoPE
    queries; beacons equal to the frozen selection widened to fp32; K and V
    equal to the cache the test tracks itself (per head, token positions
    appended and compacted with the driver's kept sets);
  * each FPS selection against the oracle (exact up to the first near tie,
    every pick within the fp32 band), each eviction's scores and kept set
    against the oracle (1e-3, tie-band rule) and its compaction bit-exact.
The test follows the driver's decisions, so that a tie broken the other way
inside the band cannot make the two runs drift apart.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_scores_close, compare_kept, host, say
from paper_2609_04971_amd import synth
from paper_2609_04971_amd.driver import PeriodicEviction

pytestmark = pytest.mark.gpu

LAYERS, B, HQ, HKV, D = 2, 1, 4, 2, 64
B_MAX, NB, NR, T0 = 64, 4, 4, 40
STEPS = (B_MAX - T0) + 2 * (B_MAX // 8)  # three evictions
U = 2.0 ** -24


def fps_tol(n, d):
    K = n + d + 8
    return 2.0 * K * U / (1.0 - K * U)


def rope(q_pre, pos):
    cos, sin = synth.rope_table(D, pos)
    x = q_pre.float()
    a, b = x[..., : D // 2], x[..., D // 2:]
    return torch.cat([a * cos - b * sin, a * sin + b * cos], -1).to(torch.bfloat16)


def check_fps(src, picks, m):
    n = src.shape[2]
    q3 = src.reshape(-1, n, D)
    g = picks.reshape(q3.shape[0], -1).numpy().astype(np.int32)
    tol = fps_tol(n, D)
    ref, tie = oracle.fps(q3, m, tie_tol=tol)
    for h in range(g.shape[0]):
        s = int(np.argmax(tie[h])) if tie[h].any() else g.shape[1]
        assert np.array_equal(g[h, :s], ref[h, :s])
    oracle.fps(q3, m, forced=g, tie_tol=tol)


def gather(src, picks):
    return torch.gather(src, 2, picks.long().unsqueeze(-1).expand(-1, -1, -1, src.shape[-1]))


def bits(t):
    return t.contiguous().view(torch.int16)


def test_periodic_eviction_lockstep_with_oracle():
    LB = LAYERS * B
    total = T0 + STEPS
    w = synth.Workload("drv", B=LB, Hq=HQ, Hkv=HKV, D=D, N=total, W=0, C=0, budget=1, n_centroids=6, sigma=0.3)
    q_pre = synth.query_stream(w, total, seed=3)                      # [LB, Hq, total, D] bf16
    gen = torch.Generator().manual_seed(4)
    Kall = torch.randn(LB, HKV, total, D, generator=gen).to(torch.bfloat16)
    Vall = torch.randn(LB, HKV, total, D, generator=gen).to(torch.bfloat16)
    q_rope = torch.stack([rope(q_pre[:, :, p], p) for p in range(total)], 2)

    def table(t):
        c, s = synth.rope_table(D, t)
        return c.cuda(), s.cuda()

    drv = PeriodicEviction(LAYERS, B, HQ, HKV, D, B_MAX, table, n_beacon=NB, n_recent=NR, record=True)
    drv.prefill(Kall[:, :, :T0].cuda(), Vall[:, :, :T0].cuda(), q_pre[:, :, :T0].cuda().contiguous())
    ev = drv.events
    assert len(ev) == 1 and ev[0][0] == "fps" and ev[0][1]["why"] == "prefill"
    check_fps(host(ev[0][1]["src"]), host(ev[0][1]["picks"]), NB)
    buf = gather(q_pre[:, :, :T0], host(ev[0][1]["picks"]))       # the head buffers, [LB, Hq, NB, D]
    pos = np.broadcast_to(np.arange(T0), (LB, HKV, T0)).copy()     # token position of every cached row
    recent, frozen, whys, seen = [], None, [], 1
    for i in range(STEPS):
        p = T0 + i
        evicted = drv.step(Kall[:, :, p].cuda(), Vall[:, :, p].cuda(), q_pre[:, :, p].cuda(),
                           q_rope[:, :, p].cuda())
        pos = np.concatenate([pos, np.full((LB, HKV, 1), p)], 2)
        L = pos.shape[2]
        if L <= B_MAX - NR:
            buf = torch.cat([buf, q_pre[:, :, p:p + 1]], 2)
        if B_MAX - NR < L <= B_MAX:
            recent.append(p)
        for kind, e in ev[seen:]:
            whys.append(e.get("why", kind))
            if kind == "fps":
                src, picks = host(e["src"]), host(e["picks"])
                want = torch.cat([frozen, q_pre[:, :, recent]], 2) if e["why"] == "merge" else buf
                assert torch.equal(bits(src), bits(want)), f"step {p}: input of the {e['why']} FPS"
                check_fps(src, picks, NB)
                buf = gather(src, picks)
                if e["why"] == "freeze":
                    assert L == B_MAX - NR
                    frozen = buf.clone()
                if e["why"] == "fill":
                    assert src.shape[2] == NB + NR
                continue
            assert kind == "evict" and L == B_MAX
            Kb, Vb = (host(x) for x in e["before"])
            idx = torch.from_numpy(pos).long().unsqueeze(-1).expand(-1, -1, -1, D)
            assert torch.equal(bits(Kb), bits(torch.gather(Kall, 2, idx))), "K before eviction"
            assert torch.equal(bits(Vb), bits(torch.gather(Vall, 2, idx))), "V before eviction"
            q_win = host(e["q_win"])
            assert torch.equal(bits(q_win), bits(q_rope[:, :, recent]))
            bc, cn = host(e["beacons"]), host(e["counts"])
            assert torch.equal(bc.view(LB, HQ, NB, D), frozen.float()) and bool((cn == 1).all())
            rc, rs = (host(x) for x in e["rope"])
            ref = oracle.evict(Kb, Vb, q_win, bc, cn, N=B_MAX, budget=drv.B_min, W=NR, rope_cos=rc, rope_sin=rs,
                               threads=4)
            assert_scores_close(host(e["scores"]).numpy(), ref["scores"])
            kg = host(e["kept"]).numpy()
            band, diff = compare_kept(kg, ref["kept"], ref["scores"], B_MAX, NR, 0, drv.B_min)
            Kc, Vc = oracle.compact(Kb, Vb, kg)  # the driver's selection, compacted by the oracle
            Kd, Vd = host(drv.K), host(drv.V)
            assert np.array_equal(bits(Kd[:, :, :drv.B_min]).numpy(), Kc.view(np.int16)[:, :, :drv.B_min])
            assert np.array_equal(bits(Vd[:, :, :drv.B_min]).numpy(), Vc.view(np.int16)[:, :, :drv.B_min])
            pos = np.take_along_axis(pos, kg.astype(np.int64), 2)
            say(f"step {p}: eviction, tie band {band}, {diff} in-band differences")
        seen = len(ev)
        if evicted:
            recent = []  # the merge after the eviction has used them
        assert evicted == (L == B_MAX)
        if evicted:
            assert drv.L == drv.B_min and pos.shape[2] == drv.B_min
    # the order of the calls
    assert whys.count("evict") == 3 and whys.count("freeze") == 3 and whys.count("merge") == 3
    for k in range(len(whys)):
        if whys[k] == "freeze":
            assert whys[k + 1] == "evict" and whys[k + 2] == "merge"
    assert "fill" in whys
