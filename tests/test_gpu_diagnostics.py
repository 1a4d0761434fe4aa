"""GPU run of the quality diagnostics: a short revisit trace through the
periodic driver in each policy (Continual FPS beacons, running-mean beacons,
recent queries only).  The test checks the bookkeeping the metrics rest on
and recomputes the metrics in numpy:
  * the cached positions the diagnostics track name the rows the driver's
    cache really holds (K bit-exact against the trace at those positions),
    also with the hole-filling compaction, whose rows leave token order;
  * the recent part of every observation set is the last n_recent queries of
    each query head; Continual FPS beacons are queries the head asked before
    the window; running-mean counts add up to every query asked so far;
  * retention and coverage equal a numpy recomputation from the recorded
    positions, observation sets and future queries."""
import numpy as np
import pytest
import torch

from gpu_util import host, say
from paper_2609_04971_amd import diagnostics, synth

pytestmark = pytest.mark.gpu

LB, HQ, HKV, D = 2, 8, 2, 64
B_MAX, NB, NR, T0, T = 128, 4, 4, 64, 192  # evictions at steps 127, 143, ..., 191
N_PLANT, HORIZON = 8, 32
G = HQ // HKV


def _np_coverage(obs, fut, mask):
    o, f = obs.astype(np.float64), fut.astype(np.float64)
    on = np.linalg.norm(o, axis=-1)
    fn = np.linalg.norm(f, axis=-1)
    c = np.einsum("hfd,hrd->hfr", f, o) / (fn[:, :, None] * np.where(on > 0, on, 1.0)[:, None, :])
    c = np.where(on[:, None, :] > 0, c, -2.0)
    best = c.max(-1)
    return best[mask].mean() if mask.any() else float("nan")


@pytest.fixture(scope="module")
def trace():
    tr = synth.revisit_trace(LB, HQ, HKV, D, T, n_plant=N_PLANT, n_groups=2, p_global=0.1, local_dim=8, seed=7)
    return {k: (v.cuda() if torch.is_tensor(v) else v) for k, v in tr.items()}, tr


@pytest.mark.parametrize("mode,compaction", [("beacon", "order"), ("ns", "order"), ("initial", "order"),
                                             ("rpc", "order"), ("beacon", "fill")])
def test_diagnostics_bookkeeping_and_metrics(trace, mode, compaction):
    # with compaction "fill" the cache is no longer in token order: the
    # tracked positions follow the rows through bkv_compact_fill's src_of
    tr, cpu = trace
    say(f"diagnostics {mode} ({compaction}): LB={LB} Hq={HQ} Hkv={HKV} D={D} B_max={B_MAX} T={T}")
    nr = 2 * NR if mode == "rpc" else NR
    res = diagnostics.run(tr, mode, B_MAX, n_beacon=NB, n_recent=nr, prompt=T0, horizon=HORIZON, record=True,
                          compaction=compaction)
    drv = res["driver"]
    assert res["steps"] == [127, 143, 159, 175, 191]
    assert np.isnan(res["coverage"][-1]) and not np.isnan(res["coverage"][:-1]).any()
    # the tracked positions name the cached rows
    pos = host(res["pos"]).long()
    assert drv.L == drv.B_min == pos.shape[2]
    want = torch.gather(cpu["K"], 2, pos.unsqueeze(-1).expand(-1, -1, -1, D))
    assert torch.equal(host(drv.K[:, :, :drv.L]).view(torch.int16), want.view(torch.int16))
    q = cpu["q"].float()
    glob = cpu["is_global"]
    for t, r, ret, cov, covg in zip(res["steps"], res["record"], res["retention"], res["coverage"],
                                    res["coverage_global"]):
        obs = host(r["obs"]).numpy()
        # the recent part: the last nr queries of each of the kv-head's query heads
        rec = q[:, :, t - nr + 1:t + 1].reshape(LB, HKV, G * nr, D).numpy()
        assert np.array_equal(obs[:, :, obs.shape[2] - G * nr:], rec)
        nbc = obs.shape[2] - G * nr
        if mode == "rpc":
            assert nbc == 0
        if mode == "beacon":
            assert nbc == G * NB
            bc = obs[:, :, :nbc].reshape(LB, HKV, G, NB, D)
            for b in range(LB):
                for h in range(HKV):
                    for g in range(G):
                        past = q[b, h * G + g, :t - nr + 1].numpy()
                        for c in range(NB):
                            assert (past == bc[b, h, g, c]).all(-1).any(), f"beacon {b},{h},{g},{c} at {t}"
        # the metrics, recomputed
        p = host(r["pos"]).numpy()
        assert abs(ret - np.mean((p < N_PLANT).sum(-1) / N_PLANT)) < 1e-6
        fut = host(r["fut"]).float().numpy().reshape(LB * HKV, -1, D)
        fm = host(r["fut_mask"]).numpy().reshape(LB * HKV, -1)
        o3 = obs.reshape(LB * HKV, -1, D)
        for got, want in ((cov, _np_coverage(o3, fut, np.ones_like(fm))), (covg, _np_coverage(o3, fut, fm))):
            # nan when no future query counts (the trace's last step evicts)
            assert (np.isnan(got) and np.isnan(want)) or abs(got - want) < 1e-5
    if mode == "ns":
        # every query asked so far has joined one slot
        assert int(host(drv.counts).sum()) == LB * HQ * T
    if mode == "initial":
        # the first NB queries of every query head, frozen at prefill (in
        # the gather's selection order: compared as a permutation)
        bc = host(drv.beacons).view(LB, HQ, NB, D)
        for b in range(LB):
            for hq in range(HQ):
                hit = (bc[b, hq][:, None, :] == q[b, hq, :NB][None, :, :]).all(-1)  # [beacon, query]
                assert sorted(hit.float().argmax(1).tolist()) == list(range(NB)) and bool(hit.any(1).all())
        assert bool((host(drv.counts) == 1).all())
    say(f"  {diagnostics.summary(res)}")


def test_beacons_keep_the_revisited_keys():
    # the Qwen3-4B head shape, two sequences: on a trace with Section 3's
    # geometry the Continual FPS beacons keep more thought keys and cover the
    # global queries better than recent queries alone (the recent-only
    # baseline gets twice the recent queries, the same observation budget)
    tr = synth.revisit_trace(2, 32, 8, 128, 2048, seed=11, device="cuda")
    got = {}
    for mode, nr in (("beacon", 16), ("ns", 16), ("initial", 16), ("rpc", 32)):
        got[mode] = diagnostics.summary(diagnostics.run(tr, mode, 1024, n_beacon=16, n_recent=nr, horizon=256))
        say(f"{mode}: {got[mode]}")
    assert got["beacon"]["retention_mean"] > got["rpc"]["retention_mean"] + 0.1
    assert got["beacon"]["coverage_global_mean"] > got["rpc"]["coverage_global_mean"] + 0.2
    assert got["beacon"]["coverage_global_mean"] > got["ns"]["coverage_global_mean"]
