"""Synthetic quality diagnostics of the eviction policies (no model, no
dataset): how well each policy keeps the keys that future queries will
revisit, and how well its observation set covers those future queries.

A trace from synth.revisit_trace plants "thought" keys that sparse global
queries keep coming back to (the thought-revisiting tokens of Section 3.1),
between local queries on recent keys.  Each policy runs the trace through
the periodic eviction driver: BeaconKV's Continual FPS beacons ("beacon"),
running-mean beacons ("ns", row a1), the prompt's first queries frozen
("initial", Table 3's Initial+Recent) and recent queries only ("rpc").  At
every eviction:
  * retention: the fraction of the planted keys still cached;
  * coverage: the mean, over the queries of the next `horizon` steps, of
    their largest cosine similarity to the pre-RoPE observation set the
    eviction used (beacons of the kv-head plus its query heads' recent
    queries), the quantity Figure 6a plots for past-query sets; reported
    over every future query and over the global ones alone.
The metrics themselves are plain set and cosine computations; the test
recomputes them from the recorded data in numpy.
"""
from __future__ import annotations

import torch

from paper_2609_04971_amd.driver import PeriodicEviction


def retention(pos, n_plant: int) -> float:
    """pos [..., L] token positions cached per head: mean fraction of the
    positions 0..n_plant-1 present."""
    return float(((pos < n_plant).sum(-1).float() / n_plant).mean())


def coverage(obs, fut, fut_mask) -> float:
    """obs [H, R, D] observation rows (zero rows ignored), fut [H, F, D]
    future queries, fut_mask [H, F] which of them count: the mean over the
    counted queries of max_r cos(f, obs_r) (nan when none counts)."""
    o = obs.float()
    f = fut.float()
    on = o.norm(dim=-1, keepdim=True)
    valid = on.squeeze(-1) > 0
    o = o / on.clamp_min(1e-30)
    f = f / f.norm(dim=-1, keepdim=True).clamp_min(1e-30)
    c = torch.matmul(f, o.transpose(1, 2).contiguous())  # [H, F, R]
    c = c.masked_fill(~valid[:, None, :], -2.0)
    best = c.max(dim=-1).values
    m = fut_mask.bool()
    return float(best[m].mean()) if bool(m.any()) else float("nan")


def _identity_rope(D, device):
    cos = torch.ones(D // 2, device=device)
    sin = torch.zeros(D // 2, device=device)
    return lambda t: (cos, sin)


def run(trace, mode: str, B_max: int, n_beacon: int = 16, n_recent: int = 16, prompt: int | None = None,
        horizon: int = 256, record: bool = False, compaction: str = "order"):
    """Run `trace` (synth.revisit_trace, on the GPU) through the periodic
    driver with policy `mode`.  Returns per-eviction retention and coverage
    (and, with record, the per-eviction observation sets, future queries
    and cached positions, the driver and the final positions)."""
    K, V, q, glob = trace["K"], trace["V"], trace["q"], trace["is_global"]
    LB, Hkv, T, D = K.shape
    Hq = q.shape[1]
    G = Hq // Hkv
    T0 = B_max // 2 if prompt is None else prompt
    drv = PeriodicEviction(1, LB, Hq, Hkv, D, B_max, _identity_rope(D, K.device), n_beacon=n_beacon,
                           n_recent=n_recent, mode=mode, device=K.device, compaction=compaction)
    drv.prefill(K[:, :, :T0].contiguous(), V[:, :, :T0].contiguous(), q[:, :, :T0].contiguous())
    pos = torch.arange(T0, device=K.device).view(1, 1, T0).expand(LB, Hkv, T0).clone()
    out = {"retention": [], "coverage": [], "coverage_global": [], "steps": []}
    rec = []
    for t in range(T0, T):
        ev = drv.step(K[:, :, t], V[:, :, t], q[:, :, t], q[:, :, t])
        pos = torch.cat([pos, torch.full((LB, Hkv, 1), t, device=K.device, dtype=pos.dtype)], 2)
        if not ev:
            continue
        pos = torch.gather(pos, 2, drv.kept.long())
        # the observation set of each kv-head: its beacons and its query heads' recent queries
        rec_q = drv.recent_pre[:, :, :n_recent].reshape(LB, Hkv, G * n_recent, D).float()
        if mode == "rpc":
            obs = rec_q
        else:
            bc = drv.beacons * (drv.counts > 0).unsqueeze(-1)
            obs = torch.cat([bc, rec_q], 2)
        end = min(T, t + 1 + horizon)
        fut = q[:, :, t + 1:end].reshape(LB, Hkv, G * (end - t - 1), D)
        fm = glob[:, :, t + 1:end].reshape(LB, Hkv, G * (end - t - 1))
        o3, f3 = obs.reshape(LB * Hkv, -1, D), fut.reshape(LB * Hkv, -1, D)
        out["retention"].append(retention(pos, trace["n_plant"]))
        out["coverage"].append(coverage(o3, f3, torch.ones_like(fm).reshape(LB * Hkv, -1)))
        out["coverage_global"].append(coverage(o3, f3, fm.reshape(LB * Hkv, -1)))
        out["steps"].append(t)
        if record:
            rec.append({"pos": pos.clone(), "obs": obs.clone(), "fut": fut.clone(), "fut_mask": fm.clone()})
    if record:
        out.update(record=rec, driver=drv, pos=pos)
    return out


def summary(res) -> dict:
    """Means over the evictions of a run's metrics, and the last retention."""
    def mean(x):
        x = [v for v in x if v == v]
        return round(sum(x) / len(x), 4) if x else None
    return {"evictions": len(res["steps"]), "retention_last": round(res["retention"][-1], 4),
            "retention_mean": mean(res["retention"]), "coverage_mean": mean(res["coverage"]),
            "coverage_global_mean": mean(res["coverage_global"])}
