"""Seeded synthetic workloads for the eviction step (inputs only).

This module draws tensors; it holds none of the method's arithmetic.  Tests
and the benchmark use it to feed the GPU library and the CPU oracle the same
inputs.  The paper's workload (Qwen3-4B and other reasoning models decoding
up to 32K tokens on math and coding benchmarks; Section 5.1, Table 4) is not
reproduced: no model weights or benchmark items are used.  Instead each
configuration has the shapes of one attention layer of the named model and
values drawn as follows:

  * keys ~ N(0, 1) per coordinate, with a few seeded outlier channels scaled
    up (and, where configured, a per-head scale), as post-RoPE keys of real
    models have;
  * queries are drawn around unit-norm cluster centroids per kv-head,
    q = sqrt(D) * (mu_k + sigma * xi), which gives attention logits of
    standard deviation ~1.5-2.5 like real attention (the sqrt(D) factor);
    where configured the centroids drift on the unit sphere from one decode
    step to the next (mu <- normalise(mu + drift * u), u a random unit
    vector), so the recent window spans slowly moving clusters;
  * a fraction of recent queries are "revisits": a key among the first 1024
    tokens, rescaled to the query's norm (the paper's thought-revisiting
    queries, Section 3.1);
  * beacons sit near the centroids (a cluster mean of n_c members is the
    centroid plus noise shrunk by sqrt(n_c)), with counts n_c in [1, 64];
  * the RoPE table is rotate-half with base 1e6 at position t = N.
Every draw comes from one torch.Generator seeded per layer; a CPU generator
and a GPU generator give different (equally valid) streams, and parity tests
always hand the *same* tensors to both sides.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    D: int
    N: int
    W: int
    C: int
    budget: int
    dtype: str = "bf16"
    layers: int = 1
    n_prefix: int = 0
    n_centroids: int = 8
    sigma: float = 0.2
    n_outlier: int = 4
    outlier_scale: float = 10.0
    revisit_frac: float = 0.0
    revisit_span: int = 1024
    zipf: float = 0.0                       # centroid popularity ~ (k+1)^-zipf
    head_scale: tuple = field(default=(1.0, 1.0))  # per-kv-head key scale ~ U(a, b)
    qscale: float | None = None             # None -> sqrt(D)
    rope_base: float = 1e6
    drift: float = 0.0                      # centroid drift per decode step (0: static centroids)

    @property
    def G(self):
        return self.Hq // self.Hkv

    @property
    def P(self):
        return self.B * self.Hkv

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five configurations of the eviction-step study.
TINY_FP32 = Workload("tiny-fp32-N512", B=1, Hq=8, Hkv=2, D=64, N=512, W=16, C=4, budget=128, dtype="fp32",
                     n_centroids=4, sigma=0.1, n_outlier=2, outlier_scale=8.0)
QWEN3_4B_4K = Workload("qwen3-4b-layer-N4096", B=16, Hq=32, Hkv=8, D=128, N=4096, W=32, C=8, budget=2048,
                       n_centroids=8, sigma=0.2, n_outlier=4, outlier_scale=10.0, revisit_frac=0.05)
QWEN3_4B_32K = Workload("qwen3-4b-36L-N32768", B=16, Hq=32, Hkv=8, D=128, N=32768, W=32, C=16, budget=4096,
                        layers=36, n_centroids=8, sigma=0.2, n_outlier=4, outlier_scale=10.0, revisit_frac=0.05)
QWEN25_7B_16K = Workload("qwen2.5-7b-28L-N16384-gqa7", B=8, Hq=28, Hkv=4, D=128, N=16384, W=64, C=16,
                         budget=2048, layers=28, n_centroids=16, sigma=0.2, zipf=1.2, revisit_frac=0.0)
LLAMA8B_64K = Workload("llama-8b-32L-N65536", B=4, Hq=32, Hkv=8, D=128, N=65536, W=128, C=32, budget=8192,
                       layers=32, n_centroids=32, sigma=0.2, head_scale=(0.5, 2.0), revisit_frac=0.02, drift=0.01)
CONFIGS = {w.name: w for w in (TINY_FP32, QWEN3_4B_4K, QWEN3_4B_32K, QWEN25_7B_16K, LLAMA8B_64K)}


def torch_dtype(w: Workload):
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def rope_table(D: int, t: int, base: float = 1e6):
    """cos/sin [D/2] fp32 of rotate-half RoPE at absolute position t."""
    i = torch.arange(D // 2, dtype=torch.float64)
    ang = t * base ** (-2.0 * i / D)
    return torch.cos(ang).float(), torch.sin(ang).float()


def _centroids(w: Workload, g, device):
    mu = torch.randn(w.B, w.Hkv, w.n_centroids, w.D, generator=g, device=device)
    return mu / mu.norm(dim=-1, keepdim=True)


def _labels(w: Workload, shape, g, device):
    if w.zipf > 0:
        p = (torch.arange(w.n_centroids, dtype=torch.float64) + 1.0) ** (-w.zipf)
        p = (p / p.sum()).to(device=device, dtype=torch.float32)
        flat = torch.multinomial(p, int(math.prod(shape)), replacement=True, generator=g)
        return flat.reshape(shape)
    return torch.randint(0, w.n_centroids, shape, generator=g, device=device)


def _queries(w: Workload, mu, T: int, g, device):
    """[B, Hq, T, D] fp32 around the kv-head's centroids.  mu is [B, Hkv,
    n_centroids, D] (the same centroids at every step) or [B, Hkv,
    n_centroids, T, D] (step t's query around the centroids of step t)."""
    qs = w.qscale if w.qscale is not None else math.sqrt(w.D)
    lab = _labels(w, (w.B, w.Hq, T), g, device)
    kv = (torch.arange(w.Hq, device=device) // w.G).view(1, w.Hq, 1).expand(w.B, w.Hq, T)
    b = torch.arange(w.B, device=device).view(w.B, 1, 1).expand(w.B, w.Hq, T)
    if mu.dim() == 5:
        t = torch.arange(T, device=device).view(1, 1, T).expand(w.B, w.Hq, T)
        base = mu[b, kv, lab, t]
    else:
        base = mu[b, kv, lab]
    return qs * (base + w.sigma * torch.randn(w.B, w.Hq, T, w.D, generator=g, device=device))


def _drift_path(w: Workload, mu, steps: int, g, device):
    """Centroids over `steps` decode steps, [B, Hkv, n_centroids, steps, D]:
    the first step's are mu, and each step moves every centroid to
    normalise(mu + drift * u) with u a random unit vector."""
    out = torch.empty(*mu.shape[:3], steps, w.D, device=device)
    cur = mu
    for t in range(steps):
        out[:, :, :, t] = cur
        u = torch.randn(mu.shape, generator=g, device=device)
        cur = cur + w.drift * u / u.norm(dim=-1, keepdim=True)
        cur = cur / cur.norm(dim=-1, keepdim=True)
    return out


def make_layer(w: Workload, seed: int = 0, device="cpu", N_cap: int | None = None, v_random: bool = True):
    """One layer's inputs.  Returns a dict of tensors on `device`:
    K, V [B,Hkv,N_cap,D]; q_win [B,Hq,W,D]; q_new [B,Hq,1,D]; beacons
    [B,Hkv,C,D] fp32; counts [B,Hkv,C] int32; rope_cos, rope_sin [D/2]."""
    N_cap = w.N if N_cap is None else N_cap
    g = _gen(seed, device)
    dt = torch_dtype(w)
    K = torch.randn(w.B, w.Hkv, N_cap, w.D, generator=g, device=device, dtype=dt)
    ch = torch.randperm(w.D, generator=g, device=device)[: w.n_outlier]
    if w.n_outlier:
        K[..., ch] *= w.outlier_scale
    if w.head_scale != (1.0, 1.0):
        lo, hi = w.head_scale
        hs = lo + (hi - lo) * torch.rand(w.B, w.Hkv, 1, 1, generator=g, device=device)
        K.mul_(hs.to(dt))
    if v_random:
        V = torch.randn(w.B, w.Hkv, N_cap, w.D, generator=g, device=device, dtype=dt)
    else:
        V = torch.empty_like(K)
    mu = _centroids(w, g, device)
    if w.drift > 0:
        # the recent queries sit at the last W steps before the current one;
        # their centroids drift from step to step, and the current step's
        # query (q_new) uses the centroids one step after the window's last
        path = _drift_path(w, mu, w.W + 1, g, device)
        q_win = _queries(w, path[:, :, :, : w.W], w.W, g, device)
    else:
        q_win = _queries(w, mu, w.W, g, device)
    if w.revisit_frac > 0 and w.W > 0:
        hit = torch.rand(w.B, w.Hq, w.W, generator=g, device=device) < w.revisit_frac
        span = max(1, min(w.revisit_span, w.N))
        j = torch.randint(0, span, (w.B, w.Hq, w.W), generator=g, device=device)
        kv = (torch.arange(w.Hq, device=device) // w.G).view(1, w.Hq, 1).expand(w.B, w.Hq, w.W)
        b = torch.arange(w.B, device=device).view(w.B, 1, 1).expand(w.B, w.Hq, w.W)
        kj = K[b, kv, j].float()
        rev = kj / kj.norm(dim=-1, keepdim=True) * q_win.norm(dim=-1, keepdim=True)
        q_win = torch.where(hit.unsqueeze(-1), rev, q_win)
    q_new = _queries(w, path[:, :, :, w.W:] if w.drift > 0 else mu, 1, g, device)
    counts = torch.randint(1, 65, (w.B, w.Hkv, w.C), generator=g, device=device, dtype=torch.int32)
    qs = w.qscale if w.qscale is not None else math.sqrt(w.D)
    cidx = torch.arange(w.C, device=device) % w.n_centroids
    noise = torch.randn(w.B, w.Hkv, w.C, w.D, generator=g, device=device)
    beacons = qs * (mu[:, :, cidx] + w.sigma * noise / counts.float().sqrt().unsqueeze(-1))
    cos, sin = rope_table(w.D, w.N, w.rope_base)
    return {
        "K": K, "V": V, "q_win": q_win.to(dt).contiguous(), "q_new": q_new.to(dt).contiguous(),
        "beacons": beacons.float().contiguous(), "counts": counts.contiguous(),
        "rope_cos": cos.to(device), "rope_sin": sin.to(device),
    }


def query_stream(w: Workload, T: int, seed: int = 0, device="cpu"):
    """A stream of T pre-RoPE decode queries [B, Hq, T, D] around the
    centroids (drifting from step to step when the workload's drift > 0)."""
    g = _gen(seed, device)
    mu = _centroids(w, g, device)
    if w.drift > 0:
        mu = _drift_path(w, mu, T, g, device)
    return _queries(w, mu, T, g, device).to(torch_dtype(w)).contiguous()


def sorted_subsets(P: int, N: int, n: int, seed: int = 0, forced_tail: int = 0):
    """kept-index patterns for compaction tests: [P, n] int32, strictly
    ascending in [0, N); the last `forced_tail` indices always included."""
    g = _gen(seed, "cpu")
    out = torch.empty(P, n, dtype=torch.int32)
    for p in range(P):
        body = torch.randperm(N - forced_tail, generator=g)[: n - forced_tail]
        tail = torch.arange(N - forced_tail, N)
        out[p] = torch.cat([body, tail]).sort().values.to(torch.int32)
    return out


def revisit_trace(LB: int, Hq: int, Hkv: int, D: int, T: int, n_plant: int = 32, n_groups: int = 4,
                  p_global: float = 0.02, local_dim: int = 16, drift: float = 0.18, align: float = 0.8,
                  local_gain: float = 0.5, global_gain: float = 2.0, sigma: float = 0.3, seed: int = 0,
                  device="cpu"):
    """A decode trace with the query geometry of Section 3 (no RoPE, so
    queries are their own pre- and post-RoPE forms):
      * local queries: each kv-head has a direction d(t) that drifts slowly
        on the unit sphere of a random local_dim-dimensional subspace
        (d(t) = normalise(d(t-1) + drift * xi), xi ~ N(0, I/local_dim)); key
        j is sqrt(D) * (align * d(j) + sqrt(1 - align^2) * z_j), z_j a random
        unit vector, and a local query is local_gain * sqrt(D) * (d(t) +
        sigma * xi') with xi' ~ N(0, I/D).  Local queries are close to their
        neighbours and attend to recent keys (Section 3.1, the local
        pattern; Figure 5a's neighbour similarity);
      * thought keys: the first n_plant tokens are sqrt(D) * p_i, p_i random
        unit vectors, in n_groups contiguous groups (the plan and
        constraints written early in a trace);
      * global queries: with probability p_global per query head and step
        (never in the first n_plant steps), a query of a random group c is
        global_gain * sqrt(D) * (u_c + sigma * xi'), u_c the normalised sum
        of the group's p_i.  Global queries of one group are close to each
        other and far from their local neighbours, and attend to their
        group's thought keys (Section 3.1, thought revisiting; Section 3.2,
        the clusters of Figure 5b).
    Returns K, V [LB, Hkv, T, D] bf16, q [LB, Hq, T, D] bf16, is_global
    [LB, Hq, T] bool, group [LB, Hq, T] int64 (-1 for local queries) and
    n_plant."""
    g = _gen(seed, device)
    G = Hq // Hkv
    sq = math.sqrt(D)
    basis = torch.linalg.qr(torch.randn(LB, Hkv, D, local_dim, generator=g, device=device))[0]
    x = torch.randn(LB, Hkv, local_dim, generator=g, device=device)
    walk = torch.empty(LB, Hkv, T, local_dim, device=device)
    steps = torch.randn(LB, Hkv, T, local_dim, generator=g, device=device) * (drift / math.sqrt(local_dim))
    x = x / x.norm(dim=-1, keepdim=True)
    for t in range(T):
        x = x + steps[:, :, t]
        x = x / x.norm(dim=-1, keepdim=True)
        walk[:, :, t] = x
    d = torch.matmul(walk, basis.transpose(-1, -2))  # [LB, Hkv, T, D] unit
    z = torch.randn(LB, Hkv, T, D, generator=g, device=device)
    z = z / z.norm(dim=-1, keepdim=True)
    K = sq * (align * d + math.sqrt(1.0 - align * align) * z)
    p = torch.randn(LB, Hkv, n_plant, D, generator=g, device=device)
    p = p / p.norm(dim=-1, keepdim=True)
    K[:, :, :n_plant] = sq * p
    V = torch.randn(LB, Hkv, T, D, generator=g, device=device)
    grp_of = torch.arange(n_plant, device=device) * n_groups // n_plant
    u = torch.zeros(LB, Hkv, n_groups, D, device=device).index_add_(2, grp_of, p)
    u = u / u.norm(dim=-1, keepdim=True)
    is_global = torch.rand(LB, Hq, T, generator=g, device=device) < p_global
    is_global[:, :, :n_plant] = False
    group = torch.randint(0, n_groups, (LB, Hq, T), generator=g, device=device)
    kv = (torch.arange(Hq, device=device) // G).view(1, Hq, 1).expand(LB, Hq, T)
    b = torch.arange(LB, device=device).view(LB, 1, 1).expand(LB, Hq, T)
    xi = torch.randn(LB, Hq, T, D, generator=g, device=device) / sq
    q_loc = local_gain * sq * (d.repeat_interleave(G, dim=1) + sigma * xi)
    q_glb = global_gain * sq * (u[b, kv, group] + sigma * xi)
    q = torch.where(is_global.unsqueeze(-1), q_glb, q_loc)
    group = torch.where(is_global, group, torch.full_like(group, -1))
    return {"K": K.to(torch.bfloat16), "V": V.to(torch.bfloat16), "q": q.to(torch.bfloat16).contiguous(),
            "is_global": is_global, "group": group, "n_plant": n_plant}
