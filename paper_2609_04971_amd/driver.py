"""Periodic BeaconKV eviction across decoding steps (Algorithm 2's phase
machine) on the library's kernels, for all layers of a model at once.

Layers are stacked into the batch dimension: "batch" here is layers * B, so
every call covers every layer (one FPS launch for every query buffer of the
model, one eviction launch for every kv-head of the model).  The caller owns
the decode loop and supplies, per step, the new token's keys and values and
the step's queries before and after RoPE (a model computes both anyway);
this module keeps the per-head state of Algorithm 2 and makes the calls:

  * prefill: the prompt's keys and values fill the cache; each query head's
    buffer starts as FPS(prompt queries, n_beacon) (Appendix D.2).
  * while L <= B_max - n_recent: the step's pre-RoPE query joins the head's
    buffer; a buffer that reaches B_Q^max = n_beacon + n_recent is compressed
    to B_Q^min = n_beacon by FPS (Section 4.2, Eq. fps_q).
  * at L = B_max - n_recent: the beacon set becomes FPS(buffer, n_beacon),
    frozen, and also widened into the fp32 beacon layout scoring reads; the
    recent set starts empty.
  * while B_max - n_recent < L <= B_max: the step's post-RoPE query joins the
    recent set (and its pre-RoPE form is kept for the merge below).
  * at L = B_max: bkv_evict_ex scores every cached key with the group's
    beacons (rotated to the current step) and recent queries, keeps
    B_min = 7/8 B_max (Section 5.1), compacts K and V; then the buffer is
    the beacon set plus the recent queries, compressed by FPS to n_beacon.

mode "rpc" is the recent-queries-only baseline on the same kernels: no
buffer, no beacons (C = 0), the last n_recent queries before each eviction.
mode "ns" keeps running-mean beacons instead of the FPS buffer: every
step's pre-RoPE queries join the nearest of G * n_beacon slots per kv-head
(bkv_beacon_update), and evictions score with those beacons as they stand.
mode "initial" is the Initial+Recent baseline of Table 3: the first
n_beacon queries of each query head (the prompt's) are frozen as its
beacons for good, next to the same recent window.

compaction "fill" evicts with bkv_score, bkv_topk and bkv_compact_fill
instead of bkv_evict_ex: the cache keeps the same rows but only the kept
rows past B_min move (into the evicted rows below it), so rows are no
longer in token order; `kept` then holds, for each row, the row it came
from (what bkv_compact_fill calls src_of), which is also what `kept` means
for the order-preserving compaction.

Everything that computes runs in the library's kernels; this module only
slices the caller's tensors and appends rows to them (the writes a serving
engine makes to its own cache).
"""
from __future__ import annotations

import torch

import paper_2609_04971_amd as bkv


class PeriodicEviction:
    def __init__(self, layers: int, B: int, Hq: int, Hkv: int, D: int, B_max: int, rope_table, n_beacon: int = 16,
                 n_recent: int = 16, n_prefix: int = 0, mode: str = "beacon", dtype=torch.bfloat16,
                 device="cuda", record: bool = False, timing: bool = False, compaction: str = "order"):
        """rope_table(t) -> (cos, sin), fp32 [D/2] device tensors of the
        model's rotate-half RoPE at absolute position t (the beacons are
        rotated to the step at which eviction runs).  record keeps every
        call's inputs and outputs in `events`; timing brackets every library
        call with HIP events on the current stream, in `times`."""
        if mode not in ("beacon", "rpc", "ns", "initial"):
            raise ValueError("mode is 'beacon', 'rpc', 'ns' or 'initial'")
        if B_max % 8:
            raise ValueError("B_max must be a multiple of 8 (B_min = 7/8 B_max)")
        if compaction not in ("order", "fill"):
            raise ValueError("compaction is 'order' or 'fill'")
        self.compaction = compaction
        self.mode = mode
        self.LB, self.Hq, self.Hkv, self.D = layers * B, Hq, Hkv, D
        self.G = Hq // Hkv
        self.B_max, self.B_min = B_max, 7 * B_max // 8
        self.nb = 0 if mode == "rpc" else n_beacon
        self.nr = n_recent
        if self.B_max - self.nr <= self.B_min:
            raise ValueError("the recent window must fit between B_min and B_max")
        self.record = record
        self.rope_table = rope_table
        dt, dev = dtype, device
        LB = self.LB
        self.K = torch.zeros(LB, Hkv, B_max, D, dtype=dt, device=dev)
        self.V = torch.zeros_like(self.K)
        self.L = 0  # cached tokens per head
        self.t = 0  # absolute position of the next token
        nb, nr = self.nb, self.nr
        if mode == "beacon":
            self.obs = torch.zeros(LB, Hq, nb + nr, D, dtype=dt, device=dev)  # pre-RoPE buffer
            self.obs_len = 0
        self.beacons = torch.zeros(LB, Hkv, self.G * nb, D, dtype=torch.float32, device=dev)
        self.counts = torch.zeros(LB, Hkv, self.G * nb, dtype=torch.int32, device=dev)
        self.recent_rope = torch.zeros(LB, Hq, nr, D, dtype=dt, device=dev)
        self.recent_pre = torch.zeros(LB, Hq, nr, D, dtype=dt, device=dev)
        self.n_rec = 0
        self.dims = bkv.dims(B=LB, Hq=Hq, Hkv=Hkv, D=D, N=B_max, N_cap=B_max, W=nr, C=self.G * nb,
                             budget=self.B_min, n_prefix=n_prefix, dtype="bf16" if dt == torch.bfloat16 else "fp32")
        self.ws = bkv.workspace(self.dims, bkv.OP_EVICT, device=dev)
        self.kept = torch.empty(LB, Hkv, self.B_min, dtype=torch.int32, device=dev)
        self.sel = torch.empty_like(self.kept) if compaction == "fill" else None  # top-k output before filling
        self.scores = torch.empty(LB, Hkv, B_max, dtype=torch.float32, device=dev)
        self.events = []  # (kind, details) of the calls made, when recording
        self.timing = timing
        self.times = []   # (kind, start event, end event), when timing

    # ---- helpers --------------------------------------------------------------
    def _log(self, kind, **kw):
        if self.record:
            self.events.append((kind, kw))

    def _call(self, kind, fn):
        if not self.timing:
            fn()
            return
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        self.times.append((kind, e0, e1))

    def _compress(self, n: int, why: str):
        picks = torch.empty(self.LB, self.Hq, min(self.nb, n), dtype=torch.int32, device=self.obs.device)
        src = self.obs[:, :, :n].clone() if self.record else None
        self._call("fps_" + why, lambda: bkv.fps_gather(self.obs, self.nb, n=n, picks=picks))
        self.obs_len = min(self.nb, n)
        self._log("fps", why=why, src=src, picks=picks)

    # ---- the phase machine -----------------------------------------------------
    def prefill(self, K, V, q_pre):
        """Prompt keys/values [LB, Hkv, T, D] and pre-RoPE queries [LB, Hq, T, D]."""
        T = K.shape[2]
        if T > self.B_max - self.nr:
            raise ValueError("the prompt must end before the recent window")
        self.K[:, :, :T] = K
        self.V[:, :, :T] = V
        self.L = self.t = T
        if self.mode == "ns":
            # bkv_beacon_update takes queries t-major, so consecutive prompt
            # chunks give the same running means as one call; chunks keep
            # each call's element count within the library's 32-bit limit
            tc = max(1, (2 ** 31 - 1) // (self.LB * self.Hq * self.D))
            for t0 in range(0, T, tc):
                qc = q_pre[:, :, t0:t0 + tc].contiguous()
                self._call("beacon_update", lambda: bkv.beacon_update(self.dims, qc, self.beacons, self.counts))
        if self.mode == "initial":
            # every one of the first min(n_beacon, T) rows is picked (m >= n): the
            # gather widens them into the beacon layout and sets their counts
            self._call("beacon_widen", lambda: bkv.fps_gather(
                q_pre, self.nb, n=min(self.nb, T), dst=self.beacons.view(self.LB, self.Hq, self.nb, self.D),
                counts=self.counts.view(self.LB, self.Hq, self.nb)))
        if self.mode == "beacon":
            picks = torch.empty(self.LB, self.Hq, min(self.nb, T), dtype=torch.int32, device=K.device)
            self._call("fps_prefill", lambda: bkv.fps_gather(q_pre, self.nb, dst=self.obs, picks=picks))
            self.obs_len = min(self.nb, T)
            self._log("fps", why="prefill", src=q_pre.clone() if self.record else None, picks=picks)

    def step(self, k, v, q_pre, q_rope):
        """One decoding step: k, v [LB, Hkv, D]; q_pre, q_rope [LB, Hq, D].
        Returns True when the step evicted."""
        self.K[:, :, self.L] = k
        self.V[:, :, self.L] = v
        self.L += 1
        self.t += 1
        L, nb, nr = self.L, self.nb, self.nr
        if self.mode == "ns":
            q_new = q_pre.reshape(self.LB, self.Hq, 1, self.D).contiguous()
            self._call("beacon_update", lambda: bkv.beacon_update(self.dims, q_new, self.beacons, self.counts))
        if self.mode == "beacon":
            if L <= self.B_max - nr:
                self.obs[:, :, self.obs_len] = q_pre
                self.obs_len += 1
                if self.obs_len >= nb + nr:
                    self._compress(self.obs_len, "fill")
            if L == self.B_max - nr:
                # freeze: the buffer's FPS selection is the beacon set, kept
                # pre-RoPE in the buffer's first rows and widened for scoring
                self._compress(self.obs_len, "freeze")
                self._call("beacon_widen", lambda: bkv.fps_gather(
                    self.obs, nb, n=self.obs_len, dst=self.beacons.view(self.LB, self.Hq, nb, self.D),
                    counts=self.counts.view(self.LB, self.Hq, nb)))
                self.n_rec = 0
        if self.B_max - nr < L <= self.B_max:
            self.recent_rope[:, :, self.n_rec] = q_rope
            self.recent_pre[:, :, self.n_rec] = q_pre
            self.n_rec += 1
        if L == self.B_max:
            self._evict()
            return True
        return False

    def _evict(self):
        rc, rs = self.rope_table(self.t - 1)  # beacons rotated to the current step
        pre = (self.K.clone(), self.V.clone()) if self.record else None
        if self.compaction == "order":
            self._call("evict", lambda: bkv.evict(self.dims, self.K, self.V, self.recent_rope, self.beacons,
                                                  self.counts, self.ws, kept=self.kept, scores=self.scores,
                                                  rope_cos=rc, rope_sin=rs))
        else:
            def evict_fill():
                bkv.score(self.dims, self.K, self.recent_rope, self.beacons, self.counts, self.scores, self.ws,
                          rope_cos=rc, rope_sin=rs)
                bkv.topk(self.dims, self.scores, self.sel)
                bkv.compact_fill(self.dims, self.K, self.V, self.sel, self.kept, self.ws)
            self._call("evict", evict_fill)
        self._log("evict", before=pre, q_win=self.recent_rope.clone() if self.record else None,
                  beacons=self.beacons.clone() if self.record else None,
                  counts=self.counts.clone() if self.record else None, rope=(rc, rs), kept=self.kept.clone(),
                  scores=self.scores.clone() if self.record else None)
        self.L = self.B_min
        if self.mode == "beacon":
            # the buffer becomes the beacon set plus the recent queries, then FPS
            n = self.obs_len
            self.obs[:, :, n:n + self.n_rec] = self.recent_pre[:, :, :self.n_rec]
            self._compress(n + self.n_rec, "merge")
        self.n_rec = 0
