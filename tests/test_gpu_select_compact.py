"""GPU parity of bkv_topk and bkv_compact: bit-exact against the oracle when
both are fed the same generator-made scores / indices."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import host, raw_bits, say
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth

pytestmark = pytest.mark.gpu


def _scores(P, N, seed, kind):
    g = torch.Generator().manual_seed(seed)
    if kind == "normal":
        s = -torch.rand(P, N, generator=g) * 12
    elif kind == "ties":  # few distinct values: radix select must split ties by index
        s = -torch.randint(0, 7, (P, N), generator=g).float() / 4
    elif kind == "equal":
        s = torch.full((P, N), -3.0)
    elif kind == "signed-zero":
        s = torch.where(torch.rand(P, N, generator=g) < 0.5, torch.tensor(-0.0), torch.tensor(0.0))
        s[:, ::7] = -1.0
    elif kind == "wide":  # spans many binades, both signs, huge and tiny
        s = torch.randn(P, N, generator=g) * torch.exp(torch.randn(P, N, generator=g) * 20)
    elif kind.startswith("cluster"):  # the threshold inside a tight cluster of n nearly equal scores
        n = int(kind[7:])
        s = -torch.rand(P, N, generator=g) * 12
        s[:, 1:1 + n] = -1.5 - torch.rand(P, n, generator=g) * 1e-3
    elif kind == "minus-inf":
        s = -torch.rand(P, N, generator=g)
        s[:, ::3] = float("-inf")
    elif kind == "plus-inf":  # a few +inf: kept whatever the threshold
        s = -torch.rand(P, N, generator=g) * 12
        s[:, 7::97] = float("inf")
    elif kind == "far":  # every score far below the split selection's bin range
        s = -1000.0 - torch.rand(P, N, generator=g) * 100
    elif kind == "mixed":  # heads alternate between spread scores and one value
        s = -torch.rand(P, N, generator=g) * 12
        s[1::2] = -2.5
    return s.contiguous()


TOPK = [
    # (B, Hkv, N, budget, W, n_prefix, kind)
    (1, 2, 512, 128, 16, 0, "normal"),
    (2, 3, 1000, 256, 8, 2, "ties"),
    (1, 4, 777, 300, 5, 4, "equal"),
    (1, 2, 300, 250, 0, 0, "signed-zero"),
    (2, 2, 4096, 2048, 32, 0, "wide"),
    (1, 2, 5000, 100, 0, 0, "minus-inf"),
    (1, 3, 100, 100, 4, 1, "normal"),      # N == budget: keep all
    (1, 3, 60, 100, 4, 1, "normal"),       # N < budget
    (1, 2, 500, 20, 12, 8, "normal"),      # k_sel == 0: forced tokens only
    (1, 1, 1, 8, 1, 0, "normal"),
    (2, 2, 65536, 8192, 128, 0, "normal"),  # the largest configuration's shape
    (16, 8, 32768, 4096, 32, 0, "ties"),    # the benchmark configuration's shape
    (16, 8, 32768, 4096, 32, 0, "normal"),  # a few dozen candidates after the first digit
    (4, 2, 32768, 4096, 32, 3, "cluster600"),   # hundreds of candidates, ranked directly
    (4, 2, 32768, 4096, 32, 3, "cluster3000"),  # too many to rank: radix passes continue
    (2, 2, 20000, 5000, 16, 0, "cluster1000"),
]


# heads split over several workgroups (a workspace given, few heads, N > 8192)
TOPK_SPLIT = [
    (1, 2, 20000, 3000, 16, 3, "normal"),     # ragged last slice
    (1, 2, 9000, 100, 20, 5, "normal"),       # just past the shortest split head
    (1, 2, 20000, 20, 12, 8, "normal"),       # k_sel == 0
    (2, 2, 20000, 2000, 8, 0, "equal"),       # every head ties in bulk: one workgroup selects it
    (2, 2, 20000, 2000, 8, 0, "mixed"),       # split heads beside whole-head ones
    (1, 2, 20000, 2000, 8, 0, "wide"),        # half the scores above the range
    (1, 2, 20000, 2000, 8, 0, "far"),         # all below the range
    (1, 2, 20000, 2000, 8, 0, "plus-inf"),
    (1, 2, 20000, 2000, 8, 0, "cluster300"),  # hundreds of candidates in the threshold bin
    (2, 2, 32768, 4096, 32, 2, "ties"),
    (4, 8, 65536, 8192, 128, 0, "normal"),    # the 64K layer's shape (32 heads of 16 slices)
]


def _topk_ws(d, split):
    if not split or bkv.workspace_bytes(d, bkv.OP_TOPK) == 0:
        return None
    return bkv.workspace(d, bkv.OP_TOPK)


@pytest.mark.parametrize("split", [False, True], ids=["one-wg", "ws"])
@pytest.mark.parametrize("case", TOPK + TOPK_SPLIT, ids=[f"{c[6]}-B{c[0]}H{c[1]}-N{c[2]}-b{c[3]}" for c in TOPK + TOPK_SPLIT])
def test_topk_bit_exact(case, split):
    B, Hkv, N, budget, W, n_prefix, kind = case
    d = bkv.dims(B=B, Hq=Hkv, Hkv=Hkv, D=128, N=N, W=W, C=1, budget=budget, n_prefix=n_prefix)
    s = _scores(B * Hkv, N, seed=N + budget, kind=kind).view(B, Hkv, N)
    ws = _topk_ws(d, split)
    say(f"topk {case} workspace={ws is not None}")
    kept = torch.full((B, Hkv, d.n_keep), -1, dtype=torch.int32, device="cuda")
    bkv.topk(d, s.cuda(), kept, ws)
    got = host(kept).numpy()
    want = oracle.topk(s.double().numpy(), budget, W, n_prefix)
    np.testing.assert_array_equal(got, want)


def test_topk_split_calls_in_a_row_and_unstamped_workspace():
    # the split selection leaves its histogram clear for the next call on the
    # same workspace; a workspace without the stamp falls back to one
    # workgroup per head and stays exact
    d = bkv.dims(B=2, Hq=2, Hkv=2, D=128, N=30000, W=16, C=1, budget=3000, n_prefix=1)
    ws = bkv.workspace(d, bkv.OP_TOPK)
    assert ws.numel() >= bkv.workspace_bytes(d, bkv.OP_TOPK) > 0
    for seed, kind in [(1, "normal"), (2, "cluster200"), (3, "normal")]:
        s = _scores(4, d.N, seed=seed, kind=kind).view(2, 2, d.N)
        kept = torch.full((2, 2, d.n_keep), -1, dtype=torch.int32, device="cuda")
        say(f"topk split, call with seed {seed}")
        bkv.topk(d, s.cuda(), kept, ws)
        np.testing.assert_array_equal(host(kept).numpy(), oracle.topk(s.double().numpy(), d.budget, d.W, 1))
    raw = torch.zeros_like(ws)
    s = _scores(4, d.N, seed=9, kind="normal").view(2, 2, d.N)
    kept = torch.full((2, 2, d.n_keep), -1, dtype=torch.int32, device="cuda")
    bkv.topk(d, s.cuda(), kept, raw)
    np.testing.assert_array_equal(host(kept).numpy(), oracle.topk(s.double().numpy(), d.budget, d.W, 1))


def _kv(P, Ncap, D, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    if dtype == torch.bfloat16:  # any 16-bit pattern, NaNs included: the copy is bitwise
        bits = torch.randint(-32768, 32768, (P, Ncap, D), generator=g, dtype=torch.int16)
        return bits.view(torch.bfloat16)
    return torch.randint(-2**31, 2**31 - 1, (P, Ncap, D), generator=g, dtype=torch.int32).view(torch.float32)


def _patterns(N, n, P, seed):
    pats = {
        "random": synth.sorted_subsets(P, N, n, seed=seed, forced_tail=min(8, n)),
        "every-other": torch.arange(0, 2 * n, 2, dtype=torch.int32).repeat(P, 1) if 2 * n <= N else None,
        "all-but-row-0": torch.arange(1, n + 1, dtype=torch.int32).repeat(P, 1) if n + 1 <= N else None,
        "identity": torch.arange(n, dtype=torch.int32).repeat(P, 1),
        "tail-block": torch.arange(N - n, N, dtype=torch.int32).repeat(P, 1),
        "one-gap": torch.cat([torch.arange(0, n // 2), torch.arange(n // 2 + 1, n + 1)]).int().repeat(P, 1)
        if n + 1 <= N else None,
    }
    return {k: v for k, v in pats.items() if v is not None}


COMPACT = [
    # (B, Hkv, N, N_cap, D, dtype, budget)
    (1, 2, 512, 512, 64, torch.float32, 128),
    (2, 2, 1000, 1100, 128, torch.bfloat16, 256),
    (1, 3, 777, 777, 64, torch.bfloat16, 300),
    (1, 2, 300, 300, 128, torch.float32, 100),
    (2, 4, 4096, 4096, 128, torch.bfloat16, 2048),
    (1, 2, 130, 130, 128, torch.bfloat16, 65),    # one partial segment
    (1, 2, 300, 300, 128, torch.bfloat16, 129),   # one full 128-row segment + a 1-row segment
]


@pytest.mark.parametrize("case", COMPACT, ids=[f"N{c[2]}-D{c[4]}-{str(c[5])[6:]}-b{c[6]}" for c in COMPACT])
def test_compact_bit_exact(case):
    B, Hkv, N, Ncap, D, dt, budget = case
    P = B * Hkv
    d = bkv.dims(B=B, Hq=Hkv, Hkv=Hkv, D=D, N=N, N_cap=Ncap, W=0, C=1, budget=budget,
                 dtype="bf16" if dt == torch.bfloat16 else "fp32")
    n = d.n_keep
    ws = bkv.workspace(d, bkv.OP_COMPACT)
    for name, kept in _patterns(N, n, P, seed=N).items():
        K0 = _kv(P, Ncap, D, dt, seed=1).view(B, Hkv, Ncap, D)
        V0 = _kv(P, Ncap, D, dt, seed=2).view(B, Hkv, Ncap, D)
        kept = kept.view(B, Hkv, n).contiguous()
        Kd, Vd = K0.cuda(), V0.cuda()
        say(f"compact {case} {name}")
        bkv.compact(d, Kd, Vd, kept.cuda(), ws)
        Kr, Vr = oracle.compact(K0, V0, kept.numpy())
        np.testing.assert_array_equal(raw_bits(Kd), Kr.view(raw_bits(Kd).dtype), err_msg=f"K {name}")
        np.testing.assert_array_equal(raw_bits(Vd), Vr.view(raw_bits(Vd).dtype), err_msg=f"V {name}")
    assert bkv.device_status(ws) == bkv.OK


def test_compact_repeated_hazard_patterns_deterministic():
    # rows that move onto rows other segments still have to read: run the
    # hazard patterns many times and require identical bits every time
    B, Hkv, N, D = 4, 8, 8192, 128
    d = bkv.dims(B=B, Hq=Hkv, Hkv=Hkv, D=D, N=N, W=0, C=1, budget=4096)
    ws = bkv.workspace(d, bkv.OP_COMPACT)
    K0 = _kv(B * Hkv, N, D, torch.bfloat16, seed=3).view(B, Hkv, N, D).cuda()
    pats = _patterns(N, 4096, B * Hkv, seed=5)
    refs = {}
    for name, kept in pats.items():
        kept = kept.view(B, Hkv, 4096).contiguous()
        Kr, _ = oracle.compact(host(K0), host(K0), kept.numpy())
        refs[name] = (kept.cuda(), torch.from_numpy(Kr.view(np.int16)).cuda())
    for rep in range(20):
        for name, (kept, Kr) in refs.items():
            Kd, Vd = K0.clone(), K0.clone()
            if rep == 0:
                say(f"compact hazard {name}")
            bkv.compact(d, Kd, Vd, kept, ws)
            assert torch.equal(Kd.view(torch.int16), Kr), f"rep {rep} {name}"
            assert torch.equal(Kd.view(torch.int16), Vd.view(torch.int16))
    assert bkv.device_status(ws) == bkv.OK


def test_compact_rejects_non_ascending_kept():
    # kept[i] >= i and inside [0, N) everywhere, but one pair of head 1 is out
    # of order: the segment holding it must move nothing and raise the device
    # error, while head 0 compacts as usual
    B, Hkv, N, D, budget = 1, 2, 512, 128, 128
    d = bkv.dims(B=B, Hq=Hkv, Hkv=Hkv, D=D, N=N, W=0, C=1, budget=budget)
    ws = bkv.workspace(d, bkv.OP_COMPACT)
    kept = torch.arange(0, 2 * budget, 2, dtype=torch.int32).repeat(B * Hkv, 1).view(B, Hkv, budget).contiguous()
    kept[0, 1, 10], kept[0, 1, 11] = int(kept[0, 1, 11]), int(kept[0, 1, 10])  # 22, 20
    assert int(kept[0, 1, 11]) >= 11
    K0 = _kv(B * Hkv, N, D, torch.bfloat16, seed=7).view(B, Hkv, N, D)
    V0 = _kv(B * Hkv, N, D, torch.bfloat16, seed=8).view(B, Hkv, N, D)
    Kd, Vd = K0.cuda(), V0.cuda()
    say("compact non-ascending kept")
    bkv.compact(d, Kd, Vd, kept.cuda(), ws)
    assert bkv.device_status(ws) == bkv.ERR_DEVICE
    Kr, Vr = oracle.compact(K0[:, :1], V0[:, :1], kept[:, :1].numpy())
    np.testing.assert_array_equal(raw_bits(Kd[:, :1]), Kr.view(np.uint16))
    np.testing.assert_array_equal(raw_bits(Vd[:, :1]), Vr.view(np.uint16))
    # the segment of head 1 holding the bad pair (rows 0..127, the whole head here): untouched
    np.testing.assert_array_equal(raw_bits(Kd[0, 1, :budget]), raw_bits(K0[0, 1, :budget]))
