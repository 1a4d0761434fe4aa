"""GPU parity of bkv_compact_fill (hole-filling compaction) against the
oracle: K, V and src_of bit-exact on the same kept sets, over sparse and
dense selections, kept rows all at the front or all past n, both dtypes,
both head sizes and the benchmark's layer shape; a kept array that is not
ascending moves nothing and is reported."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import host, say
import paper_2609_04971_amd as bkv
from paper_2609_04971_amd import synth


pytestmark = pytest.mark.gpu


def _kv(P, Ncap, D, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    if dtype == torch.bfloat16:  # any 16-bit pattern: the copy is bitwise
        return torch.randint(-32768, 32768, (P, Ncap, D), generator=g, dtype=torch.int16).view(torch.bfloat16)
    return torch.randint(-2**31, 2**31 - 1, (P, Ncap, D), generator=g, dtype=torch.int32).view(torch.float32)


def _kept(kind, P, N, n, seed):
    if kind == "random":
        return synth.sorted_subsets(P, N, n, seed=seed, forced_tail=min(8, n))
    if kind == "identity":
        return torch.arange(n, dtype=torch.int32).repeat(P, 1)
    if kind == "tail-block":  # every row past n: all positions are holes
        return torch.arange(N - n, N, dtype=torch.int32).repeat(P, 1)
    if kind == "front-heavy":  # 7/8 of the rows in place, the rest from the tail (a periodic eviction)
        g = torch.Generator().manual_seed(seed)
        out = []
        for _ in range(P):
            front = torch.randperm(n, generator=g)[: n - n // 8]
            tail = n + torch.randperm(N - n, generator=g)[: n // 8]
            out.append(torch.cat([front, tail]).sort().values)
        return torch.stack(out).int()
    raise ValueError(kind)


CASES = [
    # (B, Hkv, N, N_cap, D, dtype, budget, kind)
    (1, 2, 512, 512, 64, torch.float32, 128, "random"),
    (2, 2, 1000, 1100, 128, torch.bfloat16, 256, "random"),
    (1, 3, 777, 777, 64, torch.bfloat16, 300, "tail-block"),
    (1, 2, 300, 300, 128, torch.float32, 100, "identity"),
    (2, 4, 4096, 4096, 128, torch.bfloat16, 3584, "front-heavy"),
    (1, 2, 130, 130, 128, torch.bfloat16, 65, "random"),  # one full 64-row item and a 1-row item
    (16, 8, 32768, 32768, 128, torch.bfloat16, 4096, "random"),  # the benchmark layer's shape
]


@pytest.mark.parametrize("case", CASES, ids=[f"N{c[2]}-D{c[4]}-{str(c[5])[6:]}-b{c[6]}-{c[7]}" for c in CASES])
def test_compact_fill_bit_exact(case):
    B, Hkv, N, Ncap, D, dt, budget, kind = case
    d = bkv.dims(B=B, Hq=Hkv, Hkv=Hkv, D=D, N=N, N_cap=Ncap, W=0, C=1, budget=budget,
                 dtype="bf16" if dt == torch.bfloat16 else "fp32")
    n = d.n_keep
    say(f"compact_fill {case}")
    K, V = _kv(B * Hkv, Ncap, D, dt, N).view(B, Hkv, Ncap, D), _kv(B * Hkv, Ncap, D, dt, N + 1).view(B, Hkv, Ncap, D)
    kept = _kept(kind, B * Hkv, N, n, seed=N).view(B, Hkv, n)
    Kr, Vr, src_ref, moved = oracle.compact_fill(K, V, kept.numpy(), N=N)
    Kd, Vd, kd = K.cuda(), V.cuda(), kept.cuda()
    src = torch.full((B, Hkv, n), -1, dtype=torch.int32, device="cuda")
    ws = bkv.workspace(d, bkv.OP_COMPACT)
    bkv.compact_fill(d, Kd, Vd, kd, src, ws)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.OK
    assert np.array_equal(host(src).numpy(), src_ref)
    iv = np.int16 if dt == torch.bfloat16 else np.int32
    assert np.array_equal(host(Kd).view(torch.int16 if iv is np.int16 else torch.int32).numpy(), Kr.view(iv))
    assert np.array_equal(host(Vd).view(torch.int16 if iv is np.int16 else torch.int32).numpy(), Vr.view(iv))
    say(f"  rows moved per head: mean {moved.mean():.1f} of {n}")


def test_compact_fill_rejects_unsorted_kept():
    B, Hkv, N, D, budget = 1, 2, 400, 128, 100
    d = bkv.dims(B=B, Hq=Hkv, Hkv=Hkv, D=D, N=N, W=0, C=1, budget=budget)
    K = _kv(B * Hkv, N, D, torch.bfloat16, 5).view(B, Hkv, N, D)
    kept = _kept("random", B * Hkv, N, budget, seed=3).view(B, Hkv, budget).clone()
    kept[0, 1, 10] = kept[0, 1, 9]  # a repeated index on head 1
    Kd, kd = K.cuda(), kept.cuda()
    src = torch.full((B, Hkv, budget), -1, dtype=torch.int32, device="cuda")
    ws = bkv.workspace(d, bkv.OP_COMPACT)
    bkv.compact_fill(d, Kd, Kd.clone(), kd, src, ws)
    torch.cuda.synchronize()
    assert bkv.device_status(ws) == bkv.ERR_DEVICE
    assert np.array_equal(host(src)[0, 1].numpy(), np.arange(budget))  # the bad head moved nothing
    assert torch.equal(host(Kd)[0, 1].view(torch.int16), K[0, 1].view(torch.int16))
