"""CPU pins of the quality-diagnostic metrics (planted-key retention and
max-cosine coverage of future queries): brute force over tiny inputs with
Python loops, and hand-made cases whose answers are known."""
import math

import numpy as np
import torch

from paper_2609_04971_amd import diagnostics


def test_retention_hand_made():
    # two heads: head 0 keeps planted keys 0 and 2 of 4, head 1 keeps all four
    pos = torch.tensor([[[0, 2, 7, 9, 11]], [[3, 1, 0, 2, 8]]])
    assert diagnostics.retention(pos, 4) == (2 / 4 + 4 / 4) / 2


def test_coverage_hand_made():
    # one head, observation rows e0 and e1 (and an empty slot), queries e0,
    # (e0 + e1)/sqrt2 and -e0; only the first and last count
    obs = torch.tensor([[[1.0, 0, 0], [0, 1.0, 0], [0, 0, 0]]])
    fut = torch.tensor([[[2.0, 0, 0], [1.0, 1.0, 0], [-1.0, 0, 0]]])
    mask = torch.tensor([[True, False, True]])
    # -e0 against e0 is -1, against e1 is 0: best 0 (the empty slot is ignored)
    assert math.isclose(diagnostics.coverage(obs, fut, mask), (1.0 + 0.0) / 2, abs_tol=1e-7)
    all3 = diagnostics.coverage(obs, fut, torch.ones_like(mask))
    assert math.isclose(all3, (1.0 + 1 / math.sqrt(2) + 0.0) / 3, abs_tol=1e-6)
    assert math.isnan(diagnostics.coverage(obs, fut, torch.zeros_like(mask)))


def test_coverage_brute_force():
    rng = np.random.default_rng(0)
    H, R, F, D = 3, 5, 7, 6
    obs = rng.standard_normal((H, R, D))
    obs[1, 2] = 0.0
    fut = rng.standard_normal((H, F, D))
    mask = rng.random((H, F)) < 0.6
    vals = []
    for h in range(H):
        for f in range(F):
            if not mask[h, f]:
                continue
            best = -2.0
            for r in range(R):
                no = math.sqrt(sum(x * x for x in obs[h, r]))
                if no == 0:
                    continue
                nf = math.sqrt(sum(x * x for x in fut[h, f]))
                best = max(best, sum(a * b for a, b in zip(obs[h, r], fut[h, f])) / (no * nf))
            vals.append(best)
    got = diagnostics.coverage(torch.tensor(obs), torch.tensor(fut), torch.tensor(mask))
    assert math.isclose(got, sum(vals) / len(vals), abs_tol=1e-6)


def test_retention_brute_force():
    rng = np.random.default_rng(1)
    pos = rng.permutation(200)[:120].reshape(1, 1, 120).repeat(3, 0)
    for h in range(3):
        pos[h, 0] = rng.permutation(200)[:120]
    want = np.mean([sum(1 for p in pos[h, 0] if p < 25) / 25 for h in range(3)])
    assert math.isclose(diagnostics.retention(torch.tensor(pos), 25), want, abs_tol=1e-7)
