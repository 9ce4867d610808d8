"""The 57-case sweep (Section 4's benchmark shape) on an MI355X at full size,
in the launch configuration the benchmark times: beta = 1 results sampled
against the oracle element by element, and the alpha = 1, beta = 0 copy
checked whole by a property that holds at any size -- B is a permutation of
A, so both sort to the same bits."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_1704_04374_amd import hptt
from paper_1704_04374_amd.workloads import inputs, sweep57

pytestmark = pytest.mark.gpu

CASES = sweep57()


def test_sweep_full_size():
    seen = set()
    shared = 0
    for w in CASES:
        print(f"[sweep] {w.describe()}", flush=True)
        A, B0 = inputs(w)
        dA, dB = A.cuda(), B0.cuda()
        p = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype)
        seen.add(p.info["kernel"])
        shared += p.info["shared_runs"] > 0
        p.exec(dA, dB)
        torch.cuda.synchronize()
        rng = np.random.default_rng(w.seed_a)
        offs = np.concatenate([[0, w.numel - 1], rng.integers(0, w.numel, 4000)])
        got = dB[torch.from_numpy(offs).cuda()].cpu().numpy()
        want = orc.sample(A.numpy(), w.size_a, w.perm, w.alpha, w.beta, B0.numpy(), offs)
        assert np.array_equal(got, want), p.describe()
        # alpha = 1, beta = 0: a pure permutation of A's bits, whole
        c = hptt.create_plan(w.perm, w.size_a, 1.0, 0.0, w.dtype)
        dB.fill_(float("nan"))
        c.exec(dA, dB)
        torch.cuda.synchronize()
        ia, ib = dA.view(torch.int32), dB.view(torch.int32)
        assert torch.equal(torch.sort(ia).values, torch.sort(ib).values), c.describe()
        got = dB[torch.from_numpy(offs).cuda()].cpu().numpy()
        want = orc.sample(A.numpy(), w.size_a, w.perm, 1.0, 0.0, None, offs)
        assert np.array_equal(got, want), c.describe()
        del dA, dB
    assert {"tile", "stream"} <= seen
    assert shared >= 10  # tiles whose runs share indices
