"""The allocation-free evaluation entry point (hwsel_evaluate_noalloc), through
the C ABI, against hwsel_evaluate on the same inputs: every output bit-exact
(both run the same kernels; only where the intermediates live differs), on
two calls in a row with the second on a smaller input, so that the second
call shows nothing of the first survives in the shared scratch array."""
import numpy as np
import pytest
import torch

import oracle
import synth
from _gpu_util import say
from paper_2609_35587_amd import hwsel

pytestmark = pytest.mark.gpu


def up(a):
    return hwsel.to_device(np.ascontiguousarray(a))


def case(seed: int, P: int, max_len: int, k: int):
    rng = np.random.default_rng(seed)
    seg = synth.ragged_segments(rng, P, max_len)
    R = int(seg[-1])
    rt = rng.lognormal(0, 0.3, R).astype(np.float32)
    rt[rng.random(R) < 0.02] = np.inf
    rt[rng.random(R) < 0.01] = np.nan
    rt[rng.random(R) < 0.1] = 1.0
    idx, _ = oracle.topk(synth.random_scores(rng, R, tie_frac=0.3), seg, k)
    return up(rt), up(seg), up(idx)


def same(a: torch.Tensor, b: torch.Tensor) -> bool:
    return bool(torch.equal(a.cpu().view(torch.uint8), b.cpu().view(torch.uint8)))


def test_noalloc_matches_evaluate_on_two_calls():
    # first call: more problems than the one-workgroup path takes (selection
    # and aggregation kernels); second: fewer rows and problems (one-workgroup
    # path), run after the first on the same scratch array
    for seed, P, max_len, k in [(11, 5000, 64, 10), (12, 300, 40, 5)]:
        say(f"noalloc evaluate seed={seed} P={P} k={k}")
        rt, seg, idx = case(seed, P, max_len, k)
        ref = hwsel.hwsel_evaluate(rt, seg, idx)
        got = hwsel.hwsel_evaluate_noalloc(rt, seg, idx)
        torch.cuda.synchronize()
        for name, a, b in zip(("out", "regret", "rank", "ybar"), got, ref):
            assert same(a, b), f"{name} differs (P={P})"
    # the largest admitted P still runs, and one past it is refused
    rt, seg, idx = case(13, hwsel.HWSEL_EVAL_NOALLOC_MAX_P, 2, 1)
    ref = hwsel.hwsel_evaluate(rt, seg, idx)
    got = hwsel.hwsel_evaluate_noalloc(rt, seg, idx)
    for name, a, b in zip(("out", "regret", "rank", "ybar"), got, ref):
        assert same(a, b), f"{name} differs at the largest P"
    with pytest.raises(hwsel.HwselError):
        hwsel.hwsel_evaluate_noalloc(rt, torch.zeros(hwsel.HWSEL_EVAL_NOALLOC_MAX_P + 2, dtype=torch.int64,
                                                     device=rt.device),
                                     torch.zeros((hwsel.HWSEL_EVAL_NOALLOC_MAX_P + 1, 1), dtype=torch.int32,
                                                 device=rt.device))
