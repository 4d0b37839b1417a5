"""pnerf_resample_hypotheses_noalloc through the C ABI: the same results as
pnerf_resample_hypotheses (bit for bit: the same kernels on the same inputs)
on two calls in a row, the second with fewer hypotheses, at the largest K the
static scratch holds, and a capacity error past it."""
import math
import sys

import numpy as np
import pytest

from paper_2210_10108_amd import synth

pytestmark = pytest.mark.gpu


def _case(K, dim, seed):
    w = synth.WORKLOADS["tiny32"]
    poses = synth.perturb_poses(synth.ground_truth_pose(w, 0), K, 40, 0.3, seed)
    rng = np.random.default_rng(seed)
    state = rng.normal(size=(K, dim)).astype(np.float32)
    loss = rng.uniform(0, 1, K).astype(np.float32)
    if K > 10:
        loss[[2, 7]] = np.nan
        loss[5] = loss[4]
    return poses, state, loss


def test_noalloc_resample_matches_the_allocating_entry_point():
    import torch
    from oracle import oracle as O
    from paper_2210_10108_amd import pnerf
    pnerf.lib()
    dev = torch.device("cuda:0")
    sr, st = math.radians(5), 0.03
    # two calls in a row, the second smaller; then the largest K
    for K, keep, dim, rnd in [(1024, 0.10, 16, 3), (37, 0.3, 6, 4), (65535, 0.25, 6, 5)]:
        sys.stderr.write(f"[gpu] noalloc resample K={K}\n")
        sys.stderr.flush()
        poses, state, loss = _case(K, dim, K)
        d_loss = torch.from_numpy(loss).to(dev)
        a_p, a_s = torch.from_numpy(poses).to(dev), torch.from_numpy(state).to(dev)
        b_p, b_s = torch.from_numpy(poses).to(dev), torch.from_numpy(state).to(dev)
        pnerf.resample_hypotheses(a_p, a_s, d_loss, keep, sr, st, 1234, rnd)
        pnerf.resample_hypotheses_noalloc(b_p, b_s, d_loss, keep, sr, st, 1234, rnd)
        torch.cuda.synchronize()
        assert np.array_equal(a_p.cpu().numpy(), b_p.cpu().numpy())
        assert np.array_equal(a_s.cpu().numpy(), b_s.cpu().numpy())
        # and both against the oracle (poses within one float32 ulp per step)
        if K <= 1024:
            p_ref, s_ref, _ = O.resample(poses, state, loss, keep, sr, st, 1234, rnd)
            assert np.allclose(b_p.cpu().numpy(), p_ref, atol=1e-6, rtol=0)
            assert np.array_equal(b_s.cpu().numpy(), s_ref)
    # beyond the static scratch: refused before anything is enqueued
    K = 65536
    poses, state, loss = _case(K, 6, 1)
    p = torch.from_numpy(poses).to(dev)
    with pytest.raises(pnerf.PnerfError) as e:
        pnerf.resample_hypotheses_noalloc(p, torch.from_numpy(state).to(dev),
                                          torch.from_numpy(loss).to(dev), 0.25, sr, st, 1, 1)
    assert e.value.status == pnerf.ERR_CAPACITY and "65535" in str(e.value)
    torch.cuda.synchronize()
    assert np.array_equal(p.cpu().numpy(), poses)
