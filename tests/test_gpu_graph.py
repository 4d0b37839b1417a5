"""The loss-gradient step recorded into a HIP graph (stream capture through
torch.cuda.graph) and replayed: every replay, with new pixel ids copied into
the captured buffer and the program's own synchronisations between replays,
gives the eager path's loss, pose gradient and momentum-updated poses bit for
bit (same kernels, same inputs, fixed-order sums); a call that would need the
host (the sample totals of a batch too large for one buffer) refuses capture
instead of breaking it."""
import sys

import numpy as np
import pytest

from paper_2210_10108_amd import synth
from tests import gpu_common as G

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def announce(request):
    sys.stderr.write(f"\n[gpu] {request.node.nodeid}\n")
    sys.stderr.flush()
    yield


@pytest.fixture(scope="module")
def pn():
    from paper_2210_10108_amd import pnerf
    pnerf.lib()
    return pnerf


@pytest.mark.parametrize("name,K,P", [("tiny32", 4, 256), ("ngp800_uniform", 4, 1024)])
def test_graph_replay_matches_eager_steps(pn, name, K, P):
    import torch
    case = G.make_case(name, K=K, P=P)
    w = case.w
    obs = torch.rand(w.height, w.width, 3, generator=torch.Generator().manual_seed(1)).cuda()
    batches = [G.to_dev(synth.pixel_batch(0, i, K, P, w.width, w.height)) for i in range(4)]
    f = pn.Field(case.spec)
    poses0 = G.to_dev(case.poses)
    poses, mom = poses0.clone(), torch.zeros(K, 6, device="cuda")
    pix = batches[0].clone()
    loss = torch.empty(K, device="cuda")
    dpose = torch.empty(K, 6, device="cuda")

    def step():
        f.render_loss_grad(poses, pix, obs, case.intr, loss, dpose)
        pn.step_momentum(poses, mom, dpose, 1e-2, 0.9)

    eager = []
    for b in batches:
        pix.copy_(b)
        step()
        torch.cuda.synchronize()
        eager.append((loss.cpu().numpy(), dpose.cpu().numpy(), poses.cpu().numpy()))
    poses.copy_(poses0)
    mom.zero_()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    assert np.array_equal(poses.cpu().numpy(), case.poses)  # recorded, not run
    for i, b in enumerate(batches):
        pix.copy_(b)
        g.replay()
        torch.cuda.synchronize()
        got = (loss.cpu().numpy(), dpose.cpu().numpy(), poses.cpu().numpy())
        for a, e in zip(got, eager[i]):
            assert np.array_equal(a, e), (i, np.abs(a - e).max())
    f.close()


def test_capture_refuses_a_batch_that_needs_the_host(pn):
    import torch
    case = G.make_case("tiny32", K=4, P=256)
    # a budget below the batch's worst case: the call must read the totals
    f = pn.Field(case.spec, max_workspace_bytes=3_000_000)
    poses = G.to_dev(case.poses)
    pix = G.to_dev(case.pix)
    obs = torch.zeros(32, 32, 3, device="cuda")
    loss = torch.empty(4, device="cuda")
    dpose = torch.empty(4, 6, device="cuda")
    f.render_loss_grad(poses, pix, obs, case.intr, loss, dpose)  # eager works
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with pytest.raises(pn.PnerfError, match="stream capture"):
        with torch.cuda.graph(g):
            f.render_loss_grad(poses, pix, obs, case.intr, loss, dpose)
    torch.cuda.synchronize()
    f.render_loss_grad(poses, pix, obs, case.intr, loss, dpose)  # and still works after
    torch.cuda.synchronize()
    assert np.isfinite(loss.cpu().numpy()).all()
    f.close()
