"""Parity of the HIP path (through the C ABI) with the CPU oracle on the same
seeded inputs: sample indexing bit-exact, colour 2e-3 absolute, loss 1e-3
relative, pose gradient 1e-2 relative L2."""
import dataclasses
import math
import sys

import numpy as np
import pytest

from oracle import oracle as O
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


def gpu_march(pn, case, capacity):
    import torch
    f = pn.Field(case.spec)
    off, t, j = f.march(G.to_dev(case.poses), G.to_dev(case.pix), case.intr, capacity)
    torch.cuda.synchronize()
    out = off.cpu().numpy(), t.cpu().numpy(), j.cpu().numpy()
    f.close()
    return out


def check_march(pn, case):
    of = O.OracleField(case.spec)
    off_o, t_o, j_o, _ = of.march(case.poses, case.pix, case.intr)
    total = int(off_o[-1])
    off_g, t_g, j_g = gpu_march(pn, case, total + 100)
    assert np.array_equal(off_g, off_o)
    assert np.array_equal(t_g[:total].view(np.uint32), t_o.view(np.uint32))
    assert np.array_equal(j_g[:total], j_o)
    return total


# ---------------------------------------------------------------- indexing
def test_march_uniform_bitexact(pn):
    case = G.make_case("tiny32")
    assert check_march(pn, case) > 0


@pytest.mark.parametrize("pattern", ["checker", "sphere", "random", "empty", "full"])
def test_march_lattice_occupancy_bitexact(pn, pattern):
    R = 16
    case = G.make_case("tiny32", K=3, P=77, march_mode=1, step=math.sqrt(3) / 256,
                       max_samples=300, occ_res=R,
                       occ_bits=synth.occupancy_pattern(pattern, R, seed=4))
    n = check_march(pn, case)
    assert (n == 0) == (pattern == "empty")


def test_march_cap_bitexact(pn):
    case = G.make_case("tiny32", K=2, P=100, march_mode=1, step=math.sqrt(3) / 512,
                       max_samples=37, occ_res=8, occ_bits=synth.occupancy_pattern("full", 8))
    check_march(pn, case)


def test_march_ngp800_occ128_full_batch_bitexact(pn):
    # the 64 x 4096-ray batch with a structured 128^3 grid
    case = G.make_case("ngp800_occ128", occ_bits=synth.occupancy_pattern("sphere", 128))
    assert check_march(pn, case) > 1_000_000


def test_march_large_scene_camera_inside_box(pn):
    # [-2,2]^3 box with the camera at radius 2.5 often inside it: t_near = 0
    case = G.make_case("large4m_occ256", K=16, P=512, seed=3,
                       occ_bits=synth.occupancy_pattern("random", 256, seed=1))
    check_march(pn, case)


# ------------------------------------------------------------------ colour
def test_render_colour_tiny_full_image(pn):
    import torch
    case = G.make_case("tiny32")
    of = O.OracleField(case.spec)
    allpix = np.arange(32 * 32, dtype=np.int32)[None]
    ref = of.render(case.gt[None], allpix, case.intr)
    f = pn.Field(case.spec)
    rgb = f.render(G.to_dev(case.gt[None]), G.to_dev(allpix), case.intr)
    torch.cuda.synchronize()
    assert np.abs(rgb.cpu().numpy() - ref).max() <= G.COLOR_ATOL
    assert ref.max() > 0.05


def test_render_colour_ngp800(pn):
    import torch
    case = G.make_case("ngp800_uniform", K=4, P=1000)
    of = O.OracleField(case.spec)
    ref = of.render(case.poses, case.pix, case.intr)
    f = pn.Field(case.spec)
    rgb = f.render(G.to_dev(case.poses), G.to_dev(case.pix), case.intr)
    torch.cuda.synchronize()
    assert np.abs(rgb.cpu().numpy() - ref).max() <= G.COLOR_ATOL


# -------------------------------------------------------- loss and gradient
def run_loss_grad(pn, case, obs, max_ws=0, per_sample=False, backward=None):
    """GPU loss and gradient; with per_sample also each sample's (torque, force)
    share and each hypothesis's sample range (from the GPU's own ray offsets).
    backward: the field's backward pass (0: separate kernels, the default)."""
    import torch
    if backward is None:
        backward = 0
    f = pn.Field(case.spec, max_workspace_bytes=max_ws, overlap_chunks=1 if per_sample else 0,
                 backward=backward)
    poses, pix = G.to_dev(case.poses), G.to_dev(case.pix)
    loss, dpose = f.render_loss_grad(poses, pix, G.to_dev(obs), case.intr)
    torch.cuda.synchronize()
    n = f.last_sample_count()
    extra = {}
    if per_sample:
        extra["out6"] = f.inspect(3, n).cpu().numpy()
        extra["gh0"] = f.inspect(1, n).cpu().numpy()
        extra["gz"] = f.inspect(2, n).cpu().numpy()
        off, _, _ = f.march(poses, pix, case.intr, 0)
        extra["off"] = off.cpu().numpy()
    f.close()
    if per_sample:
        return loss.cpu().numpy(), dpose.cpu().numpy(), n, extra
    return loss.cpu().numpy(), dpose.cpu().numpy(), n


def oracle_subset(of, case, obs, hyps):
    hyps = list(hyps)
    return of.render_loss_grad(case.poses[hyps], case.pix[hyps], obs, case.intr, per_sample=True)


def check_full(pn, case, obs, ref, of, hyps=None, backward=0):
    """The whole batch on the GPU as one chunk; `ref` is the oracle's per-sample
    result for hypotheses `hyps` (all by default), computed by `of`."""
    import os
    loss, dpose, n, ex = run_loss_grad(pn, case, obs, per_sample=True, backward=backward)
    P = case.pix.shape[1]
    hyps = list(range(case.pix.shape[0])) if hyps is None else list(hyps)
    ranges = [(int(ex["off"][k * P]), int(ex["off"][(k + 1) * P])) for k in hyps]
    alt = G.Alt(of, case.poses[hyps], case.pix[hyps], obs, case.intr)
    label = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    per_sample = np.concatenate([ex["out6"], ex["gh0"][:, None], ex["gz"].reshape(-1, 3)], axis=1)
    return G.assert_loss_grad_close(loss, dpose, ref, hyps=hyps, gpu_samples=per_sample,
                                    gpu_ranges=ranges, alt=alt, label=label), ex


@pytest.mark.parametrize("overrides", [
    dict(),
    dict(background=(1.0, 1.0, 1.0)),
    dict(sh_dir_grad=1),
    dict(dense_coarse_levels=0),
])
@pytest.mark.parametrize("backward", [0, 2])
def test_loss_grad_tiny(pn, overrides, backward):
    case = G.make_case("tiny32", **overrides)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    # per sample: torque and force shares, and the stage values d loss / d h0
    # and d loss / d z, element by element (check_full)
    stats, ex = check_full(pn, case, obs, ref, of, backward=backward)
    assert stats["samples"] == int(ref["march"][0][-1])


@pytest.mark.parametrize("n_levels,dense,sh_dir", [(8, 0, 0), (12, 1, 0), (16, 1, 0), (16, 1, 1),
                                                    (12, 1, 1)])
@pytest.mark.parametrize("backward", [0, 2])
def test_loss_grad_level_counts(pn, monkeypatch, n_levels, dense, sh_dir, backward):
    """8, 12 and 16 levels: as many encoding work queues, fewer than, as many
    as and more than the 8 XCDs, with and without dense coarse levels; and
    the backward kernel built with the SH direction path at 12 and 16 levels."""
    name = f"tiny32_l{n_levels}"
    w = dataclasses.replace(synth.WORKLOADS["tiny32"], name=name, n_levels=n_levels,
                            log2_table=14)
    monkeypatch.setitem(synth.WORKLOADS, name, w)
    case = G.make_case(name, K=8, P=256, dense_coarse_levels=dense, sh_dir_grad=sh_dir)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    stats, _ = check_full(pn, case, obs, ref, of, backward=backward)
    assert stats["samples"] == int(ref["march"][0][-1])


@pytest.mark.parametrize("loss_type,param", [(1, 0.1), (2, 0.1), (3, 0.1), (4, 0.01), (5, 0.01),
                                             (6, 0.01), (7, 0.1)])
def test_loss_grad_pixel_losses(pn, loss_type, param):
    # every pixel-based RGB loss of Sec. IV-C: loss, gradient and per-sample
    # terms against the oracle
    case = G.make_case("tiny32", loss_type=loss_type, loss_param=param)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    stats, _ = check_full(pn, case, obs, ref, of)
    assert stats["samples"] == int(ref["march"][0][-1])


# (steps per box diagonal, density bias, range of the stop indices the case
# must contain): the compositing kernel takes 64 samples per step and keeps
# the first two steps for its backward sweep, so stops fall in the first step,
# in the second, and later (with longer rays that never stop beside them)
@pytest.mark.parametrize("div,bias,stops", [(96, 3.0, (0, 64)), (384, 2.5, (64, 128)),
                                            (768, 2.5, (128, 10**9))])
@pytest.mark.parametrize("backward", [0, 2])
def test_loss_grad_early_stop_and_occupancy(pn, div, bias, stops, backward):
    R = 16
    case = G.make_case("tiny32", K=3, P=200, march_mode=1, step=math.sqrt(3) / div,
                       max_samples=600, t_stop=1e-2, occ_res=R, density_bias=bias,
                       occ_bits=synth.occupancy_pattern("sphere", R), background=(0.5, 0.2, 0.9))
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    cnt = np.diff(ref["march"][0])
    stopped = ref["stop"] < cnt
    assert np.sum(stopped & (ref["stop"] >= stops[0]) & (ref["stop"] < stops[1])) >= 5
    if stops[0] >= 128:
        assert np.sum(~stopped & (cnt > 128)) >= 5
    check_full(pn, case, obs, ref, of, backward=backward)


def test_loss_grad_empty_grid_is_background_only(pn):
    R = 8
    case = G.make_case("tiny32", K=2, P=50, march_mode=1, step=0.01, max_samples=100,
                       occ_res=R, occ_bits=synth.occupancy_pattern("empty", R),
                       background=(0.3, 0.6, 0.1))
    of = O.OracleField(case.spec)
    obs = np.random.default_rng(0).uniform(0, 1, (32, 32, 3)).astype(np.float32)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr)
    loss, dpose, n = run_loss_grad(pn, case, obs)
    assert n == 0 and np.all(dpose == 0)
    assert np.allclose(loss, ref["loss"], rtol=1e-5)


@pytest.mark.parametrize("K,P", [(1, 1), (1, 257), (5, 63), (7, 1)])
@pytest.mark.parametrize("backward", [0, 2])
def test_loss_grad_ragged_shapes(pn, K, P, backward):
    case = G.make_case("tiny32", K=K, P=P, pix_seed=K * 100 + P)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    check_full(pn, case, obs, ref, of, backward=backward)


@pytest.mark.parametrize("name,kw", [
    ("tiny32", dict(K=5, P=63)),
    ("tiny32", dict(K=3, P=200, march_mode=1, step=math.sqrt(3) / 384, max_samples=600,
                    t_stop=1e-2, occ_res=16, density_bias=2.5, sh_dir_grad=1,
                    occ_bits=synth.occupancy_pattern("sphere", 16))),
    ("ngp800_uniform", dict(K=4)),
])
def test_backward_paths_agree(pn, name, kw):
    """The fused per-ray kernel with and without its per-sample stores, and the
    separate kernels: the same loss and gradient up to summation order (the
    fused kernel sums each ray first), and the fused kernel's stores change
    nothing."""
    case = G.make_case(name, **kw)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    res = {bw: run_loss_grad(pn, case, obs, backward=bw) for bw in (0, 1, 2)}
    assert res[0][2] == res[1][2] == res[2][2]
    for bw, ref_bw, tol in ((2, 1, 1e-6), (1, 0, 1e-4)):
        assert np.allclose(res[bw][0], res[ref_bw][0], rtol=tol, atol=0), bw
        err = np.linalg.norm(res[bw][1] - res[ref_bw][1]) / np.linalg.norm(res[ref_bw][1])
        assert err <= tol, (bw, err)


def test_inspect_needs_a_backward_that_keeps_samples(pn):
    import torch
    case = G.make_case("tiny32", K=2, P=40)
    obs = np.random.default_rng(0).uniform(0, 1, (32, 32, 3)).astype(np.float32)
    f = pn.Field(case.spec, overlap_chunks=1, backward=1)
    f.render_loss_grad(G.to_dev(case.poses), G.to_dev(case.pix), G.to_dev(obs), case.intr)
    torch.cuda.synchronize()
    n = f.last_sample_count()
    assert n > 0
    f.inspect(0, n)  # the sample positions are there
    with pytest.raises(RuntimeError, match="per-sample intermediates"):
        f.inspect(3, n)
    f.close()


@pytest.mark.parametrize("seed", [1, 2, 3, 4])
@pytest.mark.parametrize("lattice", [False, True])
def test_loss_grad_other_seeds(pn, seed, lattice):
    """Other fields, poses and pixel batches (seeds 1-4), uniform and lattice
    marching with early stop: per-sample parity as above, the fused backward
    keeping its per-sample values on odd seeds."""
    kw = dict(K=3, P=300, pix_seed=seed)
    if lattice:
        kw.update(march_mode=1, step=math.sqrt(3) / 192, max_samples=400, t_stop=1e-2, occ_res=16,
                  density_bias=2.0, occ_bits=synth.occupancy_pattern("sphere", 16))
    case = G.make_case("tiny32", seed=seed, **kw)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    stats, _ = check_full(pn, case, obs, ref, of, backward=2 if seed % 2 else 0)
    assert stats["samples"] == int(ref["march"][0][-1]) > 0


def test_loss_grad_uniform_scanned_offsets(pn):
    """Uniform sampling over more rays than the write pass scans itself (96
    scan blocks of 256 rays, against 64): the counts known at ray set-up go
    through the separate scan finish."""
    case = G.make_case("tiny32", K=24, P=1024, pix_seed=7)
    assert case.pix.size > 64 * 256
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    stats, _ = check_full(pn, case, obs, ref, of)
    assert stats["samples"] == int(ref["march"][0][-1])


def test_loss_grad_most_hypotheses(pn):
    """K = 65535 hypotheses of one pixel each (the reduction's grid rows), and
    one more is an argument error, not a failed launch.  The observed image is
    random, so that no one-pixel loss is a near-zero residual, whose relative
    error float32 colour alone would set."""
    import torch
    case = G.make_case("tiny32", K=65535, P=1, pix_seed=11)
    of = O.OracleField(case.spec)
    obs = np.random.default_rng(5).uniform(0.0, 1.0, (32, 32, 3)).astype(np.float32)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    check_full(pn, case, obs, ref, of)
    f = pn.Field(case.spec)
    poses = G.to_dev(np.concatenate([case.poses, case.poses[:1]]))
    pix = G.to_dev(np.concatenate([case.pix, case.pix[:1]]))
    with pytest.raises(pn.PnerfError) as e:
        f.render_loss_grad(poses, pix, G.to_dev(obs), case.intr)
    assert e.value.status == pn.ERR_INVALID_ARG and "65535" in str(e.value)
    torch.cuda.synchronize()
    f.close()


def test_loss_grad_refuses_a_batch_whose_counts_could_overflow(pn):
    """2^19 rays of up to 4096 samples each could count 2^31 samples, past the
    32-bit counts: refused with a capacity error before any device work, and
    the field still works afterwards."""
    import torch
    case = G.make_case("tiny32", K=1, P=4, n_uniform=4096)
    f = pn.Field(case.spec)
    P = 1 << 19
    poses = G.to_dev(case.poses)
    pix = torch.zeros(1, P, dtype=torch.int32, device=G.torch_dev())
    obs = torch.zeros(32, 32, 3, dtype=torch.float32, device=G.torch_dev())
    with pytest.raises(pn.PnerfError) as e:
        f.render_loss_grad(poses, pix, obs, case.intr)
    assert e.value.status == pn.ERR_CAPACITY and "2147483647" in str(e.value)
    loss, dpose = f.render_loss_grad(poses, G.to_dev(case.pix), obs, case.intr)
    torch.cuda.synchronize()
    n = f.last_sample_count()
    assert n % 4096 == 0 and 0 < n <= 4 * 4096   # every ray that meets the box has 4096
    assert np.isfinite(loss.cpu().numpy()).all()
    f.close()


def test_loss_grad_zero_at_ground_truth(pn):
    case = G.make_case("tiny32")
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    case.poses[:] = case.gt[None]
    loss, dpose, _ = run_loss_grad(pn, case, obs)
    assert np.all(loss < 1e-10)
    assert np.abs(dpose).max() < 1e-5


def test_loss_grad_ngp800_uniform_full_batch(pn):
    case = G.make_case("ngp800_uniform")
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    stats, _ = check_full(pn, case, obs, ref, of)
    assert stats["samples"] == int(ref["march"][0][-1])


@pytest.mark.parametrize("backward", [0, 2])
def test_loss_grad_ngp800_occ128_full_batch_sampled_hypotheses(pn, backward):
    # the full 64 x 4096 batch on the GPU; hypotheses are independent, so the
    # oracle recomputes a sample of them; occupancy grid built by the oracle
    w = synth.WORKLOADS["ngp800_occ128"]
    case = G.make_case("ngp800_occ128")
    of0 = O.OracleField(dataclasses.replace(case.spec, occ_res=0, occ_bits=None))
    bits = of0.build_occupancy(128, w.occ_threshold)
    case = dataclasses.replace(case, spec=dataclasses.replace(case.spec, occ_bits=bits))
    of = O.OracleField(case.spec)
    hyps = [0, 31, 63]
    obs = G.oracle_observation(of, case.gt, case.pix[hyps], case.intr)
    ref = oracle_subset(of, case, obs, hyps)
    check_full(pn, case, obs, ref, of, hyps=hyps, backward=backward)


def test_loss_grad_chunked_matches_single_chunk(pn):
    case = G.make_case("tiny32", K=4, P=256)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    l1, g1, _ = run_loss_grad(pn, case, obs)
    l2, g2, _ = run_loss_grad(pn, case, obs, max_ws=1_000_000)  # forces one hypothesis per chunk
    assert np.allclose(l1, l2, rtol=1e-5) and np.allclose(g1, g2, rtol=1e-4, atol=1e-9)


def test_loss_grad_device_sized_matches_host_planned(pn):
    # with room for every ray's sample cap (32 x 1024 samples here) the call
    # sizes its buffer for that worst case and never reads the totals back; a
    # budget below the worst case but above the actual total makes the host
    # read them and plan the same single chunk: same bits, same sample count
    case = G.make_case("tiny32", K=4, P=256)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr)
    l1, g1, n1 = run_loss_grad(pn, case, obs)
    l2, g2, n2 = run_loss_grad(pn, case, obs, max_ws=3_000_000)  # about 21k samples
    assert n1 == n2 == int(ref["march"][0][-1]) < 32 * 1024
    assert np.array_equal(l1, l2) and np.array_equal(g1, g2)


@pytest.mark.parametrize("chunks,backward,mlp_precision", [(2, 0, 0), (4, 0, 0), (7, 0, 0), (3, 1, 0),
                                                           (3, 0, 1)])
def test_loss_grad_overlapped_chunks_match_one_chunk(pn, chunks, backward, mlp_precision):
    # the pipelined loss gradient (encoding of one chunk alongside the networks
    # of the previous, two streams and sample buffers) gives the same bits as
    # one chunk on the caller's stream: per-sample work does not depend on the
    # chunking and every hypothesis is reduced in the same fixed order
    import torch
    case = G.make_case("ngp800_uniform", K=16, P=1024)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    out = []
    for oc in (1, chunks):
        f = pn.Field(case.spec, overlap_chunks=oc, backward=backward, mlp_precision=mlp_precision)
        loss, dpose = f.render_loss_grad(G.to_dev(case.poses), G.to_dev(case.pix), G.to_dev(obs),
                                         case.intr)
        torch.cuda.synchronize()
        n = f.last_sample_count()
        out.append((loss.cpu().numpy(), dpose.cpu().numpy(), n))
        f.close()
    assert out[0][2] == out[1][2] > 65536
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])


def test_loss_grad_deterministic(pn):
    case = G.make_case("tiny32")
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    a = run_loss_grad(pn, case, obs)
    b = run_loss_grad(pn, case, obs)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


# ------------------------------------------------------------ pose kernels
def test_step_momentum_matches_oracle(pn):
    import torch
    rng = np.random.default_rng(0)
    K = 37
    w = synth.WORKLOADS["tiny32"]
    poses = synth.perturb_poses(synth.ground_truth_pose(w, 0), K, 40, 0.3, 0)
    mom = rng.normal(size=(K, 6)).astype(np.float32) * 0.1
    g = rng.normal(size=(K, 6)).astype(np.float32)
    p_ref, m_ref = poses, mom
    p_d, m_d, g_d = G.to_dev(poses), G.to_dev(mom), G.to_dev(g)
    for _ in range(5):
        p_ref, m_ref = O.step_momentum(p_ref, m_ref, g, 1e-2, 0.9)
        pn.step_momentum(p_d, m_d, g_d, 1e-2, 0.9)
    torch.cuda.synchronize()
    assert np.allclose(p_d.cpu().numpy(), p_ref, atol=1e-6, rtol=0)
    assert np.allclose(m_d.cpu().numpy(), m_ref, atol=1e-6, rtol=1e-6)


@pytest.mark.parametrize("K,keep", [(256, 0.25), (1024, 0.10), (37, 0.3), (1, 0.5)])
def test_resample_matches_oracle(pn, K, keep):
    import torch
    w = synth.WORKLOADS["tiny32"]
    poses = synth.perturb_poses(synth.ground_truth_pose(w, 0), K, 40, 0.3, 1)
    rng = np.random.default_rng(K)
    mom = rng.normal(size=(K, 6)).astype(np.float32)
    loss = rng.uniform(0, 1, K).astype(np.float32)
    if K > 10:
        loss[[2, 7]] = np.nan
        loss[5] = loss[4]
    sr, st = math.radians(5), 0.03
    p_ref, m_ref, _ = O.resample(poses, mom, loss, keep, sr, st, 1234, 3)
    p_d, m_d = G.to_dev(poses), G.to_dev(mom)
    pn.resample_hypotheses(p_d, m_d, G.to_dev(loss), keep, sr, st, 1234, 3)
    torch.cuda.synchronize()
    pg, mg = p_d.cpu().numpy(), m_d.cpu().numpy()
    assert np.array_equal(mg, m_ref)                 # kept momenta exact, redrawn ones zero
    assert np.allclose(pg, p_ref, atol=1e-6, rtol=0)


def test_device_occupancy_build_matches_oracle(pn):
    R = 32
    case = G.make_case("tiny32")
    of = O.OracleField(case.spec)
    # threshold at the median centre density so that about half the cells are set
    sig = []
    for lin in range(0, R ** 3, 97):
        x, y, z = lin % R, (lin // R) % R, lin // (R * R)
        c = (np.array([x, y, z]) + 0.5) / R
        feat, _ = of.encode(c.astype(np.float32), c)
        sig.append(math.exp(of.density_mlp(feat)[0] - 1.0))
    thr = float(np.median(sig))
    ref = synth.unpack_bits(of.build_occupancy(R, thr), R)
    spec = dataclasses.replace(case.spec, occ_res=R, occ_bits=None, occ_threshold=thr,
                               march_mode=1, step=0.01, max_samples=10)
    f = pn.Field(spec)
    got = synth.unpack_bits(f.occupancy(), R)
    f.close()
    diff = np.argwhere(got != ref)
    assert 0.2 < ref.mean() < 0.8
    for z, y, x in diff:   # disagreements only where sigma is within rounding of thr
        c = (np.array([x, y, z]) + 0.5) / R
        feat, _ = of.encode(c.astype(np.float32), c)
        s = math.exp(of.density_mlp(feat)[0] - 1.0)
        assert abs(s - thr) <= 1e-5 * thr


# ----------------------------------------------------- fp16 storage, large scene
def f16_case(name, **kw):
    """A workload's case with the hash table and MLP weights stored in fp16."""
    case = G.make_case(name, **kw)
    sp = case.spec
    h = lambda a: np.asarray(a).astype(np.float16)
    spec = dataclasses.replace(sp, param_dtype="f16", table=h(sp.table),
                               w_density1=h(sp.w_density1), w_density2=h(sp.w_density2),
                               w_color1=h(sp.w_color1), w_color2=h(sp.w_color2),
                               w_color3=h(sp.w_color3))
    return dataclasses.replace(case, spec=spec)


@pytest.mark.parametrize("overrides", [dict(), dict(sh_dir_grad=1)])
def test_loss_grad_tiny_fp16_storage(pn, overrides):
    case = f16_case("tiny32", **overrides)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    stats, ex = check_full(pn, case, obs, ref, of)
    assert stats["samples"] == int(ref["march"][0][-1])


_OCC_CACHE = {}


def with_oracle_occupancy(case, R, thr):
    """The case with the occupancy grid the oracle builds from the field's
    density (cached per field: the 256^3 grid takes seconds)."""
    key = (case.w.name, case.spec.log2_table, case.spec.param_dtype, R, thr,
           float(np.asarray(case.spec.table).ravel()[:8].astype(np.float64).sum()))
    if key not in _OCC_CACHE:
        of0 = O.OracleField(dataclasses.replace(case.spec, occ_res=0, occ_bits=None))
        _OCC_CACHE[key] = of0.build_occupancy(R, thr)
    return dataclasses.replace(case, spec=dataclasses.replace(case.spec, occ_bits=_OCC_CACHE[key]))


def check_sampled_hypotheses(pn, case, hyps):
    """The whole batch on the GPU (chunked over hypotheses as the library
    decides), the oracle on a few hypotheses; per-hypothesis loss and gradient."""
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix[hyps], case.intr)
    ref = oracle_subset(of, case, obs, hyps)
    loss, dpose, n = run_loss_grad(pn, case, obs)
    G.assert_loss_grad_close(loss, dpose, ref, hyps=hyps)
    return n


def test_loss_grad_cam640_f16_full_batch_sampled_hypotheses(pn):
    # 256 x 2048 rays, 640x480 camera with principal point (325.3, 242.0),
    # table and weights in fp16, 128^3 occupancy, lattice marching with early stop
    w = synth.WORKLOADS["cam640_f16_occ128"]
    case = with_oracle_occupancy(G.make_case("cam640_f16_occ128"), w.occ_res, w.occ_threshold)
    assert case.spec.table.dtype == np.float16
    n = check_sampled_hypotheses(pn, case, [0, 128, 255])
    assert n > 10_000_000


def test_loss_grad_large_scene_full_batch_sampled_hypotheses(pn):
    # 1024 x 512 rays in the [-2,2]^3 box, T = 2^21, 256^3 occupancy, up to 2048
    # samples per ray (processed in several hypothesis chunks)
    w = synth.WORKLOADS["large4m_occ256"]
    case = with_oracle_occupancy(G.make_case("large4m_occ256"), w.occ_res, w.occ_threshold)
    n = check_sampled_hypotheses(pn, case, [0, 511, 1023])
    assert n > 100_000_000


# -------------------------------------------------------- structured density
def test_device_occupancy_build_bump_field_matches_oracle(pn):
    w = synth.WORKLOADS["ngp800_bump_occ128"]
    case = G.make_case("ngp800_bump_occ128", K=2, P=64)
    of0 = O.OracleField(dataclasses.replace(case.spec, occ_res=0, occ_bits=None))
    R = w.occ_res
    ref = synth.unpack_bits(of0.build_occupancy(R, w.occ_threshold), R)
    f = pn.Field(dataclasses.replace(case.spec, occ_bits=None))
    got = synth.unpack_bits(f.occupancy(), R)
    f.close()
    assert 0.05 < ref.mean() < 0.5
    diff = np.argwhere(got != ref)
    assert len(diff) <= 64
    for z, y, x in diff:   # disagreements only where sigma is within rounding of thr
        c = (np.array([x, y, z]) + 0.5) / R
        feat, _ = of0.encode(c.astype(np.float32), c)
        s = math.exp(of0.density_mlp(feat)[0] + case.spec.density_bias)
        assert abs(s - w.occ_threshold) <= 1e-5 * w.occ_threshold


@pytest.mark.parametrize("name,K,P", [("tiny_bump", None, None), ("ngp800_bump_occ128", None, None)])
def test_march_bump_bitexact(pn, name, K, P):
    w = synth.WORKLOADS[name]
    case = with_oracle_occupancy(G.make_case(name, K=K, P=P), w.occ_res, w.occ_threshold)
    total = check_march(pn, case)
    assert 0 < total < case.pix.size * 64     # most candidates skipped


def test_loss_grad_tiny_bump(pn):
    w = synth.WORKLOADS["tiny_bump"]
    case = with_oracle_occupancy(G.make_case("tiny_bump"), w.occ_res, w.occ_threshold)
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    stats, ex = check_full(pn, case, obs, ref, of)
    cnt = np.diff(ref["march"][0])
    assert np.sum(ref["stop"] < cnt) >= 5     # early termination took effect


def test_loss_grad_ngp800_bump_full_batch_sampled_hypotheses(pn):
    w = synth.WORKLOADS["ngp800_bump_occ128"]
    case = with_oracle_occupancy(G.make_case("ngp800_bump_occ128"), w.occ_res, w.occ_threshold)
    n = check_sampled_hypotheses(pn, case, [0, 31, 63])
    assert n > 0


# ------------------------------------- full-size workloads: colour, per sample
def workload_case(name, seed=0):
    """The workload's full batch (fp16 storage where the workload says so) with
    the oracle's density-built occupancy grid."""
    w = synth.WORKLOADS[name]
    case = f16_case(name, seed=seed) if w.param_dtype == "f16" else G.make_case(name, seed=seed)
    return with_oracle_occupancy(case, w.occ_res, w.occ_threshold)


@pytest.mark.parametrize("name,hyps", [("ngp800_occ128", [0, 37, 63]),
                                       ("cam640_f16_occ128", [0, 129, 255]),
                                       ("large4m_occ256", [0, 600, 1023])])
def test_render_colour_full_batch_sampled_hypotheses(pn, name, hyps):
    """pnerf_render over the whole batch (chunked as the library decides); the
    oracle renders the sampled hypotheses: colour within 2e-3 absolute
    (Sec. III, volume rendering), on lattice marching with occupancy and early
    stop, the fp16-stored field and the 2^21-entry [-2,2]^3 field."""
    import torch
    case = workload_case(name)
    f = pn.Field(case.spec)
    rgb = f.render(G.to_dev(case.poses), G.to_dev(case.pix), case.intr)
    torch.cuda.synchronize()
    got = rgb.cpu().numpy()
    f.close()
    of = O.OracleField(case.spec)
    ref = of.render(case.poses[hyps], case.pix[hyps], case.intr)
    err = np.abs(got[hyps] - ref).max()
    sys.stderr.write(f"[parity] {name} colour: max abs error {err:.3g}\n")
    assert err <= G.COLOR_ATOL
    assert ref.max() > 0.05


@pytest.mark.parametrize("name,hyps,backward,seed", [("cam640_f16_occ128", [3, 200], 0, 0),
                                                     ("large4m_occ256", [5, 700], 0, 0),
                                                     ("large4m_occ256", [5, 700], 2, 0),
                                                     ("large4m_occ256", [11, 512], 0, 1)])
def test_loss_grad_sampled_hypotheses_per_sample(pn, name, hyps, backward, seed):
    """The sampled hypotheses of a full-size workload as a batch of their own
    (one chunk, so every sample can be inspected): per-hypothesis sample counts
    exactly, per-sample torque and force shares and the stage values d loss /
    d h0 and d loss / d z, loss and pose gradient (Eq. 2, Eq. 3)."""
    full = workload_case(name, seed)
    case = dataclasses.replace(full, poses=full.poses[hyps], pix=full.pix[hyps])
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    stats, _ = check_full(pn, case, obs, ref, of, backward=backward)
    assert stats["samples"] == int(ref["march"][0][-1]) > 100_000


def test_march_large_scene_density_grid_bitexact(pn):
    """200 hypotheses of the [-2,2]^3 workload on its density-built 256^3 grid
    (the random field sets every cell): ray offsets, sample distances and
    lattice indices bit-exact."""
    w = synth.WORKLOADS["large4m_occ256"]
    case = with_oracle_occupancy(G.make_case("large4m_occ256"), w.occ_res, w.occ_threshold)
    case = dataclasses.replace(case, poses=case.poses[:200], pix=case.pix[:200])
    assert check_march(pn, case) > 50_000_000
