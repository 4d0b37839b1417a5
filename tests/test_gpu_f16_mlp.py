"""The fp16 network arithmetic (mlp_precision = 1: fp16 MFMA, each weight as
two fp16 parts, each activation rounded to fp16, fp32 accumulation) against
the oracle on the same seeded inputs: colour within 2e-3 absolute, loss within
1e-3 relative, and the pose gradient within 5e-2 relative L2 (the bound for
fp16 MFMA in the networks) under the threshold decisions the GPU took.  The
activations' fp16 rounding (2^-12) decides ReLUs whose pre-activation lies
within about 1e-3 of the sum of its terms' magnitudes either way, so the
parity checker runs with margins sized for it: such samples are set aside and
matched against the oracle's shading with those units flipped, every other
sample element by element."""
import dataclasses
import math
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2210_10108_amd import synth
from tests import gpu_common as G

pytestmark = pytest.mark.gpu

GRAD_RTOL_F16 = 5e-2
# the parity checker's margins and tolerances for fp16 activations (the
# split-bf16 path's are 1e-4, 2e-3, 1e-3 and 0.10)
F16_CHECKER = dict(MARGIN_RELU=5e-4, SAMPLE_TOL=5e-3, STAGE_TOL=2e-3, MAX_SET_ASIDE=0.5)


@pytest.fixture(autouse=True)
def f16_checker(monkeypatch):
    for k, v in F16_CHECKER.items():
        monkeypatch.setattr(G, k, v)


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


def gpu_loss_grad(pn, case, obs, mlp_precision=1, per_sample=True, backward=0):
    import torch
    f = pn.Field(case.spec, overlap_chunks=1, backward=backward, mlp_precision=mlp_precision)
    poses, pix = G.to_dev(case.poses), G.to_dev(case.pix)
    loss, dpose = f.render_loss_grad(poses, pix, G.to_dev(obs), case.intr)
    torch.cuda.synchronize()
    n = f.last_sample_count()
    ex = {}
    if per_sample:
        ex["out6"] = f.inspect(3, n).cpu().numpy()
        ex["gh0"] = f.inspect(1, n).cpu().numpy()
        ex["gz"] = f.inspect(2, n).cpu().numpy().reshape(-1, 3)
    f.close()
    return loss.cpu().numpy(), dpose.cpu().numpy(), n, ex


def per_sample_errors(ref, ex, P):
    """Per sample and per quantity (torque share, force share, dL/dh0, dL/dz):
    the largest component error relative to the hypothesis's largest value."""
    so = ref["samples"]
    off = ref["march"][0]
    K = (len(off) - 1) // P
    pairs = {"torque": (ex["out6"][:, 0:3], so[:, 13:16]), "force": (ex["out6"][:, 3:6], so[:, 8:11]),
             "gh0": (ex["gh0"][:, None], so[:, 4:5]), "gz": (ex["gz"], so[:, 5:8])}
    out = {}
    for name, (g, o) in pairs.items():
        err = np.zeros(len(so))
        for k in range(K):
            a, b = int(off[k * P]), int(off[(k + 1) * P])
            if b == a:
                continue
            scale = np.abs(o[a:b]).max()
            if scale > 0:
                err[a:b] = np.abs(g[a:b] - o[a:b]).max(axis=1) / scale
        out[name] = err
    return out


def check_f16(label, case, of, obs, ref, loss, dpose, n, ex):
    K, P = case.pix.shape
    assert n == int(ref["march"][0][-1])
    msg = f"[f16] {label}:"
    for name, e in per_sample_errors(ref, ex, P).items():
        msg += f" {name} median {np.median(e):.1e} q99 {np.quantile(e, 0.99):.1e} max {e.max():.1e};"
    sys.stderr.write(msg + "\n")
    alt = G.Alt(of, case.poses, case.pix, obs, case.intr)
    per_sample = np.concatenate([ex["out6"], ex["gh0"][:, None], ex["gz"]], axis=1)
    return G.assert_loss_grad_close(loss, dpose, ref, gpu_samples=per_sample, alt=alt,
                                    grad_rtol=GRAD_RTOL_F16, label="f16 " + label)


def oracle_case(case):
    of = O.OracleField(case.spec)
    obs = G.oracle_observation(of, case.gt, case.pix, case.intr)
    ref = of.render_loss_grad(case.poses, case.pix, obs, case.intr, per_sample=True)
    return of, obs, ref


@pytest.mark.parametrize("overrides", [dict(), dict(sh_dir_grad=1), dict(background=(1.0, 1.0, 1.0))])
def test_f16_loss_grad_tiny(pn, overrides):
    case = G.make_case("tiny32", **overrides)
    of, obs, ref = oracle_case(case)
    check_f16("tiny32 " + str(overrides), case, of, obs, ref, *gpu_loss_grad(pn, case, obs))


@pytest.mark.parametrize("n_levels,sh_dir,backward", [(8, 0, 0), (12, 1, 0), (16, 0, 0), (12, 0, 2)])
def test_f16_loss_grad_level_counts(pn, monkeypatch, n_levels, sh_dir, backward):
    name = f"tiny32_l{n_levels}"
    w = dataclasses.replace(synth.WORKLOADS["tiny32"], name=name, n_levels=n_levels, log2_table=14)
    monkeypatch.setitem(synth.WORKLOADS, name, w)
    case = G.make_case(name, K=8, P=256, dense_coarse_levels=1, sh_dir_grad=sh_dir)
    of, obs, ref = oracle_case(case)
    check_f16(name, case, of, obs, ref, *gpu_loss_grad(pn, case, obs, backward=backward))


@pytest.mark.parametrize("sh_dir,backward", [(0, 0), (1, 0), (1, 2)])
def test_f16_loss_grad_early_stop_and_occupancy(pn, sh_dir, backward):
    R = 16
    case = G.make_case("tiny32", K=3, P=200, march_mode=1, step=math.sqrt(3) / 384,
                       max_samples=600, t_stop=1e-2, occ_res=R, density_bias=2.5,
                       occ_bits=synth.occupancy_pattern("sphere", R), background=(0.5, 0.2, 0.9),
                       sh_dir_grad=sh_dir)
    of, obs, ref = oracle_case(case)
    assert np.sum(ref["stop"] < np.diff(ref["march"][0])) >= 5
    check_f16(f"early stop sh_dir={sh_dir} backward={backward}", case, of, obs, ref,
              *gpu_loss_grad(pn, case, obs, backward=backward))


def test_f16_loss_grad_tiny_gradients_are_scaled(pn):
    """Relative L2 with epsilon 1e6: every gradient is about 1e-6 of the usual
    size, far below fp16's normal range before the per-sample scaling."""
    case = G.make_case("tiny32", loss_type=4, loss_param=1e6)
    of, obs, ref = oracle_case(case)
    assert np.abs(ref["samples"][:, 8:11]).max() < 1e-6
    check_f16("scaled", case, of, obs, ref, *gpu_loss_grad(pn, case, obs))


def test_f16_fused_backward_matches_separate(pn):
    case = G.make_case("tiny32", K=5, P=63)
    of, obs, ref = oracle_case(case)
    res = {bw: gpu_loss_grad(pn, case, obs, backward=bw, per_sample=bw != 1) for bw in (0, 1, 2)}
    check_f16("fused keep", case, of, obs, ref, *res[2])
    for bw in (1, 2):
        err = G.rel_l2(res[bw][1], res[0][1])
        assert err <= 1e-4, (bw, err)


def test_f16_differs_from_split_bf16_within_tolerance(pn):
    # the fp16 kernels ran (their results are not the split-bf16 path's bits)
    # and agree with it within the fp16 tolerance
    case = G.make_case("ngp800_uniform", K=4)
    obs = G.oracle_observation(O.OracleField(case.spec), case.gt, case.pix, case.intr)
    l0, g0, n0, _ = gpu_loss_grad(pn, case, obs, mlp_precision=0, per_sample=False)
    l1, g1, n1, _ = gpu_loss_grad(pn, case, obs, mlp_precision=1, per_sample=False)
    assert n0 == n1
    assert not np.array_equal(g0, g1)
    assert max(G.rel_l2(g1[k], g0[k]) for k in range(4)) <= GRAD_RTOL_F16
    assert np.abs(l1 - l0).max() <= G.LOSS_RTOL * np.abs(l0).max()


@pytest.mark.parametrize("name,hyps", [("ngp800_occ128", [0, 63]), ("cam640_f16_occ128", [3, 200]),
                                       ("large4m_occ256", [5, 700])])
def test_f16_loss_grad_sampled_hypotheses(pn, name, hyps):
    from tests.test_gpu_parity import workload_case
    full = workload_case(name)
    case = dataclasses.replace(full, poses=full.poses[hyps], pix=full.pix[hyps])
    of, obs, ref = oracle_case(case)
    check_f16(name, case, of, obs, ref, *gpu_loss_grad(pn, case, obs))


@pytest.mark.parametrize("name,K,P", [("tiny32", 1, 1024), ("ngp800_uniform", 4, 1000)])
def test_f16_render_colour(pn, name, K, P):
    import torch
    case = G.make_case(name, K=K, P=P)
    if name == "tiny32":
        case = dataclasses.replace(case, poses=case.gt[None],
                                   pix=np.arange(32 * 32, dtype=np.int32)[None])
    ref = O.OracleField(case.spec).render(case.poses, case.pix, case.intr)
    f = pn.Field(case.spec, mlp_precision=1)
    rgb = f.render(G.to_dev(case.poses), G.to_dev(case.pix), case.intr)
    torch.cuda.synchronize()
    f.close()
    err = np.abs(rgb.cpu().numpy() - ref).max()
    sys.stderr.write(f"[f16] {name} colour: max abs error {err:.3g}\n")
    assert err <= G.COLOR_ATOL


@pytest.mark.parametrize("name,hyps", [("cam640_f16_occ128", [0, 255]), ("large4m_occ256", [0, 1023])])
def test_f16_render_colour_full_batch_sampled_hypotheses(pn, name, hyps):
    """pnerf_render with the fp16 networks over a whole workload batch (chunked as
    the library decides): colour within 2e-3 on the sampled hypotheses."""
    import torch
    from tests.test_gpu_parity import workload_case
    case = workload_case(name)
    f = pn.Field(case.spec, mlp_precision=1)
    rgb = f.render(G.to_dev(case.poses), G.to_dev(case.pix), case.intr)
    torch.cuda.synchronize()
    got = rgb.cpu().numpy()
    f.close()
    ref = O.OracleField(case.spec).render(case.poses[hyps], case.pix[hyps], case.intr)
    err = np.abs(got[hyps] - ref).max()
    sys.stderr.write(f"[f16] {name} colour: max abs error {err:.3g}\n")
    assert err <= G.COLOR_ATOL
