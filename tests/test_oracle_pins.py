"""Pins of the CPU oracle against values fixed by mathematics or by libraries,
not by the oracle itself: closed forms, invariants, textbook special cases,
library routines (numpy, scipy) and brute force on tiny inputs.  CPU only."""
import dataclasses
import math

import numpy as np
import pytest
from scipy.spatial.transform import Rotation
from scipy import special

from paper_2210_10108_amd import synth


def tiny_spec(**kw):
    w = synth.WORKLOADS["tiny32"]
    return w, synth.field_spec(w, synth.make_field(w, 0), **kw)


# ------------------------------------------------------------------ hashing
# Vertex indices evaluated by hand from the spatial hash of the multiresolution
# encoding (tests/golden/hash_vertices.txt, which states the definition).
def _hash_pins():
    import os
    pins = {}
    path = os.path.join(os.path.dirname(__file__), "golden", "hash_vertices.txt")
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            log2T, i, j, k, h = (int(v) for v in line.split())
            pins.setdefault(log2T, {})[(i, j, k)] = h
    return pins


HASH_PINS = _hash_pins()


@pytest.mark.parametrize("log2T", [12, 19])
def test_hash_pins(oracle_lib, log2T):
    w, spec = tiny_spec()
    # all levels hashed: dense indexing switched off
    spec = dataclasses.replace(spec, log2_table=log2T, dense_coarse_levels=0,
                               table=np.zeros((4, 1 << log2T, 2), np.float32))
    of = oracle_lib.OracleField(spec)
    for (i, j, k), want in HASH_PINS[log2T].items():
        assert of.grid_index(0, i, j, k) == want


def test_dense_index_rule(oracle_lib):
    # N=16 -> 17^3 = 4913 vertices: hashed in a 2^12 table, dense in 2^19
    w, spec = tiny_spec()
    of12 = oracle_lib.OracleField(spec)
    assert of12.grid_index(0, 1, 2, 3) == (1 ^ (2 * 2654435761) ^ (3 * 805459861)) % 4096
    spec19 = dataclasses.replace(spec, log2_table=19, table=np.zeros((4, 1 << 19, 2), np.float32))
    of19 = oracle_lib.OracleField(spec19)
    assert of19.grid_index(0, 1, 2, 3) == 1 + 2 * 17 + 3 * 17 * 17
    # level 3 (N=64): 65^3 = 274625 <= 2^19 -> still dense
    assert of19.grid_index(3, 1, 1, 1) == 1 + 65 + 65 * 65
    # N=100: 101^3 > 2^19 -> hashed
    spec100 = dataclasses.replace(spec19, level_res=np.array([16, 25, 40, 100], np.int32))
    assert oracle_lib.OracleField(spec100).grid_index(3, 1, 1, 1) == 339493


def test_level_resolutions():
    # geometric ladder N_min * b^l, exact powers must not floor one low
    assert list(synth.level_resolutions(4, 16, 64)) == [16, 25, 40, 64]
    assert list(synth.level_resolutions(16, 16, 2048)) == [
        16, 22, 30, 42, 58, 80, 111, 153, 212, 294, 406, 561, 776, 1072, 1482, 2048]
    assert list(synth.level_resolutions(16, 16, 8192)) == [
        16, 24, 36, 55, 84, 128, 194, 294, 445, 675, 1024, 1552, 2352, 3565, 5404, 8192]


# ------------------------------------------------------------- trilinear
def dense_linear_spec(a, b):
    """All four levels dense; entry of vertex v = a . v + b (per feature)."""
    res = np.array([3, 5, 8, 12], np.int32)
    T = 1 << 12
    table = np.zeros((4, T, 2), np.float32)
    for l, N in enumerate(res):
        n1 = N + 1
        ii, jj, kk = np.meshgrid(np.arange(n1), np.arange(n1), np.arange(n1), indexing="ij")
        idx = (ii + jj * n1 + kk * n1 * n1).ravel()
        v = np.stack([ii.ravel(), jj.ravel(), kk.ravel()], 1).astype(np.float64)
        for q in range(2):
            table[l, idx, q] = v @ a[q] + b[q]
    w, spec = tiny_spec()
    return dataclasses.replace(spec, level_res=res, table=table)


def test_trilinear_reproduces_linear_functions(oracle_lib):
    a = np.array([[0.25, -0.5, 0.125], [-0.75, 0.0625, 0.5]])
    b = np.array([0.5, -0.25])
    spec = dense_linear_spec(a, b)
    of = oracle_lib.OracleField(spec)
    rng = np.random.default_rng(5)
    for _ in range(50):
        x = rng.uniform(0, 1, 3).astype(np.float32)
        feat, jac = of.encode(x)
        for l, N in enumerate(spec.level_res):
            for q in range(2):
                want = a[q] @ (x.astype(np.float64) * N) + b[q]
                assert feat[2 * l + q] == pytest.approx(want, abs=1e-12)
                assert np.allclose(jac[:, 2 * l + q], a[q] * N, atol=1e-12)


def test_trilinear_partition_of_unity_and_vertices(oracle_lib):
    w, spec = tiny_spec()
    ones = np.ones_like(spec.table)
    of1 = oracle_lib.OracleField(dataclasses.replace(spec, table=ones))
    rng = np.random.default_rng(1)
    for _ in range(20):
        x = rng.uniform(0, 1, 3).astype(np.float32)
        feat, jac = of1.encode(x)
        assert np.allclose(feat, 1.0, atol=1e-14) and np.allclose(jac, 0.0, atol=1e-12)
    # at a vertex of a hashed level the feature equals that vertex's entry
    of = oracle_lib.OracleField(spec)
    N = int(spec.level_res[0])
    for (i, j, k) in [(3, 5, 7), (1, 1, 1), (0, 1, 0)]:
        x = np.array([i / N, j / N, k / N], np.float32)
        feat, _ = of.encode(x, x.astype(np.float64))
        h = ((i * 1) ^ ((j * 2654435761) & 0xFFFFFFFF) ^ ((k * 805459861) & 0xFFFFFFFF)) % 4096
        assert np.allclose(feat[0:2], spec.table[0, h], atol=1e-7)


def test_trilinear_continuity_and_jacobian_fd(oracle_lib):
    w, spec = tiny_spec()
    of = oracle_lib.OracleField(spec)
    N = int(spec.level_res[2])
    # continuity across a cell face of level 2 (x = 10/N), both sides use their own cell
    eps = 1e-6
    x_lo = np.array([10 / N - eps, 0.31, 0.62])
    x_hi = np.array([10 / N + eps, 0.31, 0.62])
    f_lo, _ = of.encode(x_lo.astype(np.float32), x_lo)
    f_hi, _ = of.encode(x_hi.astype(np.float32), x_hi)
    assert np.max(np.abs(f_lo - f_hi)) < 1e-3
    # Jacobian against central differences inside one cell (cells frozen via x32)
    rng = np.random.default_rng(2)
    for _ in range(10):
        x = rng.uniform(0.05, 0.95, 3)
        x32 = x.astype(np.float32)
        feat, jac = of.encode(x32, x)
        h = 1e-7
        for a in range(3):
            xp, xm = x.copy(), x.copy()
            xp[a] += h
            xm[a] -= h
            fp, _ = of.encode(x32, xp)
            fm, _ = of.encode(x32, xm)
            assert np.allclose((fp - fm) / (2 * h), jac[a], rtol=1e-6, atol=1e-6)


# ------------------------------------------------------ spherical harmonics
def real_sh_scipy(l, m, d):
    """Real orthonormal SH without the Condon-Shortley phase from scipy's complex Y_l^m."""
    theta = math.acos(max(-1.0, min(1.0, d[2])))
    phi = math.atan2(d[1], d[0])
    if m == 0:
        return special.sph_harm_y(l, 0, theta, phi).real
    y = special.sph_harm_y(l, abs(m), theta, phi)
    cs = (-1) ** m  # scipy includes (-1)^m; remove it
    return math.sqrt(2) * cs * (y.real if m > 0 else y.imag)


def test_sh16_matches_scipy(oracle_lib):
    rng = np.random.default_rng(3)
    for _ in range(20):
        d = rng.normal(size=3)
        d /= np.linalg.norm(d)
        v, _ = oracle_lib.sh16(d)
        want = [real_sh_scipy(l, m, d) for l in range(4) for m in range(-l, l + 1)]
        assert np.allclose(v, want, atol=1e-12)
    v, _ = oracle_lib.sh16(np.array([0, 0, 1.0]))
    assert v[0] == pytest.approx(1 / (2 * math.sqrt(math.pi)), abs=1e-15)


def test_sh16_orthonormal_by_exact_quadrature(oracle_lib):
    # Gauss-Legendre in cos(theta) x uniform phi integrates degree <= 6 exactly
    xs, ws = np.polynomial.legendre.leggauss(8)
    nphi = 16
    G = np.zeros((16, 16))
    for z, wz in zip(xs, ws):
        for k in range(nphi):
            phi = 2 * math.pi * k / nphi
            s = math.sqrt(1 - z * z)
            v, _ = oracle_lib.sh16(np.array([s * math.cos(phi), s * math.sin(phi), z]))
            G += np.outer(v, v) * wz * (2 * math.pi / nphi)
    assert np.allclose(G, np.eye(16), atol=1e-12)


def test_sh16_gradient_fd(oracle_lib):
    d = np.array([0.3, -0.5, 0.81])
    _, g = oracle_lib.sh16(d)
    h = 1e-6
    for a in range(3):
        dp, dm = d.copy(), d.copy()
        dp[a] += h
        dm[a] -= h
        fd = (oracle_lib.sh16(dp)[0] - oracle_lib.sh16(dm)[0]) / (2 * h)
        assert np.allclose(fd, g[:, a], atol=1e-8)


# ------------------------------------------------------------------ MLPs
def test_mlps_equal_numpy_chain(oracle_lib):
    w, spec = tiny_spec()
    of = oracle_lib.OracleField(spec)
    rng = np.random.default_rng(4)
    relu = lambda z: np.maximum(z, 0)
    W = lambda a: np.asarray(a, np.float64)
    for _ in range(5):
        f = rng.normal(size=8)
        h = of.density_mlp(f)
        assert np.allclose(h, relu(f @ W(spec.w_density1)) @ W(spec.w_density2), atol=1e-12)
        xc = rng.normal(size=32)
        rgb = of.color_mlp(xc)
        z = relu(relu(xc @ W(spec.w_color1)) @ W(spec.w_color2)) @ W(spec.w_color3)
        assert np.allclose(rgb, 1 / (1 + np.exp(-z)), atol=1e-12)


# -------------------------------------------------------------- composite
def test_composite_constant_closed_form(oracle_lib):
    sigma, delta, n = 1.7, 0.05, 40
    c = np.array([0.2, 0.6, 0.9])
    bg = np.array([1.0, 0.5, 0.25])
    C, trans, weight, used = oracle_lib.composite(np.full(n, sigma), np.tile(c, (n, 1)), delta, bg)
    e = math.exp(-sigma * n * delta)
    assert np.allclose(C, c * (1 - e) + bg * e, atol=1e-14)
    assert np.all(np.diff(trans) <= 0) and weight.sum() == pytest.approx(1 - trans[-1], abs=1e-14)
    # derivative w.r.t. a common sigma = sum of the per-sample derivatives
    gs, gr = oracle_lib.composite_grad(np.full(n, sigma), np.tile(c, (n, 1)), delta,
                                       np.array([1.0, 0, 0]), bg)
    want = (c[0] - bg[0]) * n * delta * e
    assert gs.sum() == pytest.approx(want, rel=1e-12)
    assert np.allclose(gr[:, 0], weight, atol=1e-15) and np.allclose(gr[:, 1:], 0)
    # zero density: pure background
    C0, _, _, _ = oracle_lib.composite(np.zeros(n), np.tile(c, (n, 1)), delta, bg)
    assert np.allclose(C0, bg)


def test_composite_early_stop(oracle_lib):
    sigma, delta, n = 50.0, 0.05, 100
    C, trans, weight, used = oracle_lib.composite(np.full(n, sigma), np.full((n, 3), 0.5), delta,
                                                  t_stop=1e-4)
    # T_{i+1} = exp(-sigma delta (i+1)) < 1e-4 first at i+1 = ceil(ln(1e4)/(sigma delta))
    assert used == math.ceil(math.log(1e4) / (sigma * delta))
    assert trans[-1] < 1e-4 <= trans[-2]


def test_composite_grad_fd(oracle_lib):
    rng = np.random.default_rng(6)
    n = 12
    sig = rng.uniform(0.1, 3, n)
    rgb = rng.uniform(0, 1, (n, 3))
    bg = np.array([0.3, 0.1, 0.7])
    gC = np.array([0.4, -1.0, 0.25])
    gs, gr = oracle_lib.composite_grad(sig, rgb, 0.07, gC, bg)
    h = 1e-6
    for i in range(n):
        sp, sm = sig.copy(), sig.copy()
        sp[i] += h
        sm[i] -= h
        fd = (oracle_lib.composite(sp, rgb, 0.07, bg)[0] - oracle_lib.composite(sm, rgb, 0.07, bg)[0])
        assert gs[i] == pytest.approx(gC @ fd / (2 * h), rel=1e-7, abs=1e-10)


# --------------------------------------------------------------------- rays
def test_ray_principal_point_and_directions(oracle_lib):
    w, _ = tiny_spec()
    pose = synth.ground_truth_pose(w, 3)
    intr = dict(width=32, height=32, fx=40.0, fy=40.0, cx=16.5, cy=16.5)
    o, d = oracle_lib.ray_f32(pose, intr, 16 * 32 + 16)   # pixel centre (16.5, 16.5)
    assert np.allclose(d, pose[:, 2], atol=1e-7) and np.allclose(o, pose[:, 3])
    # brute force for every pixel of the image
    R = pose[:, :3].astype(np.float64)
    for pix in range(0, 32 * 32, 37):
        u, v = pix % 32, pix // 32
        dc = np.array([(u + 0.5 - 16.5) / 40.0, (v + 0.5 - 16.5) / 40.0, 1.0])
        want = R @ dc
        want /= np.linalg.norm(want)
        assert np.allclose(oracle_lib.ray_f32(pose, intr, pix)[1], want, atol=1e-6)


def _inside(p, lo, hi, tol):
    return np.all(p >= np.array(lo) - tol) and np.all(p <= np.array(hi) + tol)


def test_march_uniform_brute_force(oracle_lib):
    w, spec = tiny_spec()
    of = oracle_lib.OracleField(spec)
    intr = synth.intrinsics(w)
    pose = synth.ground_truth_pose(w, 0)
    pix = np.arange(32 * 32, dtype=np.int32)[None]
    off, t, j, delta = of.march(pose[None], pix, intr)
    counts = np.diff(off)
    assert set(np.unique(counts)) <= {0, 32}
    for r in range(0, 1024, 7):
        o, d = oracle_lib.ray_f32(pose, intr, r)
        o, d = o.astype(np.float64), d.astype(np.float64)
        # brute force: sample the line densely, find where it is inside the box
        ts = np.linspace(0, 6, 60001)
        pts = o[None] + ts[:, None] * d[None]
        ins = np.all((pts >= -0.5) & (pts <= 0.5), axis=1)
        if counts[r] == 0:
            assert ins.sum() <= 1
            continue
        tt = t[off[r]:off[r + 1]].astype(np.float64)
        t_in = ts[ins]
        tn, tf = t_in.min(), t_in.max()
        assert np.allclose(tt, tn + (np.arange(32) + 0.5) * (tf - tn) / 32, atol=3e-4)
        assert delta[r] * 32 == pytest.approx(tf - tn, abs=3e-4)
        assert np.array_equal(j[off[r]:off[r + 1]], np.arange(32))


def test_march_lattice_occupancy_brute_force(oracle_lib):
    w, spec = tiny_spec()
    R = 16
    occ = synth.occupancy_pattern("checker", R)
    grid = synth.unpack_bits(occ, R)
    spec = dataclasses.replace(spec, march_mode=1, step=math.sqrt(3) / 128, max_samples=1000,
                               occ_res=R, occ_bits=occ)
    of = oracle_lib.OracleField(spec)
    intr = synth.intrinsics(w)
    pose = synth.ground_truth_pose(w, 1)
    pix = np.arange(0, 32 * 32, 5, dtype=np.int32)[None]
    off, t, j, delta = of.march(pose[None], pix, intr)
    assert np.all(delta == np.float32(spec.step))
    n_checked = 0
    for r in range(pix.shape[1]):
        o, d = oracle_lib.ray_f32(pose, intr, pix[0, r])
        o, d = o.astype(np.float64), d.astype(np.float64)
        jj = j[off[r]:off[r + 1]]
        tt = t[off[r]:off[r + 1]].astype(np.float64)
        assert np.all(np.diff(jj) > 0)
        if len(jj) == 0:
            continue
        # every lattice point j below the last kept one: kept iff its cell is occupied
        t0 = tt[0] - (jj[0] + 0.5) * spec.step
        for jl in range(int(jj[-1]) + 1):
            tl = t0 + (jl + 0.5) * spec.step
            p = o + tl * d
            assert _inside(p, (-0.5,) * 3, (0.5,) * 3, 1e-5)
            cell = np.clip(np.floor((p + 0.5) * R).astype(int), 0, R - 1)
            frac = (p + 0.5) * R - np.floor((p + 0.5) * R)
            if np.any(np.minimum(frac, 1 - frac) < 1e-4):
                continue  # on a cell face: either answer is correct
            assert grid[cell[2], cell[1], cell[0]] == (jl in set(jj.tolist()))
            n_checked += 1
    assert n_checked > 500


def test_march_lattice_cap_and_full_grid(oracle_lib):
    w, spec = tiny_spec()
    R = 8
    full = synth.occupancy_pattern("full", R)
    step = math.sqrt(3) / 256
    base = dict(march_mode=1, step=step, occ_res=R, occ_bits=full)
    of = oracle_lib.OracleField(dataclasses.replace(spec, max_samples=100000, **base))
    of_cap = oracle_lib.OracleField(dataclasses.replace(spec, max_samples=20, **base))
    intr = synth.intrinsics(w)
    pose = synth.ground_truth_pose(w, 2)
    pix = np.arange(0, 1024, 3, dtype=np.int32)[None]
    off, t, j, _ = of.march(pose[None], pix, intr)
    off_c, t_c, j_c, _ = of_cap.march(pose[None], pix, intr)
    n = np.diff(off)
    assert np.array_equal(np.diff(off_c), np.minimum(n, 20))
    for r in range(pix.shape[1]):
        # full grid: all lattice points 0..n-1 are kept, in order, the next one is past t_far
        assert np.array_equal(j[off[r]:off[r + 1]], np.arange(n[r]))
        assert np.array_equal(t_c[off_c[r]:off_c[r + 1]], t[off[r]:off[r] + min(n[r], 20)])


# --------------------------------------------------------------------- loss
def test_huber_loss_on_background_rays(oracle_lib):
    # sigma ~ 0 makes every ray show the background, so the loss is Huber(bg - I)
    w, spec = tiny_spec()
    bg = (0.3, 0.5, 0.05)
    of = oracle_lib.OracleField(dataclasses.replace(spec, density_bias=-200.0, background=bg))
    intr = synth.intrinsics(w)
    pose = synth.ground_truth_pose(w, 0)
    pix = np.array([[5, 100, 700, 1000]], np.int32)
    obs = np.zeros((32, 32, 3), np.float32)
    vals = np.array([[0.35, 0.2, 0.06], [0.3, 0.9, 0.0], [1.0, 0.5, 0.05], [0.25, 0.45, 0.1]],
                    np.float32)
    for p, v in zip(pix[0], vals):
        obs[p // 32, p % 32] = v
    out = of.render_loss_grad(pose[None], pix, obs, intr)
    r = np.array(bg)[None] - vals.astype(np.float64)
    dl = 0.1
    H = np.where(np.abs(r) <= dl, 0.5 * r * r, dl * (np.abs(r) - 0.5 * dl))
    assert out["loss"][0] == pytest.approx(H.sum() / (3 * 4), rel=1e-12)
    assert np.allclose(out["rgb"][0], np.array(bg)[None], atol=1e-12)


# --------------------------------------------------------------- pose maths
def test_exp_so3_textbook(oracle_lib):
    for th in [0.0, 1e-6, 1e-3, 0.5, 2.0, 3.1]:
        c, s = math.cos(th), math.sin(th)
        Rz = np.array([[c, -s, 0], [s, c, 0], [0, 0, 1]])
        assert np.allclose(oracle_lib.exp_so3([0, 0, th]), Rz, atol=1e-13)
    rng = np.random.default_rng(7)
    for _ in range(10):
        w = rng.normal(size=3) * rng.choice([1e-5, 0.1, 1.5])
        R = oracle_lib.exp_so3(w)
        assert np.allclose(R, Rotation.from_rotvec(w).as_matrix(), atol=1e-13)
        assert np.allclose(R @ oracle_lib.exp_so3(-w), np.eye(3), atol=1e-13)
        assert np.linalg.det(R) == pytest.approx(1.0, abs=1e-13)


def test_momentum_closed_form(oracle_lib):
    w, _ = tiny_spec()
    pose0 = synth.ground_truth_pose(w, 0)[None]
    g = np.array([[0.0, 0.0, 0.3, 0.2, -0.1, 0.05]], np.float32)
    lr, beta, n = 1e-2, 0.9, 30
    pose, m = pose0.copy(), np.zeros((1, 6), np.float32)
    for _ in range(n):
        pose, m = oracle_lib.step_momentum(pose, m, g, lr, beta)
    g64 = g.astype(np.float64)[0]
    assert np.allclose(m[0], g64 * (1 - beta ** n) / (1 - beta), rtol=1e-5)
    s = (n - beta * (1 - beta ** n) / (1 - beta)) / (1 - beta)   # sum_i (1-beta^i)/(1-beta)
    assert np.allclose(pose[0, :, 3], pose0[0, :, 3] - lr * s * g64[3:], atol=2e-6)
    Rz = Rotation.from_rotvec(-lr * s * g64[:3]).as_matrix()
    assert np.allclose(pose[0, :, :3], Rz @ pose0[0, :, :3], atol=2e-6)


def test_momentum_keeps_rotation_orthonormal(oracle_lib):
    w, _ = tiny_spec()
    pose = synth.perturb_poses(synth.ground_truth_pose(w, 0), 4, 30, 0.2, 0)
    m = np.zeros((4, 6), np.float32)
    rng = np.random.default_rng(8)
    for _ in range(1000):
        pose, m = oracle_lib.step_momentum(pose, m, rng.normal(size=(4, 6)).astype(np.float32),
                                           1e-2, 0.9)
    for k in range(4):
        R = pose[k, :, :3].astype(np.float64)
        assert np.abs(R.T @ R - np.eye(3)).max() < 1e-5


# ------------------------------------------------------------------- Adam
def _torch_adam_increments(grads, lr, beta1, beta2, eps, decay_base, decay_steps, staircase):
    """Per-step updates of torch.optim.Adam (float64) on a parameter that starts
    at 0, with torch's own schedulers for the two readings of the decay."""
    import torch
    theta = torch.zeros(grads.shape[1], dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([theta], lr=lr, betas=(beta1, beta2), eps=eps)
    if decay_steps == 0:
        sched = None
    elif staircase:
        sched = torch.optim.lr_scheduler.StepLR(opt, step_size=decay_steps, gamma=decay_base)
    else:
        sched = torch.optim.lr_scheduler.ExponentialLR(opt, gamma=decay_base ** (1.0 / decay_steps))
    out = []
    for g in grads:
        before = theta.detach().clone()
        theta.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        if sched is not None:
            sched.step()
        out.append((theta.detach() - before).numpy())
    return np.array(out)


def _adam_run(oracle_lib, pose0, grads, **kw):
    pose, st = pose0.copy(), np.zeros((pose0.shape[0], oracle_lib.ADAM_STATE), np.float32)
    for t, g in enumerate(grads):
        pose, st = oracle_lib.step_adam(pose, st, g, t, **kw)
    return pose, st


@pytest.mark.parametrize("decay_steps,staircase", [(0, 0), (64, 0), (64, 1)])
def test_adam_per_component_matches_torch_adam(oracle_lib, decay_steps, staircase):
    """Sec. IV-A/IV-D Adam with per-component second moments: the translation
    follows torch's Adam on the camera centre, and the orientation is the
    product of the rotations given by torch's Adam steps on a rotation vector."""
    w, _ = tiny_spec()
    pose0 = synth.ground_truth_pose(w, 0)[None]
    rng = np.random.default_rng(5)
    n = 150
    scales = np.array([1e-3, 0.3, 4.0, 2e-2, 1.0, 0.1])
    grads = (rng.normal(size=(n, 1, 6)) * scales).astype(np.float32)
    grads[rng.uniform(size=grads.shape) < 0.05] = 0.0
    hp = dict(lr_rot=5e-3, lr_trans=3e-3, beta1=0.9, beta2=0.999, eps=1e-8, decay_base=0.33,
              decay_steps=decay_steps, staircase=staircase)
    pose, st = _adam_run(oracle_lib, pose0, grads, **hp)
    g64 = grads[:, 0].astype(np.float64)
    common = dict(beta1=0.9, beta2=0.999, eps=1e-8, decay_base=0.33, decay_steps=decay_steps,
                  staircase=staircase)
    du = _torch_adam_increments(g64[:, 3:], 3e-3, **common)
    dw = _torch_adam_increments(g64[:, :3], 5e-3, **common)
    tol = n * 2.0 ** -23  # float32 pose storage after each of the n steps
    assert np.allclose(pose[0, :, 3], pose0[0, :, 3] + du.sum(0), atol=tol, rtol=0)
    R = pose0[0, :, :3].astype(np.float64)
    for inc in dw:
        R = Rotation.from_rotvec(inc).as_matrix() @ R
    assert np.allclose(pose[0, :, :3], R, atol=tol, rtol=0)
    assert st[0, 12] == n and np.all(st[0, 13:] == 0)
    # the moments are Adam's exponential averages of g and g^2; float storage
    # each step bounds their relative error by 2^-24 / (1 - beta)
    b = 0.9 ** np.arange(n)[::-1]
    assert np.allclose(st[0, :6], 0.1 * (b[:, None] * g64).sum(0), rtol=1e-5, atol=1e-12)
    b2 = 0.999 ** np.arange(n)[::-1]
    assert np.allclose(st[0, 6:12], 1e-3 * (b2[:, None] * g64 ** 2).sum(0), rtol=1e-4,
                       atol=1e-15)


def test_adam_restarts_bias_correction_after_reset(oracle_lib):
    """A hypothesis whose state was cleared at global step s0 (a redrawn slot)
    continues as a fresh Adam run -- its bias correction counts its own steps --
    while the learning rate keeps decaying with the global step."""
    w, _ = tiny_spec()
    pose0 = synth.ground_truth_pose(w, 0)[None]
    rng = np.random.default_rng(6)
    s0, n, D = 40, 30, 64
    grads = (rng.normal(size=(s0 + n, 1, 6)) * [0.3, 1, 0.02, 1, 0.1, 2]).astype(np.float32)
    hp = dict(lr_rot=5e-3, lr_trans=3e-3, decay_base=0.33, decay_steps=D)
    pose, st = pose0.copy(), np.zeros((1, oracle_lib.ADAM_STATE), np.float32)
    for t in range(s0):
        pose, st = oracle_lib.step_adam(pose, st, grads[t], t, **hp)
    mid = pose.copy()
    st[:] = 0.0
    for t in range(s0, s0 + n):
        pose, st = oracle_lib.step_adam(pose, st, grads[t], t, **hp)
    g64 = grads[s0:, 0].astype(np.float64)
    f0 = 0.33 ** (s0 / D)
    common = dict(beta1=0.9, beta2=0.999, eps=1e-8, decay_base=0.33, decay_steps=D, staircase=0)
    du = _torch_adam_increments(g64[:, 3:], 3e-3 * f0, **common)
    dw = _torch_adam_increments(g64[:, :3], 5e-3 * f0, **common)
    tol = n * 2.0 ** -23
    assert np.allclose(pose[0, :, 3], mid[0, :, 3] + du.sum(0), atol=tol, rtol=0)
    R = mid[0, :, :3].astype(np.float64)
    for inc in dw:
        R = Rotation.from_rotvec(inc).as_matrix() @ R
    assert np.allclose(pose[0, :, :3], R, atol=tol, rtol=0)
    assert st[0, 12] == n


@pytest.mark.parametrize("staircase", [0, 1])
def test_adam_per_subspace_constant_gradient_closed_form(oracle_lib, staircase):
    """A constant gradient makes the bias-corrected moments exactly g and |g|^2,
    so every step moves lr(t) |g| / (|g| + eps) against g; the rotations share
    one axis and compose to a single Exp."""
    w, _ = tiny_spec()
    pose0 = synth.ground_truth_pose(w, 1)[None]
    g = np.array([[0.02, -0.05, 0.01, 0.3, 0.0, -0.4]], np.float32)
    n, D, base, eps = 300, 64, 0.33, 1e-8
    pose, _ = _adam_run(oracle_lib, pose0, [g] * n, lr_rot=5e-3, lr_trans=3e-3, decay_base=base,
                        decay_steps=D, staircase=staircase, second_moment=1, eps=eps)
    t = np.arange(n)
    f = base ** (np.floor(t / D) if staircase else t / D)
    g64 = g[0].astype(np.float64)
    gw, gt = g64[:3], g64[3:]
    shift = -3e-3 * f.sum() * gt / (np.linalg.norm(gt) + eps)
    turn = -5e-3 * f.sum() * gw / (np.linalg.norm(gw) + eps)
    # the pose is stored in float32 after each step: with a constant increment
    # the rounding can be systematic, n half-ulps of a unit-sized value at most
    tol = n * 2.0 ** -23
    assert np.allclose(pose[0, :, 3], pose0[0, :, 3] + shift, atol=tol, rtol=0)
    R = Rotation.from_rotvec(turn).as_matrix() @ pose0[0, :, :3].astype(np.float64)
    assert np.allclose(pose[0, :, :3], R, atol=tol, rtol=0)


def test_adam_per_subspace_is_rotation_invariant(oracle_lib):
    """Rotating the world by Q (pose -> Q pose, torque and force -> Q g) rotates
    the per-subspace Adam trajectory by Q; per-component second moments are tied
    to the world axes and do not have this symmetry."""
    w, _ = tiny_spec()
    pose0 = synth.perturb_poses(synth.ground_truth_pose(w, 2), 3, 20, 0.1, 3)
    rng = np.random.default_rng(11)
    grads = rng.normal(size=(60, 3, 6)).astype(np.float64) * [0.1, 0.1, 0.1, 1, 1, 1]
    Q = Rotation.from_rotvec([0.7, -0.4, 1.1]).as_matrix()
    qpose0 = np.einsum("ij,kjl->kil", Q, pose0.astype(np.float64)).astype(np.float32)
    qgrads = np.concatenate([grads[..., :3] @ Q.T, grads[..., 3:] @ Q.T], axis=-1)
    errs = []
    for mode in (1, 0):
        a, _ = _adam_run(oracle_lib, pose0, grads.astype(np.float32), lr_rot=2e-2,
                         lr_trans=2e-2, second_moment=mode)
        b, _ = _adam_run(oracle_lib, qpose0, qgrads.astype(np.float32), lr_rot=2e-2,
                         lr_trans=2e-2, second_moment=mode)
        errs.append(np.abs(np.einsum("ij,kjl->kil", Q, a.astype(np.float64)) - b).max())
    assert errs[0] < 1e-5
    assert errs[1] > 1e-3


def _hat4(xi):
    w, v = xi[:3], xi[3:]
    M = np.zeros((4, 4))
    M[:3, :3] = [[0, -w[2], w[1]], [w[2], 0, -w[0]], [-w[1], w[0], 0]]
    M[:3, 3] = v
    return M


def _fit_loss(R, o, pts, tgt):
    """A smooth pose loss: camera-frame points mapped to the world by (R, o)
    against fixed world targets."""
    return float(np.sum((pts @ R.T + o - tgt) ** 2))


@pytest.mark.parametrize("lr_rot,lr_trans", [(5e-3, 3e-3), (1e-5, 3e-3), (0.5, 1.0)])
def test_adam_se3_twist_step_matches_expm(oracle_lib, lr_rot, lr_trans):
    """The coupled se(3) representation compared in Sec. IV-A: the optimiser
    runs on the twist about the world origin and moves T to Exp(u) T.  The
    twist gradient is taken by central differences through scipy's matrix
    exponential, the input dpose by central differences in the library's own
    parametrisation (rotation about the camera centre, shift of the centre).
    A first per-subspace Adam step from a fresh state moves the twist by
    -lr G / (|G| + eps) in each subspace, applied with expm (the large step
    makes the second-order terms of the exponential's translation visible)."""
    from scipy.linalg import expm
    rng = np.random.default_rng(21)
    w, _ = tiny_spec()
    poses = synth.perturb_poses(synth.ground_truth_pose(w, 4), 3, 25, 0.3, 5)
    pts = rng.normal(size=(6, 3))
    tgt = rng.normal(size=(6, 3))
    h = 1e-6
    dpose = np.zeros((3, 6), np.float32)
    G = np.zeros((3, 6))
    for k in range(3):
        T = np.eye(4)
        T[:3, :] = poses[k].astype(np.float64)
        R, o = T[:3, :3], T[:3, 3]
        for a in range(3):
            e = np.zeros(3)
            e[a] = h
            Rp, Rm = Rotation.from_rotvec(e).as_matrix() @ R, Rotation.from_rotvec(-e).as_matrix() @ R
            dpose[k, a] = (_fit_loss(Rp, o, pts, tgt) - _fit_loss(Rm, o, pts, tgt)) / (2 * h)
            dpose[k, 3 + a] = (_fit_loss(R, o + e, pts, tgt) - _fit_loss(R, o - e, pts, tgt)) / (2 * h)
        for i in range(6):
            xi = np.zeros(6)
            xi[i] = h
            Tp, Tm = expm(_hat4(xi)) @ T, expm(_hat4(-xi)) @ T
            G[k, i] = (_fit_loss(Tp[:3, :3], Tp[:3, 3], pts, tgt) -
                       _fit_loss(Tm[:3, :3], Tm[:3, 3], pts, tgt)) / (2 * h)
    lr = np.array([lr_rot, lr_trans])
    eps = 1e-8
    st = np.zeros((3, oracle_lib.ADAM_STATE), np.float32)
    out, st1 = oracle_lib.step_adam(poses, st, dpose, 0, lr_rot, lr_trans, eps=eps,
                                    second_moment=1, representation=1)
    for k in range(3):
        # the float32 dpose carries ~1e-7 relative error into G
        Gk = G[k]
        u = np.concatenate([-lr[s] * Gk[3 * s:3 * s + 3] / (np.linalg.norm(Gk[3 * s:3 * s + 3]) + eps)
                            for s in range(2)])
        T = np.eye(4)
        T[:3, :] = poses[k].astype(np.float64)
        want = (expm(_hat4(u)) @ T)[:3, :]
        assert np.allclose(out[k], want, atol=4e-7 * max(1.0, np.abs(want).max()), rtol=0), k
    # the first moments are (1 - beta1) times the twist gradient
    assert np.allclose(st1[:, :6], 0.1 * G, rtol=1e-5, atol=1e-9)
    # the decoupled representation moves differently from the same gradient
    out0, _ = oracle_lib.step_adam(poses, st, dpose, 0, lr_rot, lr_trans, eps=eps,
                                   second_moment=1)
    assert np.abs(out0 - out).max() > 1e-5


def test_adam_keeps_rotation_orthonormal(oracle_lib):
    w, _ = tiny_spec()
    pose = synth.perturb_poses(synth.ground_truth_pose(w, 0), 4, 30, 0.2, 0)
    rng = np.random.default_rng(12)
    pose, _ = _adam_run(oracle_lib, pose, rng.normal(size=(1000, 4, 6)).astype(np.float32),
                        lr_rot=5e-3, lr_trans=3e-3, decay_base=0.33, decay_steps=256)
    for k in range(4):
        R = pose[k, :, :3].astype(np.float64)
        assert np.abs(R.T @ R - np.eye(3)).max() < 1e-5


# --------------------------------------------------------------- resampling
def test_splitmix64_published_vectors(oracle_lib):
    # reference outputs of SplitMix64 started at state 0
    assert oracle_lib.splitmix64_stream(0, 3) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4,
                                                   0x06C45D188009454F]


def test_box_muller_normals_statistics(oracle_lib):
    z = np.array([oracle_lib.normals6(1234, r, s) for r in range(4) for s in range(1500)]).ravel()
    assert abs(z.mean()) < 0.02 and abs(z.std() - 1) < 0.02
    assert abs(np.mean(z ** 4) - 3) < 0.15                 # Gaussian kurtosis


def test_resample_keeps_argsort_and_redraws_rest(oracle_lib):
    w, _ = tiny_spec()
    K = 37
    poses = synth.perturb_poses(synth.ground_truth_pose(w, 0), K, 30, 0.2, 1)
    mom = np.random.default_rng(9).normal(size=(K, 6)).astype(np.float32)
    loss = np.random.default_rng(10).uniform(0, 1, K).astype(np.float32)
    loss[[3, 11]] = np.nan
    loss[[5, 6]] = loss[4]                                  # ties break by index
    out_p, out_m, rank = oracle_lib.resample(poses, mom, loss, 0.25, math.radians(5), 0.03, 77, 2)
    order = np.argsort(loss, kind="stable")                 # numpy puts NaN last
    assert np.array_equal(np.argsort(rank), order)
    n_keep = int(K * 0.25)
    kept = set(order[:n_keep].tolist())
    redrawn = [i for i in range(K) if i not in kept]
    assert len(redrawn) == K - n_keep
    for q, i in enumerate(redrawn):
        parent = order[q % n_keep]
        Rrel = out_p[i, :, :3].astype(np.float64) @ poses[parent, :, :3].T.astype(np.float64)
        ang = np.linalg.norm(Rotation.from_matrix(Rrel).as_rotvec())
        assert ang < math.radians(5) * 6
        assert np.linalg.norm(out_p[i, :, 3] - poses[parent, :, 3]) < 0.03 * 7
        assert np.all(out_m[i] == 0)
    for i in kept:
        assert np.array_equal(out_p[i], poses[i]) and np.array_equal(out_m[i], mom[i])


def test_resample_clears_adam_state_rows(oracle_lib):
    w, _ = tiny_spec()
    K = 16
    poses = synth.perturb_poses(synth.ground_truth_pose(w, 0), K, 30, 0.2, 1)
    st = np.random.default_rng(2).normal(size=(K, oracle_lib.ADAM_STATE)).astype(np.float32)
    loss = np.random.default_rng(3).uniform(0, 1, K).astype(np.float32)
    out_p, out_s, rank = oracle_lib.resample(poses, st, loss, 0.25, 0.05, 0.03, 5, 1)
    for i in range(K):
        if rank[i] < 4:
            assert np.array_equal(out_s[i], st[i]) and np.array_equal(out_p[i], poses[i])
        else:
            assert np.all(out_s[i] == 0)
    # the state width does not change which slots are kept or where they go
    p6, _, rank6 = oracle_lib.resample(poses, st[:, :6], loss, 0.25, 0.05, 0.03, 5, 1)
    p0, _, _ = oracle_lib.resample(poses, None, loss, 0.25, 0.05, 0.03, 5, 1)
    assert np.array_equal(rank6, rank) and np.array_equal(p6, out_p) and np.array_equal(p0, out_p)


# ------------------------------------------------------ structured density
def test_bump_field_density_closed_form(oracle_lib):
    """On the bump field only feature 0 of the dense level 0 drives the
    density: sigma(p) = exp(GAIN relu(trilinear blend of the bump's vertex
    values at p) - OFFSET), the blend written out with numpy."""
    w = synth.WORKLOADS["tiny_bump"]
    fa = synth.make_field(w, 0)
    of = oracle_lib.OracleField(synth.field_spec(w, fa, occ_res=0))
    N = int(fa.level_res[0])
    n1 = N + 1
    vals = fa.table[0, :n1 ** 3, 0].astype(np.float64).reshape(n1, n1, n1)  # [k][j][i]
    rng = np.random.default_rng(3)
    for x in rng.uniform(0.0, 1.0, size=(50, 3)):
        feat, _ = of.encode(x.astype(np.float32), x)
        sigma = math.exp(of.density_mlp(feat)[0] + fa.density_bias)
        pos = x * N
        i0 = np.minimum(pos.astype(int), N - 1)
        t = pos - i0
        v = 0.0
        for dk in (0, 1):
            for dj in (0, 1):
                for di in (0, 1):
                    wgt = ((t[0] if di else 1 - t[0]) * (t[1] if dj else 1 - t[1]) *
                           (t[2] if dk else 1 - t[2]))
                    v += wgt * vals[i0[2] + dk, i0[1] + dj, i0[0] + di]
        want = math.exp(synth.BUMP_GAIN * max(v, 0.0) - synth.BUMP_OFFSET)
        assert sigma == pytest.approx(want, rel=1e-6)


def test_bump_workload_skips_and_stops_early(oracle_lib):
    """The structured workload exercises occupancy skipping and early ray
    termination (the random fields leave every cell occupied and no ray
    opaque)."""
    import dataclasses
    w = synth.WORKLOADS["tiny_bump"]
    spec = synth.field_spec(w, synth.make_field(w, 0))
    of0 = oracle_lib.OracleField(dataclasses.replace(spec, occ_res=0, occ_bits=None))
    bits = of0.build_occupancy(w.occ_res, w.occ_threshold)
    occ = synth.unpack_bits(bits, w.occ_res)
    assert 0.05 < occ.mean() < 0.5
    of = oracle_lib.OracleField(dataclasses.replace(spec, occ_bits=bits))
    gt = synth.ground_truth_pose(w, 0)
    poses = synth.perturb_poses(gt, w.K, w.max_rot_deg, w.max_trans, 0)
    pix = synth.pixel_batch(0, 0, w.K, w.P, w.width, w.height)
    intr = synth.intrinsics(w)
    m = of.march(poses, pix, intr)
    cnt = np.diff(m[0])
    out = of.shade(poses.astype(np.float64), pix, np.zeros((w.height, w.width, 3), np.float32),
                   intr, m)
    hit = cnt > 0
    assert 0.05 < hit.mean() < 0.9
    assert np.sum(out["stop"][hit] < cnt[hit]) >= 5          # opaque rays stop early


# --------------------------------------------------------------- occupancy
def test_occupancy_build(oracle_lib):
    w, spec = tiny_spec()
    R = 8
    for bias, want in [(-200.0, 0), (200.0, 1)]:
        of = oracle_lib.OracleField(dataclasses.replace(spec, density_bias=bias))
        bits = synth.unpack_bits(of.build_occupancy(R, 0.01), R)
        assert np.all(bits == bool(want))
    # threshold between the min and max centre density: compare with a numpy evaluation
    of = oracle_lib.OracleField(spec)
    sig = np.zeros((R, R, R))
    relu = lambda z: np.maximum(z, 0)
    for z in range(R):
        for y in range(R):
            for x in range(R):
                c = (np.array([x, y, z]) + 0.5) / R
                feat, _ = of.encode(c.astype(np.float32), c)
                h = relu(feat @ spec.w_density1.astype(np.float64)) @ spec.w_density2.astype(np.float64)
                sig[z, y, x] = math.exp(h[0] - 1.0)
    thr = float(np.median(sig))
    bits = synth.unpack_bits(of.build_occupancy(R, thr), R)
    assert np.array_equal(bits, sig > thr)


# ------------------------------------------------------------ pixel losses
# Loss types of the pixel-based RGB losses (paper Sec. IV-C): 0 Huber, 1 L1,
# 2 L2, 3 Log L1, 4 Relative L2, 5 MAPE, 6 sMAPE, 7 Smooth L1.
LOSSES = range(8)


def test_pixel_losses_identities(oracle_lib):
    O = oracle_lib
    rng = np.random.default_rng(7)
    for C, y in rng.uniform(-0.2, 1.2, size=(200, 2)):
        r = C - y
        eps, th = 0.01, 0.1
        v = {t: O.pixel_loss(t, C, y, th if t in (0, 7) else eps)[0] for t in LOSSES}
        l1, l2 = O.pixel_loss(1, C, y, 1.0)[0], O.pixel_loss(2, C, y, 1.0)[0]
        # definitions tied to each other rather than restated
        assert math.isclose(l1, abs(C - y), rel_tol=0, abs_tol=1e-15)
        assert math.isclose(l2, l1 * l1, rel_tol=1e-13)
        assert math.isclose(v[7], v[0] / th, rel_tol=1e-13)          # Smooth L1_b = Huber_b / b
        assert math.isclose(v[3], math.log1p(l1), rel_tol=1e-13)      # log of (1 + L1)
        assert math.isclose(v[4] * (y * y + eps), l2, rel_tol=1e-13)  # L2 relative to the target
        assert math.isclose(v[5] * (abs(y) + eps), l1, rel_tol=1e-13) # L1 relative to the target
        # sMAPE: symmetric in (prediction, target), bounded by 2
        assert math.isclose(v[6], O.pixel_loss(6, y, C, eps)[0], rel_tol=1e-13)
        assert 0.0 <= v[6] <= 2.0
        if abs(r) <= th:   # Huber is half of L2 inside its threshold
            assert math.isclose(v[0], 0.5 * l2, rel_tol=1e-13)
        assert all(x >= 0.0 for x in v.values())
    for t in LOSSES:       # no loss at a perfect match
        assert O.pixel_loss(t, 0.37, 0.37, 0.05)[0] == 0.0


@pytest.mark.parametrize("loss_type", LOSSES)
def test_pixel_loss_derivative_fd(oracle_lib, loss_type):
    O = oracle_lib
    rng = np.random.default_rng(loss_type)
    p = 0.1 if loss_type in (0, 7) else 0.01
    n = 0
    for C, y in rng.uniform(0.0, 1.0, size=(200, 2)):
        v, g, kink = O.pixel_loss(loss_type, C, y, p)
        if kink < 1e-3 or (loss_type in (0, 7) and abs(abs(C - y) - p) < 1e-3):
            continue
        h = 1e-7
        fd = (O.pixel_loss(loss_type, C + h, y, p)[0] - O.pixel_loss(loss_type, C - h, y, p)[0]) / (2 * h)
        assert abs(fd - g) <= 1e-6 * max(1.0, abs(g)), (C, y, fd, g)
        n += 1
    assert n > 150
