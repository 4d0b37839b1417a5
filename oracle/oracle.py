"""ctypes binding of the CPU oracle (oracle/pnerf_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg.  The product path never loads it.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "pnerf_oracle.c")
# PNERF_ORACLE_LIB: load another build of the same source (the sanitizer test's)
LIB = os.environ.get("PNERF_ORACLE_LIB") or os.path.join(HERE, "liboracle.so")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc: -O2, no contraction, no fast-math, OpenMP."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-fPIC", "-shared", "-Wall", SRC, "-o", LIB + ".tmp", "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(LIB + ".tmp", LIB)
    return LIB


class _Intr(C.Structure):
    _fields_ = [("width", C.c_int32), ("height", C.c_int32), ("fx", C.c_float),
                ("fy", C.c_float), ("cx", C.c_float), ("cy", C.c_float)]


class _Field(C.Structure):
    _fields_ = [("L", C.c_int32), ("F", C.c_int32), ("T", C.c_uint32),
                ("level_res", C.c_void_p), ("dense_coarse", C.c_int32),
                ("table", C.c_void_p), ("din", C.c_int32),
                ("wd1", C.c_void_p), ("wd2", C.c_void_p),
                ("wc1", C.c_void_p), ("wc2", C.c_void_p), ("wc3", C.c_void_p),
                ("density_bias", C.c_double),
                ("aabb_min", C.c_float * 3), ("aabb_max", C.c_float * 3),
                ("march_mode", C.c_int32), ("n_uniform", C.c_int32), ("step", C.c_float),
                ("max_samples", C.c_int32), ("t_stop", C.c_double),
                ("occ_res", C.c_int32), ("occ_bits", C.c_void_p),
                ("bg", C.c_double * 3), ("loss_type", C.c_int32), ("loss_param", C.c_double),
                ("sh_dir_grad", C.c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=False)
        L = C.CDLL(LIB)
        vp, i32, i64, u32, u64, f32, f64 = (C.c_void_p, C.c_int32, C.c_int64, C.c_uint32,
                                            C.c_uint64, C.c_float, C.c_double)
        L.orc_grid_index.restype = u32
        L.orc_grid_index.argtypes = [vp, i32, u32, u32, u32]
        L.orc_ray_f32.argtypes = [vp, vp, i32, vp, vp]
        L.orc_march.restype = i32
        L.orc_march.argtypes = [vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, i64, i32]
        L.orc_shade.restype = i32
        L.orc_shade.argtypes = [vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                vp, vp, i32]
        L.orc_shade_ray_variant.restype = i32
        L.orc_shade_ray_variant.argtypes = [vp, vp, i32, i32, vp, vp, vp, i32, f32, vp, vp, vp,
                                            vp, vp, vp, vp]
        L.orc_shade_ray_jobs.restype = i32
        L.orc_shade_ray_jobs.argtypes = [vp, vp, i32, vp, vp, vp, f64, i32, vp, vp, vp, vp, vp,
                                         vp, i32]
        L.orc_encode.argtypes = [vp, vp, vp, vp, vp, vp]
        L.orc_sh16.argtypes = [vp, vp, vp]
        L.orc_density_mlp.argtypes = [vp, vp, vp]
        L.orc_color_mlp.argtypes = [vp, vp, vp]
        L.orc_composite.argtypes = [i32, vp, vp, f64, vp, f64, vp, vp, vp, vp]
        L.orc_composite_grad.argtypes = [i32, vp, vp, f64, vp, f64, vp, vp, vp]
        L.orc_exp_so3.argtypes = [vp, vp]
        L.orc_pixel_loss.restype = f64
        L.orc_pixel_loss.argtypes = [i32, f64, f64, f64, vp, vp]
        L.orc_step_momentum.argtypes = [i32, vp, vp, vp, f32, f32]
        L.orc_step_adam.argtypes = [i32, vp, vp, vp, i32, vp]
        L.orc_resample.argtypes = [i32, vp, vp, i32, vp, f32, f32, f32, u64, u32, vp]
        L.orc_splitmix64_next.restype = u64
        L.orc_splitmix64_next.argtypes = [vp]
        L.orc_normals6.argtypes = [u64, u32, u32, vp]
        L.orc_build_occupancy.argtypes = [vp, i32, f32, vp, i32]
        _lib = L
    return _lib


def _p(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def n_threads_default() -> int:
    """Host threads for the oracle: the process's CPU affinity, capped by
    OMP_NUM_THREADS when that is set."""
    n = len(os.sched_getaffinity(0))
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, n)


def intr_struct(intr: dict) -> _Intr:
    return _Intr(int(intr["width"]), int(intr["height"]), float(intr["fx"]), float(intr["fy"]),
                 float(intr["cx"]), float(intr["cy"]))


SAMPLE_COLS = 17  # columns of the per-sample output (ORC_SAMPLE_COLS)


class _Variant(C.Structure):
    _fields_ = [("relu_margin", C.c_double), ("relu_pattern", C.c_void_p),
                ("relu_pattern_all", C.c_int32), ("stop", C.c_int32), ("loss_sign", C.c_int32 * 3)]


# one ray of a batch of variant shadings (orc_ray_job)
RAY_JOB = np.dtype([("hyp", np.int32), ("pix", np.int32), ("t0", np.int64), ("n", np.int32),
                    ("delta", np.float32), ("stop", np.int32), ("loss_sign", np.int32, 3),
                    ("relu_pattern", np.int32)], align=True)


class OracleField:
    """A field (synth.FieldSpec) converted to the oracle's double-precision form."""

    def __init__(self, spec):
        self.spec = spec
        f64 = lambda a: np.ascontiguousarray(np.asarray(a).astype(np.float64))
        self.level_res = np.ascontiguousarray(spec.level_res, dtype=np.int32)
        self.table = f64(spec.table)
        self.wd1, self.wd2 = f64(spec.w_density1), f64(spec.w_density2)
        self.wc1, self.wc2, self.wc3 = f64(spec.w_color1), f64(spec.w_color2), f64(spec.w_color3)
        self.occ = (None if spec.occ_bits is None
                    else np.ascontiguousarray(spec.occ_bits, dtype=np.uint32))
        if spec.occ_res > 0 and self.occ is None:
            raise ValueError("oracle needs explicit occupancy bits when occ_res > 0")
        s = _Field()
        s.L, s.F, s.T = spec.n_levels, spec.n_features, 1 << spec.log2_table
        s.level_res = _p(self.level_res).value
        s.dense_coarse = spec.dense_coarse_levels
        s.table = _p(self.table).value
        s.din = spec.n_levels * spec.n_features
        s.wd1, s.wd2 = _p(self.wd1).value, _p(self.wd2).value
        s.wc1, s.wc2, s.wc3 = _p(self.wc1).value, _p(self.wc2).value, _p(self.wc3).value
        s.density_bias = spec.density_bias
        s.aabb_min = (C.c_float * 3)(*spec.aabb_min)
        s.aabb_max = (C.c_float * 3)(*spec.aabb_max)
        s.march_mode, s.n_uniform, s.step = spec.march_mode, spec.n_uniform, spec.step
        s.max_samples, s.t_stop = spec.max_samples, spec.t_stop
        s.occ_res = spec.occ_res
        s.occ_bits = None if self.occ is None else _p(self.occ).value
        s.bg = (C.c_double * 3)(*spec.background)
        s.loss_type, s.loss_param, s.sh_dir_grad = spec.loss_type, spec.loss_param, spec.sh_dir_grad
        self.s = s

    @property
    def ptr(self):
        return C.byref(self.s)

    # ------------------------------------------------------------ pieces
    def grid_index(self, level: int, i: int, j: int, k: int) -> int:
        return lib().orc_grid_index(self.ptr, level, i, j, k)

    def encode(self, x32, x64=None, clamped=(0, 0, 0)):
        x32 = np.ascontiguousarray(x32, dtype=np.float32)
        x64 = np.ascontiguousarray(x32 if x64 is None else x64, dtype=np.float64)
        cl = np.ascontiguousarray(clamped, dtype=np.int32)
        din = self.s.din
        feat = np.zeros(din)
        jac = np.zeros((3, din))
        lib().orc_encode(self.ptr, _p(x32), _p(x64), _p(cl), _p(feat), _p(jac))
        return feat, jac

    def density_mlp(self, feat):
        feat = np.ascontiguousarray(feat, dtype=np.float64)
        h = np.zeros(16)
        lib().orc_density_mlp(self.ptr, _p(feat), _p(h))
        return h

    def color_mlp(self, xc):
        xc = np.ascontiguousarray(xc, dtype=np.float64)
        rgb = np.zeros(3)
        lib().orc_color_mlp(self.ptr, _p(xc), _p(rgb))
        return rgb

    # ------------------------------------------------------------ path
    def march(self, poses, pix, intr, capacity=None, threads=None):
        poses = np.ascontiguousarray(poses, dtype=np.float32).reshape(-1, 12)
        pix = np.ascontiguousarray(pix, dtype=np.int32)
        K, P = pix.shape
        off = np.zeros(K * P + 1, dtype=np.int64)
        delta = np.zeros(K * P, dtype=np.float32)
        it = intr_struct(intr)
        nt = threads or n_threads_default()
        lib().orc_march(self.ptr, K, _p(poses), P, _p(pix), C.byref(it), _p(off), None, None,
                        _p(delta), 0, nt)
        total = int(off[-1])
        if capacity is not None and total > capacity:
            return off, None, None, delta
        t = np.zeros(max(total, 1), dtype=np.float32)
        j = np.zeros(max(total, 1), dtype=np.int32)
        rc = lib().orc_march(self.ptr, K, _p(poses), P, _p(pix), C.byref(it), _p(off), _p(t),
                             _p(j), _p(delta), max(total, 1), nt)
        assert rc == 0
        return off, t[:total], j[:total], delta

    def shade(self, poses64, pix, obs, intr, march, sh_dirs=None, threads=None,
              per_sample=False):
        poses64 = np.ascontiguousarray(poses64, dtype=np.float64).reshape(-1, 12)
        pix = np.ascontiguousarray(pix, dtype=np.int32)
        K, P = pix.shape
        obs = np.ascontiguousarray(obs, dtype=np.float32)
        off, t, _, delta = march
        t = np.ascontiguousarray(t if t.size else np.zeros(1, np.float32), dtype=np.float32)
        sd = None if sh_dirs is None else np.ascontiguousarray(sh_dirs, dtype=np.float64)
        loss = np.zeros(K)
        dpose = np.zeros((K, 6))
        rgb = np.zeros((K * P, 3))
        stop = np.zeros(K * P, dtype=np.int32)
        sig = np.zeros(1, dtype=np.uint64)
        so = np.zeros((max(int(off[-1]), 1), SAMPLE_COLS)) if per_sample else None
        it = intr_struct(intr)
        rc = lib().orc_shade(self.ptr, K, _p(poses64), P, _p(pix), _p(obs), C.byref(it), _p(off),
                             _p(t), _p(delta), _p(sd), _p(loss), _p(dpose), _p(rgb), _p(stop),
                             _p(sig), _p(so), threads or n_threads_default())
        if rc != 0:
            raise ValueError("oracle: unsupported field configuration")
        out = dict(loss=loss, dpose=dpose, rgb=rgb.reshape(K, P, 3), stop=stop,
                   signature=int(sig[0]))
        if per_sample:
            out["samples"] = so[: int(off[-1])]
        return out

    def shade_ray_variant(self, pose, P, pix, obs, intr, t, delta, relu_margin=0.0,
                          relu_pattern=None, stop=-1, loss_sign=(0, 0, 0)):
        """One ray (pixel `pix` of a hypothesis with `pose` and P pixels, samples t
        at spacing delta) with chosen threshold decisions taken the other way
        (orc_shade_ray_variant).  Returns dict(samples [n][SAMPLE_COLS], near [n],
        loss, g [6], rgb [3], stop)."""
        pose = np.ascontiguousarray(np.asarray(pose, np.float32).astype(np.float64).reshape(12))
        t = np.ascontiguousarray(t, dtype=np.float32)
        n = int(t.size)
        obs = np.ascontiguousarray(obs, dtype=np.float32)
        pat = None if relu_pattern is None else np.ascontiguousarray(relu_pattern, np.int32)
        assert pat is None or pat.size == n
        v = _Variant(float(relu_margin), None if pat is None else _p(pat).value, 0, int(stop),
                     (C.c_int32 * 3)(*[int(x) for x in loss_sign]))
        so = np.zeros((max(n, 1), SAMPLE_COLS))
        near = np.zeros(max(n, 1), np.int32)
        loss = np.zeros(1)
        g = np.zeros(6)
        rgb = np.zeros(3)
        used = np.zeros(1, np.int32)
        it = intr_struct(intr)
        tt = t if n else np.zeros(1, np.float32)
        rc = lib().orc_shade_ray_variant(self.ptr, _p(pose), int(P), int(pix), _p(obs),
                                         C.byref(it), _p(tt), n, float(delta), C.byref(v),
                                         _p(so), _p(near), _p(loss), _p(g), _p(rgb), _p(used))
        if rc != 0:
            raise ValueError("oracle: unsupported field configuration")
        return dict(samples=so[:n], near=near[:n], loss=float(loss[0]), g=g, rgb=rgb,
                    stop=int(used[0]))

    def shade_ray_jobs(self, poses, P, obs, intr, t, jobs, relu_margin, threads=None):
        """Many rays with chosen decisions taken the other way (orc_shade_ray_jobs).
        jobs: a RAY_JOB array.  Returns (samples [sum n][SAMPLE_COLS], near [sum n],
        first row of each job [n_jobs], loss [n_jobs], g [n_jobs][6])."""
        poses = np.ascontiguousarray(np.asarray(poses, np.float32).astype(np.float64).reshape(-1, 12))
        jobs = np.ascontiguousarray(jobs, dtype=RAY_JOB)
        nj = len(jobs)
        rows = np.zeros(max(nj, 1), np.int64)
        if nj:
            rows[1:nj] = np.cumsum(jobs["n"].astype(np.int64))[:-1]
        total = int(jobs["n"].sum()) if nj else 0
        so = np.zeros((max(total, 1), SAMPLE_COLS))
        near = np.zeros(max(total, 1), np.int32)
        loss = np.zeros(max(nj, 1))
        g = np.zeros((max(nj, 1), 6))
        t = np.ascontiguousarray(t if np.size(t) else np.zeros(1, np.float32), dtype=np.float32)
        obs = np.ascontiguousarray(obs, dtype=np.float32)
        it = intr_struct(intr)
        rc = lib().orc_shade_ray_jobs(self.ptr, _p(poses), int(P), _p(obs), C.byref(it), _p(t),
                                      float(relu_margin), nj, _p(jobs), _p(rows), _p(so), _p(near),
                                      _p(loss), _p(g), threads or n_threads_default())
        if rc != 0:
            raise ValueError("oracle: unsupported field configuration")
        return so[:total], near[:total], rows[:nj], loss[:nj], g[:nj]

    def render_loss_grad(self, poses, pix, obs, intr, threads=None, per_sample=False):
        m = self.march(poses, pix, intr, threads=threads)
        out = self.shade(np.asarray(poses, dtype=np.float32).astype(np.float64), pix, obs, intr, m,
                         threads=threads, per_sample=per_sample)
        out["march"] = m
        return out

    def render(self, poses, pix, intr, threads=None):
        pix = np.asarray(pix, dtype=np.int32)
        obs = np.zeros((intr["height"], intr["width"], 3), dtype=np.float32)
        return self.render_loss_grad(poses, pix, obs, intr, threads)["rgb"]

    def build_occupancy(self, R: int, threshold: float, threads=None):
        words = np.zeros((R * R * R + 31) // 32, dtype=np.uint32)
        lib().orc_build_occupancy(self.ptr, R, threshold, _p(words), threads or n_threads_default())
        return words


# ---------------------------------------------------------------- free functions
def ray_f32(pose, intr, pix):
    pose = np.ascontiguousarray(pose, dtype=np.float32).reshape(12)
    o = np.zeros(3, np.float32)
    d = np.zeros(3, np.float32)
    it = intr_struct(intr)
    lib().orc_ray_f32(_p(pose), C.byref(it), int(pix), _p(o), _p(d))
    return o, d


def sh16(d):
    d = np.ascontiguousarray(d, dtype=np.float64)
    out = np.zeros(16)
    grad = np.zeros((16, 3))
    lib().orc_sh16(_p(d), _p(out), _p(grad))
    return out, grad


def composite(sigma, rgb, delta, bg=(0, 0, 0), t_stop=0.0):
    sigma = np.ascontiguousarray(sigma, dtype=np.float64)
    rgb = np.ascontiguousarray(rgb, dtype=np.float64).reshape(-1, 3)
    n = sigma.size
    bg = np.ascontiguousarray(bg, dtype=np.float64)
    Cc = np.zeros(3)
    trans = np.zeros(n + 1)
    weight = np.zeros(n + 1)
    used = np.zeros(1, np.int32)
    lib().orc_composite(n, _p(sigma), _p(rgb), delta, _p(bg), t_stop, _p(Cc), _p(trans),
                        _p(weight), _p(used))
    u = int(used[0])
    return Cc, trans[:u + 1], weight[:u], u


def composite_grad(sigma, rgb, delta, gC, bg=(0, 0, 0), t_stop=0.0):
    sigma = np.ascontiguousarray(sigma, dtype=np.float64)
    rgb = np.ascontiguousarray(rgb, dtype=np.float64).reshape(-1, 3)
    n = sigma.size
    bg = np.ascontiguousarray(bg, dtype=np.float64)
    gC = np.ascontiguousarray(gC, dtype=np.float64)
    gs = np.zeros(n)
    gr = np.zeros((n, 3))
    lib().orc_composite_grad(n, _p(sigma), _p(rgb), delta, _p(bg), t_stop, _p(gC), _p(gs), _p(gr))
    return gs, gr


def pixel_loss(loss_type, C, y, p):
    """(loss, d loss / d C, kink distance) of one channel."""
    g = np.zeros(1)
    k = np.zeros(1)
    v = lib().orc_pixel_loss(int(loss_type), float(C), float(y), float(p), _p(g), _p(k))
    return v, float(g[0]), float(k[0])


def exp_so3(w):
    w = np.ascontiguousarray(w, dtype=np.float64)
    R = np.zeros(9)
    lib().orc_exp_so3(_p(w), _p(R))
    return R.reshape(3, 3)


def step_momentum(poses, momentum, dpose, lr, beta):
    poses = np.array(poses, dtype=np.float32, copy=True)
    momentum = np.array(momentum, dtype=np.float32, copy=True)
    dpose = np.ascontiguousarray(dpose, dtype=np.float32)
    K = poses.shape[0]
    lib().orc_step_momentum(K, _p(poses), _p(momentum), _p(dpose), lr, beta)
    return poses, momentum


ADAM_STATE = 16  # floats per hypothesis: m[6], v[6], step count, 3 zeros


class _Adam(C.Structure):
    _fields_ = [("lr_rot", C.c_float), ("lr_trans", C.c_float), ("beta1", C.c_float),
                ("beta2", C.c_float), ("eps", C.c_float), ("decay_base", C.c_float),
                ("decay_steps", C.c_int32), ("staircase", C.c_int32),
                ("second_moment", C.c_int32), ("representation", C.c_int32)]


def step_adam(poses, state, dpose, step, lr_rot, lr_trans, beta1=0.9, beta2=0.999, eps=1e-8,
              decay_base=1.0, decay_steps=0, staircase=0, second_moment=0, representation=0):
    """Adam on SO(3) x T(3) (Sec. IV-A; setting of Sec. IV-D), or on the coupled se(3) twist
    (representation = 1); returns new (poses, state)."""
    poses = np.array(poses, dtype=np.float32, copy=True)
    state = np.array(state, dtype=np.float32, copy=True)
    dpose = np.ascontiguousarray(dpose, dtype=np.float32)
    K = poses.shape[0]
    assert state.shape == (K, ADAM_STATE) and dpose.shape == (K, 6)
    a = _Adam(lr_rot, lr_trans, beta1, beta2, eps, decay_base, decay_steps, staircase,
              second_moment, representation)
    lib().orc_step_adam(K, _p(poses), _p(state), _p(dpose), step, C.byref(a))
    return poses, state


def resample(poses, state, loss, keep_frac, sigma_rot, sigma_trans, seed, round_idx):
    """Monte Carlo resampling (Sec. IV-B); state is [K][state_dim] (or None);
    returns new (poses, state, rank)."""
    poses = np.array(poses, dtype=np.float32, copy=True)
    K = poses.shape[0]
    if state is None:
        state = np.zeros((K, 0), np.float32)
    state = np.array(state, dtype=np.float32, copy=True).reshape(K, -1)
    loss = np.ascontiguousarray(loss, dtype=np.float32)
    rank = np.zeros(K, np.int32)
    lib().orc_resample(K, _p(poses), _p(state), state.shape[1], _p(loss), keep_frac, sigma_rot,
                       sigma_trans, seed, round_idx, _p(rank))
    return poses, state, rank


def splitmix64_stream(seed: int, n: int):
    st = np.array([seed], dtype=np.uint64)
    return [int(lib().orc_splitmix64_next(_p(st))) for _ in range(n)]


def normals6(seed, round_idx, slot):
    n = np.zeros(6)
    lib().orc_normals6(seed, round_idx, slot, _p(n))
    return n
