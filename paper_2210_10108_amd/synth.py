"""Seeded synthetic workloads for the pose-inversion hot path.

This module only draws inputs: a frozen Instant-NGP-style field (hash table
and MLP weights), a ground-truth camera, perturbed pose hypotheses, pixel
batches and structured occupancy bitfields.  It holds none of the method's
arithmetic (no rendering, no gradients, no pose updates); both the HIP path
and the CPU oracle consume what it produces.

The paper (Sec. III, "Preliminaries" and "Approach") inverts a trained
Instant NGP model.  Trained weights and the NeRF-Synthetic / LLFF datasets are
not available, so the field is random with the sizes of the paper's setting,
and the observed image is rendered from the field itself at a seeded
ground-truth pose (done by the caller, not here).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
from scipy.spatial.transform import Rotation

HIDDEN = 64          # width of every hidden layer
DENSITY_OUT = 16     # density-MLP outputs: sigma logit + 15 features
COLOR_IN = 32        # 15 features + 16 SH coefficients + 1 zero pad


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic pose-inversion workload (field, camera, batch, schedule)."""
    name: str
    n_levels: int
    n_features: int
    log2_table: int
    n_min: int
    n_max: int
    param_dtype: str            # "f32" or "f16" (table and MLP weights)
    aabb_min: tuple
    aabb_max: tuple
    march_mode: int             # 0: uniform samples in the AABB, 1: lattice
    n_uniform: int
    step: float
    max_samples: int
    t_stop: float
    occ_res: int                # 0: no occupancy grid
    occ_threshold: float
    width: int
    height: int
    focal: float
    cx: float
    cy: float
    K: int                      # pose hypotheses
    P: int                      # pixels (rays) per hypothesis per iteration
    max_rot_deg: float
    max_trans: float
    iters: int
    lr: float = 1e-2
    beta: float = 0.9
    huber_delta: float = 0.1
    resample_every: int = 0
    keep_frac: float = 1.0
    resample_sigma_rot_deg: float = 5.0
    resample_sigma_trans: float = 0.03
    cam_radius: float = 2.5
    density: str = "random"     # "random", or "bump": an object in empty space

    @property
    def table_size(self) -> int:
        return 1 << self.log2_table

    @property
    def density_in(self) -> int:
        return self.n_levels * self.n_features

    @property
    def n_rays(self) -> int:
        return self.K * self.P

    def max_samples_per_ray(self) -> int:
        """Upper bound on kept samples per ray (used to size buffers)."""
        if self.march_mode == 0:
            return self.n_uniform
        ext = [b - a for a, b in zip(self.aabb_min, self.aabb_max)]
        diag = math.sqrt(sum(e * e for e in ext))
        return min(self.max_samples, int(math.ceil(diag / self.step)) + 1)


_UNIT = ((-0.5, -0.5, -0.5), (0.5, 0.5, 0.5))

WORKLOADS = {
    # tiny smoke case: the oracle finishes it in well under a second
    "tiny32": Workload("tiny32", 4, 2, 12, 16, 64, "f32", *_UNIT, 0, 32, 0.0, 32, 0.0,
                     0, 0.01, 32, 32, 40.0, 16.0, 16.0, 4, 256, 20.0, 0.15, 10),
    # Instant-NGP-sized field, 800x800 observation, uniform samples
    "ngp800_uniform": Workload("ngp800_uniform", 16, 2, 19, 16, 2048, "f32", *_UNIT, 0, 128, 0.0, 128, 0.0,
                       0, 0.01, 800, 800, 1111.0, 400.0, 400.0, 16, 1024, 30.0, 0.2, 300),
    # as ngp800 plus a 128^3 occupancy grid and lattice marching with early stop
    "ngp800_occ128": Workload("ngp800_occ128", 16, 2, 19, 16, 2048, "f32", *_UNIT, 1, 0,
                           math.sqrt(3.0) / 1024.0, 1024, 1e-4, 128, 0.01,
                           800, 800, 1111.0, 400.0, 400.0, 64, 4096, 30.0, 0.2, 300),
    # real-camera shape, fp16 storage, Monte Carlo resampling
    "cam640_f16_occ128": Workload("cam640_f16_occ128", 16, 2, 19, 16, 2048, "f16", *_UNIT, 1, 0,
                           math.sqrt(3.0) / 1024.0, 1024, 1e-4, 128, 0.01,
                           640, 480, 572.0, 325.3, 242.0, 256, 2048, 45.0, 0.3, 300,
                           resample_every=50, keep_frac=0.25),
    # large scene: [-2,2]^3, 2^21 table, 256^3 occupancy, up to 2048 samples per ray
    "large4m_occ256": Workload("large4m_occ256", 16, 2, 21, 16, 8192, "f32", (-2.0, -2.0, -2.0), (2.0, 2.0, 2.0),
                      1, 0, 4.0 * math.sqrt(3.0) / 2048.0, 2048, 1e-4, 256, 0.01,
                      800, 800, 1111.0, 400.0, 400.0, 1024, 512, 60.0, 0.5, 1000,
                      resample_every=100, keep_frac=0.10),
    # structured density: one object (a smooth density bump) in empty space, so
    # that occupancy skipping and early ray termination take effect, as they
    # do on the paper's object scenes
    "ngp800_bump_occ128": Workload("ngp800_bump_occ128", 16, 2, 19, 16, 2048, "f32", *_UNIT, 1, 0,
                                   math.sqrt(3.0) / 1024.0, 1024, 1e-4, 128, 0.01,
                                   800, 800, 1111.0, 400.0, 400.0, 64, 4096, 30.0, 0.2, 300,
                                   density="bump"),
    "tiny_bump": Workload("tiny_bump", 4, 2, 13, 16, 64, "f32", *_UNIT, 1, 0,
                          math.sqrt(3.0) / 128.0, 256, 1e-4, 32, 0.01,
                          32, 32, 40.0, 16.0, 16.0, 4, 256, 20.0, 0.15, 10, density="bump"),
}
ORDER = ["tiny32", "ngp800_uniform", "ngp800_occ128", "cam640_f16_occ128", "large4m_occ256",
         "ngp800_bump_occ128", "tiny_bump"]


def level_resolutions(n_levels: int, n_min: int, n_max: int) -> np.ndarray:
    """Per-level grid resolution N_l of a geometric multiresolution ladder.

    N_l = floor(N_min * b**l) with b = exp((ln N_max - ln N_min)/(L-1)); a
    1e-9 guard keeps exact powers (64, 128, 1024, 8192) from flooring one low.
    """
    if n_levels == 1:
        return np.array([n_min], dtype=np.int32)
    b = math.exp((math.log(n_max) - math.log(n_min)) / (n_levels - 1))
    return np.array([int(math.floor(n_min * b ** l + 1e-9)) for l in range(n_levels)],
                    dtype=np.int32)


def _glorot(rng: np.random.Generator, fan_in: int, fan_out: int) -> np.ndarray:
    a = math.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-a, a, size=(fan_in, fan_out)).astype(np.float32)


@dataclasses.dataclass
class FieldArrays:
    """Host copies of a frozen field; weights are [in][out] (out = in @ W)."""
    level_res: np.ndarray       # int32 [L]
    table: np.ndarray           # [L][T][F], float32 or float16
    w_density1: np.ndarray      # [L*F][64]
    w_density2: np.ndarray      # [64][16]
    w_color1: np.ndarray        # [32][64]
    w_color2: np.ndarray        # [64][64]
    w_color3: np.ndarray        # [64][3]
    density_bias: float = -1.0


# Density bump of the "bump" fields: centre and radius in the unit box,
# sigma = exp(BUMP_GAIN * relu(feature) - BUMP_OFFSET) with feature 0 of level 0
# holding exp(-|p - c|^2 / r^2) at the level's vertices.
BUMP_CENTER = (0.0, 0.0, 0.0)
BUMP_RADIUS = 0.3
BUMP_GAIN = 12.0
BUMP_OFFSET = 6.0


def make_field(w: Workload, seed: int) -> FieldArrays:
    """Draw the frozen field of workload `w` from `seed`.

    Stream order: table, W_d1, W_d2, W_c1, W_c2, W_c3.  Table entries are
    U(-1, 1); weights are Glorot-uniform on the padded shapes.

    density = "bump" then shapes the density into one object in empty space:
    feature 0 of level 0 (a dense level: vertex (i, j, k) at entry
    i + j n1 + k n1^2) takes exp(-|p - c|^2 / r^2) at the vertex positions, the
    first density-layer unit reads only that feature, the sigma logit reads
    only that unit (gain BUMP_GAIN), and the density bias is -BUMP_OFFSET.  The
    other weights, the other features and the colour stay random.
    """
    rng = np.random.default_rng(seed)
    L, F, T = w.n_levels, w.n_features, w.table_size
    table = rng.uniform(-1.0, 1.0, size=(L, T, F)).astype(np.float32)
    wd1 = _glorot(rng, w.density_in, HIDDEN)
    wd2 = _glorot(rng, HIDDEN, DENSITY_OUT)
    wc1 = _glorot(rng, COLOR_IN, HIDDEN)
    wc2 = _glorot(rng, HIDDEN, HIDDEN)
    wc3 = _glorot(rng, HIDDEN, 3)
    density_bias = -1.0
    if w.density == "bump":
        N = int(level_resolutions(L, w.n_min, w.n_max)[0])
        n1 = N + 1
        if n1 ** 3 > T:
            raise ValueError("the bump needs a dense level 0: (N_min + 1)^3 <= T")
        g = np.arange(n1, dtype=np.float64) / N
        lo = np.asarray(w.aabb_min, np.float64)
        ext = np.asarray(w.aabb_max, np.float64) - lo
        x = lo[0] + g * ext[0] - BUMP_CENTER[0]
        y = lo[1] + g * ext[1] - BUMP_CENTER[1]
        z = lo[2] + g * ext[2] - BUMP_CENTER[2]
        d2 = x[None, None, :] ** 2 + y[None, :, None] ** 2 + z[:, None, None] ** 2  # [k][j][i]
        table[0, :n1 ** 3, 0] = np.exp(-d2 / BUMP_RADIUS ** 2).reshape(-1).astype(np.float32)
        wd1[:, 0] = 0.0
        wd1[0, 0] = 1.0
        wd2[:, 0] = 0.0
        wd2[0, 0] = BUMP_GAIN
        density_bias = -BUMP_OFFSET
    if w.param_dtype == "f16":
        cast = lambda a: a.astype(np.float16)
    else:
        cast = lambda a: a
    return FieldArrays(level_resolutions(L, w.n_min, w.n_max), cast(table), cast(wd1),
                       cast(wd2), cast(wc1), cast(wc2), cast(wc3), density_bias)


def look_at_pose(cam_pos: np.ndarray, target=(0.0, 0.0, 0.0)) -> np.ndarray:
    """Camera-to-world [R | o] (3x4, float32), OpenCV axes: x right, y down, z forward.

    World up is +z, or +y when the viewing direction is nearly vertical.
    """
    o = np.asarray(cam_pos, dtype=np.float64)
    f = np.asarray(target, dtype=np.float64) - o
    f /= np.linalg.norm(f)
    up = np.array([0.0, 0.0, 1.0])
    if abs(f @ up) > 0.99:
        up = np.array([0.0, 1.0, 0.0])
    right = np.cross(f, up)
    right /= np.linalg.norm(right)
    down = np.cross(f, right)
    pose = np.zeros((3, 4), dtype=np.float64)
    pose[:, 0], pose[:, 1], pose[:, 2], pose[:, 3] = right, down, f, o
    return pose.astype(np.float32)


def _unit_vectors(rng: np.random.Generator, n: int) -> np.ndarray:
    v = rng.normal(size=(n, 3))
    return v / np.linalg.norm(v, axis=1, keepdims=True)


def ground_truth_pose(w: Workload, seed: int) -> np.ndarray:
    """Seeded ground-truth camera at radius `cam_radius` looking at the origin."""
    rng = np.random.default_rng([seed, 1])
    u = _unit_vectors(rng, 1)[0]
    return look_at_pose(w.cam_radius * u)


def perturb_poses(gt: np.ndarray, K: int, max_rot_deg: float, max_trans: float,
                  seed: int) -> np.ndarray:
    """K hypotheses around `gt`: rotation by U(0, max) degrees about a random axis
    (applied in the world frame about the camera centre) plus a translation of
    U(0, max) length in a random direction.  Returns float32 [K][3][4]."""
    rng = np.random.default_rng([seed, 2])
    axes = _unit_vectors(rng, K)
    ang = np.deg2rad(rng.uniform(0.0, max_rot_deg, size=K))
    tdir = _unit_vectors(rng, K)
    tmag = rng.uniform(0.0, max_trans, size=K)
    Rp = Rotation.from_rotvec(axes * ang[:, None]).as_matrix()
    out = np.empty((K, 3, 4), dtype=np.float64)
    out[:, :, :3] = Rp @ gt[:, :3].astype(np.float64)
    out[:, :, 3] = gt[:, 3].astype(np.float64) + tdir * tmag[:, None]
    return out.astype(np.float32)


def pixel_batch(seed: int, it: int, K: int, P: int, width: int, height: int) -> np.ndarray:
    """Pixel ids [K][P] (int32, row-major v*W+u), uniform with replacement,
    from a Philox counter stream keyed on (seed, iteration)."""
    bitgen = np.random.Philox(key=np.array([seed & 0xFFFFFFFFFFFFFFFF, it], dtype=np.uint64))
    rng = np.random.Generator(bitgen)
    return rng.integers(0, width * height, size=(K, P), dtype=np.int32)


def intrinsics(w: Workload):
    return dict(width=w.width, height=w.height, fx=w.focal, fy=w.focal, cx=w.cx, cy=w.cy)


# ---------------------------------------------------------------- occupancy
def pack_bits(occ: np.ndarray) -> np.ndarray:
    """Pack a boolean [R][R][R] grid indexed [z][y][x] into LSB-first uint32
    words of the linear index x + R*(y + R*z)."""
    flat = occ.reshape(-1).astype(np.uint8)
    n = flat.size
    words = np.zeros((n + 31) // 32, dtype=np.uint32)
    idx = np.nonzero(flat)[0]
    np.bitwise_or.at(words, idx >> 5, (np.uint32(1) << (idx & 31).astype(np.uint32)))
    return words


def unpack_bits(words: np.ndarray, R: int) -> np.ndarray:
    n = R * R * R
    idx = np.arange(n)
    bits = (words[idx >> 5] >> (idx & 31).astype(np.uint32)) & 1
    return bits.astype(bool).reshape(R, R, R)


def occupancy_pattern(kind: str, R: int, seed: int = 0) -> np.ndarray:
    """Structured occupancy grids for stress cases: 'full', 'empty', 'sphere',
    'checker' (3-D checkerboard of 4^3 blocks) or 'random' (50 %)."""
    z, y, x = np.meshgrid(np.arange(R), np.arange(R), np.arange(R), indexing="ij")
    if kind == "full":
        occ = np.ones((R, R, R), bool)
    elif kind == "empty":
        occ = np.zeros((R, R, R), bool)
    elif kind == "sphere":
        c = (R - 1) / 2.0
        occ = (x - c) ** 2 + (y - c) ** 2 + (z - c) ** 2 <= (0.35 * R) ** 2
    elif kind == "checker":
        occ = ((x // 4 + y // 4 + z // 4) % 2) == 0
    elif kind == "random":
        occ = np.random.default_rng([seed, 3]).random((R, R, R)) < 0.5
    else:
        raise ValueError(kind)
    return pack_bits(occ)


# ------------------------------------------------------------- field spec
@dataclasses.dataclass
class FieldSpec:
    """Everything that defines a frozen field and how its rays are sampled.

    Consumed unchanged by the HIP binding and by the CPU oracle.  Weight
    matrices are [in][out]; the table is [L][T][F]; `occ_bits` is None (no grid,
    or build it on the device when `occ_res` > 0) or packed LSB-first words."""
    n_levels: int
    n_features: int
    log2_table: int
    level_res: np.ndarray
    dense_coarse_levels: int
    param_dtype: str
    table: np.ndarray
    w_density1: np.ndarray
    w_density2: np.ndarray
    w_color1: np.ndarray
    w_color2: np.ndarray
    w_color3: np.ndarray
    density_bias: float
    aabb_min: tuple
    aabb_max: tuple
    march_mode: int
    n_uniform: int
    step: float
    max_samples: int
    t_stop: float
    occ_res: int
    occ_bits: np.ndarray | None
    occ_threshold: float
    background: tuple = (0.0, 0.0, 0.0)
    loss_type: int = 0
    loss_param: float = 0.1
    sh_dir_grad: int = 0

    @property
    def table_size(self) -> int:
        return 1 << self.log2_table


def field_spec(w: Workload, fa: FieldArrays, occ_bits: np.ndarray | None = None,
               **overrides) -> FieldSpec:
    """FieldSpec of workload `w` with field `fa`; keyword overrides replace fields."""
    spec = FieldSpec(
        n_levels=w.n_levels, n_features=w.n_features, log2_table=w.log2_table,
        level_res=fa.level_res, dense_coarse_levels=1, param_dtype=w.param_dtype,
        table=fa.table, w_density1=fa.w_density1, w_density2=fa.w_density2,
        w_color1=fa.w_color1, w_color2=fa.w_color2, w_color3=fa.w_color3,
        density_bias=fa.density_bias, aabb_min=tuple(w.aabb_min), aabb_max=tuple(w.aabb_max),
        march_mode=w.march_mode, n_uniform=w.n_uniform, step=w.step,
        max_samples=w.max_samples, t_stop=w.t_stop, occ_res=w.occ_res, occ_bits=occ_bits,
        occ_threshold=w.occ_threshold, loss_param=w.huber_delta)
    return dataclasses.replace(spec, **overrides)
