"""Python binding of libpnerf.so (C ABI in include/pnerf.h).

Argument marshalling only: every step of the hot path runs in the HIP library.
Device arrays are torch tensors on a ROCm device; torch provides device memory
and the stream.  Importing this module does not need a GPU; creating a field
or calling an entry point does, and raises if the library is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpnerf.so")

OK, ERR_INVALID_ARG, ERR_OUT_OF_MEMORY, ERR_DEVICE, ERR_CAPACITY, ERR_NOT_SUPPORTED = range(6)


class PnerfError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"pnerf status {status}: {msg}")
        self.status = status


class Intrinsics(C.Structure):
    _fields_ = [("width", C.c_int32), ("height", C.c_int32), ("fx", C.c_float),
                ("fy", C.c_float), ("cx", C.c_float), ("cy", C.c_float)]


class FieldParams(C.Structure):
    _fields_ = [("n_levels", C.c_int32), ("n_features", C.c_int32),
                ("log2_table_size", C.c_int32), ("level_res", C.c_void_p),
                ("dense_coarse_levels", C.c_int32), ("param_dtype", C.c_int32),
                ("table", C.c_void_p), ("w_density1", C.c_void_p), ("w_density2", C.c_void_p),
                ("w_color1", C.c_void_p), ("w_color2", C.c_void_p), ("w_color3", C.c_void_p),
                ("density_bias", C.c_float), ("aabb_min", C.c_float * 3),
                ("aabb_max", C.c_float * 3), ("march_mode", C.c_int32),
                ("n_uniform", C.c_int32), ("step", C.c_float), ("max_samples", C.c_int32),
                ("t_stop", C.c_float), ("occ_res", C.c_int32), ("occ_bits", C.c_void_p),
                ("occ_threshold", C.c_float), ("background", C.c_float * 3),
                ("loss_type", C.c_int32), ("loss_param", C.c_float),
                ("sh_dir_grad", C.c_int32), ("max_workspace_bytes", C.c_int64),
                ("overlap_chunks", C.c_int32), ("backward", C.c_int32),
                ("mlp_precision", C.c_int32)]


_lib = None

# name -> (restype, argtypes); every function declared in include/pnerf.h
_SIGS = {
    "pnerf_create_field": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p]),
    "pnerf_destroy_field": (None, [C.c_void_p]),
    "pnerf_render_loss_grad": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                                         C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                         C.c_void_p]),
    "pnerf_step_momentum": (C.c_int, [C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_float,
                                      C.c_float, C.c_void_p]),
    "pnerf_step_adam": (C.c_int, [C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32,
                                  C.c_void_p, C.c_void_p]),
    "pnerf_resample_hypotheses": (C.c_int, [C.c_int32, C.c_void_p, C.c_void_p, C.c_int32,
                                            C.c_void_p, C.c_float, C.c_float, C.c_float,
                                            C.c_uint64, C.c_uint32, C.c_void_p]),
    "pnerf_render": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                               C.c_void_p, C.c_void_p, C.c_void_p]),
    "pnerf_march": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                              C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64,
                              C.c_void_p]),
    "pnerf_field_inspect": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_int64,
                                      C.c_void_p]),
    "pnerf_field_occupancy": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p]),
    "pnerf_field_last_sample_count": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p]),
    "pnerf_field_set_profiling": (C.c_int, [C.c_void_p, C.c_int32]),
    "pnerf_field_profile_read": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                           C.c_void_p]),
    "pnerf_resample_hypotheses_noalloc": (C.c_int, [C.c_int32, C.c_void_p, C.c_void_p,
                                                    C.c_int32, C.c_void_p, C.c_float, C.c_float,
                                                    C.c_float, C.c_uint64, C.c_uint32,
                                                    C.c_void_p]),
    "pnerf_plan_counted_batch": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_void_p]),
    "pnerf_plan_chunks": (C.c_int, [C.c_void_p, C.c_int32, C.c_int64, C.c_int64, C.c_void_p,
                                    C.c_void_p, C.c_void_p]),
    "pnerf_last_error": (C.c_char_p, []),
}


def lib() -> C.CDLL:
    """Load libpnerf.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        # torch's HIP runtime must be the one in the process: import it first so
        # that libpnerf.so binds to the already-loaded libamdhip64.so.7
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python paper_2210_10108_amd/build.py` (or __graft_entry__.build())")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != OK:
        raise PnerfError(status, lib().pnerf_last_error().decode())


def _stream(stream=None) -> C.c_void_p:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _dev(t, dtype, shape=None, name="tensor"):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return C.c_void_p(t.data_ptr())


def intrinsics(d) -> Intrinsics:
    return Intrinsics(int(d["width"]), int(d["height"]), float(d["fx"]), float(d["fy"]),
                      float(d["cx"]), float(d["cy"]))


class Field:
    """A frozen field on the current device (wraps pnerf_create_field).

    spec: a synth.FieldSpec (table, weights, marching, loss).  The keyword
    arguments are the pnerf_field_params fields of the same names:
    max_workspace_bytes (0: the library's default budget), overlap_chunks,
    backward (0 separate kernels, 1 fused per-ray kernel, 2 fused keeping the
    per-sample intermediates) and mlp_precision (0 split-bf16, 1 fp16 MFMA)."""

    def __init__(self, spec, stream=None, max_workspace_bytes: int = 0, overlap_chunks: int = 0,
                 backward: int = 0, mlp_precision: int = 0):
        self._h = C.c_void_p()
        f16 = spec.param_dtype == "f16"
        npdt = np.float16 if f16 else np.float32
        keep = self._keep = []

        def arr(a, dt):
            a = np.ascontiguousarray(np.asarray(a), dtype=dt)
            keep.append(a)
            return a.ctypes.data_as(C.c_void_p)

        p = FieldParams()
        p.n_levels, p.n_features, p.log2_table_size = spec.n_levels, spec.n_features, spec.log2_table
        p.level_res = arr(spec.level_res, np.int32)
        p.dense_coarse_levels = spec.dense_coarse_levels
        p.param_dtype = 1 if f16 else 0
        p.table = arr(spec.table, npdt)
        p.w_density1 = arr(spec.w_density1, npdt)
        p.w_density2 = arr(spec.w_density2, npdt)
        p.w_color1 = arr(spec.w_color1, npdt)
        p.w_color2 = arr(spec.w_color2, npdt)
        p.w_color3 = arr(spec.w_color3, npdt)
        p.density_bias = spec.density_bias
        p.aabb_min = (C.c_float * 3)(*spec.aabb_min)
        p.aabb_max = (C.c_float * 3)(*spec.aabb_max)
        p.march_mode, p.n_uniform, p.step = spec.march_mode, spec.n_uniform, spec.step
        p.max_samples, p.t_stop = spec.max_samples, spec.t_stop
        p.occ_res = spec.occ_res
        p.occ_bits = None if spec.occ_bits is None else arr(spec.occ_bits, np.uint32)
        p.occ_threshold = spec.occ_threshold
        p.background = (C.c_float * 3)(*spec.background)
        p.loss_type, p.loss_param, p.sh_dir_grad = spec.loss_type, spec.loss_param, spec.sh_dir_grad
        p.max_workspace_bytes = int(max_workspace_bytes)
        p.overlap_chunks = int(overlap_chunks)
        p.backward = int(backward)
        p.mlp_precision = int(mlp_precision)
        self.spec = spec
        self.occ_res = spec.occ_res
        _check(lib().pnerf_create_field(C.byref(p), _stream(stream), C.byref(self._h)))
        self._keep = None  # create_field deep-copied everything

    def close(self):
        if self._h:
            lib().pnerf_destroy_field(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- calls
    def render_loss_grad(self, poses, pixel_ids, observed, intr, loss=None, dpose=None,
                         stream=None):
        import torch
        K, P = pixel_ids.shape
        if loss is None:
            loss = torch.empty(K, dtype=torch.float32, device=poses.device)
        if dpose is None:
            dpose = torch.empty(K, 6, dtype=torch.float32, device=poses.device)
        it = intrinsics(intr)
        _check(lib().pnerf_render_loss_grad(
            self._h, K, _dev(poses, torch.float32, (K, 3, 4), "poses"), P,
            _dev(pixel_ids, torch.int32, (K, P), "pixel_ids"),
            _dev(observed, torch.float32, (it.height, it.width, 3), "observed"), C.byref(it),
            _dev(loss, torch.float32, (K,), "loss"), _dev(dpose, torch.float32, (K, 6), "dpose"),
            _stream(stream)))
        return loss, dpose

    def render(self, poses, pixel_ids, intr, rgb=None, stream=None):
        import torch
        K, P = pixel_ids.shape
        if rgb is None:
            rgb = torch.empty(K, P, 3, dtype=torch.float32, device=poses.device)
        it = intrinsics(intr)
        _check(lib().pnerf_render(
            self._h, K, _dev(poses, torch.float32, (K, 3, 4), "poses"), P,
            _dev(pixel_ids, torch.int32, (K, P), "pixel_ids"), C.byref(it),
            _dev(rgb, torch.float32, (K, P, 3), "rgb"), _stream(stream)))
        return rgb

    def march(self, poses, pixel_ids, intr, capacity: int, stream=None):
        """Returns (ray_offset int64 [K*P+1], t [capacity], lattice_j [capacity])."""
        import torch
        K, P = pixel_ids.shape
        dev = poses.device
        off = torch.empty(K * P + 1, dtype=torch.int64, device=dev)
        cap = max(int(capacity), 1)
        t = torch.zeros(cap, dtype=torch.float32, device=dev)
        j = torch.zeros(cap, dtype=torch.int32, device=dev)
        it = intrinsics(intr)
        _check(lib().pnerf_march(
            self._h, K, _dev(poses, torch.float32, (K, 3, 4), "poses"), P,
            _dev(pixel_ids, torch.int32, (K, P), "pixel_ids"), C.byref(it),
            _dev(off, torch.int64), _dev(t, torch.float32), _dev(j, torch.int32), int(capacity),
            _stream(stream)))
        return off, t, j

    def inspect(self, what: int, n: int, stream=None):
        """Per-sample intermediates of the last call (see pnerf_field_inspect)."""
        import torch
        width = {0: 1, 1: 1, 2: 3, 3: 6}[what]
        dst = torch.zeros(max(n, 1) * width, dtype=torch.float32, device="cuda")
        _check(lib().pnerf_field_inspect(self._h, what, _dev(dst, torch.float32), n,
                                         _stream(stream)))
        return dst[: n * width].reshape(n, width) if width > 1 else dst[:n]

    def occupancy(self, stream=None) -> np.ndarray:
        R = self.occ_res
        words = np.zeros((R * R * R + 31) // 32, dtype=np.uint32)
        _check(lib().pnerf_field_occupancy(self._h, words.ctypes.data_as(C.c_void_p),
                                           _stream(stream)))
        return words

    def last_sample_count(self, stream=None) -> int:
        n = C.c_int64()
        _check(lib().pnerf_field_last_sample_count(self._h, C.byref(n), _stream(stream)))
        return n.value

    def set_profiling(self, enable: bool):
        _check(lib().pnerf_field_set_profiling(self._h, 1 if enable else 0))

    def profile(self):
        """[(kernel name, launches, total ms)] since profiling was enabled."""
        out, i = [], 0
        while True:
            name = C.c_char_p()
            n = C.c_int64()
            ms = C.c_double()
            st = lib().pnerf_field_profile_read(self._h, i, C.byref(name), C.byref(n), C.byref(ms))
            if st != OK:
                break
            out.append((name.value.decode(), n.value, ms.value))
            i += 1
        return out


def step_momentum(poses, momentum, dpose, lr: float, beta: float, stream=None):
    import torch
    K = poses.shape[0]
    _check(lib().pnerf_step_momentum(
        K, _dev(poses, torch.float32, (K, 3, 4), "poses"),
        _dev(momentum, torch.float32, (K, 6), "momentum"),
        _dev(dpose, torch.float32, (K, 6), "dpose"), lr, beta, _stream(stream)))


ADAM_STATE = 16  # floats of Adam state per hypothesis (PNERF_ADAM_STATE)


class AdamParams(C.Structure):
    """pnerf_adam_params; the defaults are the setting of Sec. IV-D."""
    _fields_ = [("lr_rot", C.c_float), ("lr_trans", C.c_float), ("beta1", C.c_float),
                ("beta2", C.c_float), ("eps", C.c_float), ("decay_base", C.c_float),
                ("decay_steps", C.c_int32), ("staircase", C.c_int32),
                ("second_moment", C.c_int32), ("representation", C.c_int32)]

    def __init__(self, lr_rot=5e-3, lr_trans=3e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                 decay_base=0.33, decay_steps=256, staircase=0, second_moment=0,
                 representation=0):
        super().__init__(lr_rot, lr_trans, beta1, beta2, eps, decay_base, decay_steps,
                         staircase, second_moment, representation)


def step_adam(poses, state, dpose, step: int, params: AdamParams, stream=None):
    import torch
    K = poses.shape[0]
    _check(lib().pnerf_step_adam(
        K, _dev(poses, torch.float32, (K, 3, 4), "poses"),
        _dev(state, torch.float32, (K, ADAM_STATE), "state"),
        _dev(dpose, torch.float32, (K, 6), "dpose"), step, C.byref(params), _stream(stream)))


def resample_hypotheses(poses, state, loss, keep_frac: float, sigma_rot: float,
                        sigma_trans: float, seed: int, round_idx: int, stream=None):
    """state: the optimiser state [K][D] (momentum D = 6, Adam D = ADAM_STATE)
    or None; redrawn rows restart at 0."""
    import torch
    K = poses.shape[0]
    dim = 0 if state is None else int(state.shape[1])
    _check(lib().pnerf_resample_hypotheses(
        K, _dev(poses, torch.float32, (K, 3, 4), "poses"),
        None if state is None else _dev(state, torch.float32, (K, dim), "state"), dim,
        _dev(loss, torch.float32, (K,), "loss"), keep_frac, sigma_rot, sigma_trans,
        seed & 0xFFFFFFFFFFFFFFFF, round_idx, _stream(stream)))


def resample_hypotheses_noalloc(poses, state, loss, keep_frac: float, sigma_rot: float,
                                sigma_trans: float, seed: int, round_idx: int, stream=None):
    """pnerf_resample_hypotheses_noalloc: resample_hypotheses without any
    allocation (static ranking scratch per GPU, K <= 65535)."""
    import torch
    K = poses.shape[0]
    dim = 0 if state is None else int(state.shape[1])
    _check(lib().pnerf_resample_hypotheses_noalloc(
        K, _dev(poses, torch.float32, (K, 3, 4), "poses"),
        None if state is None else _dev(state, torch.float32, (K, dim), "state"), dim,
        _dev(loss, torch.float32, (K,), "loss"), keep_frac, sigma_rot, sigma_trans,
        seed & 0xFFFFFFFFFFFFFFFF, round_idx, _stream(stream)))


def plan_counted_batch(K: int, P: int, max_per_ray: int) -> int:
    """Hypotheses per counted batch (pnerf_plan_counted_batch; host only)."""
    n = C.c_int32()
    _check(lib().pnerf_plan_counted_batch(K, P, max_per_ray, C.byref(n)))
    return n.value


def plan_chunks(hyp_samples, capacity: int, goal: int):
    """Chunks of whole hypotheses (pnerf_plan_chunks; host only): returns the
    cut points [c + 1] and the samples of every chunk [c]."""
    import numpy as np
    h = np.ascontiguousarray(hyp_samples, dtype=np.int32)
    n = len(h)
    cut = np.zeros(n + 1, np.int32)
    sums = np.zeros(max(n, 1), np.int64)
    c = C.c_int32()
    _check(lib().pnerf_plan_chunks(h.ctypes.data_as(C.c_void_p), n, capacity, goal,
                                   cut.ctypes.data_as(C.c_void_p),
                                   sums.ctypes.data_as(C.c_void_p), C.byref(c)))
    return cut[:c.value + 1].copy(), sums[:c.value].copy()
