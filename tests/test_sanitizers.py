"""The CPU oracle and the host side of the HIP library under AddressSanitizer
and UndefinedBehaviorSanitizer, on the CPU (no device code is sanitized):

* the oracle built by gcc with both sanitizers, driven through its Python
  binding over marching, shading with per-sample outputs, variant shading,
  the pose updates, resampling and the occupancy build;
* libpnerf's host pass built by hipcc with the sanitizers after -Xarch_host,
  driven by tests/sanitize/host_driver.c: batch planning, argument
  validation, and field creation up to its first device allocation."""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")


def _clean(out):
    return "AddressSanitizer" not in out and "runtime error:" not in out


def test_oracle_under_sanitizers(tmp_path):
    lib = tmp_path / "liboracle_san.so"
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                    "-fopenmp", "-fPIC", "-shared", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "oracle", "pnerf_oracle.c"), "-o", str(lib), "-lm"],
                   check=True)
    script = tmp_path / "drive.py"
    script.write_text(textwrap.dedent(f"""
        import math, sys
        sys.path.insert(0, {ROOT!r})
        import numpy as np
        from oracle import oracle as O
        from paper_2210_10108_amd import synth
        assert O.LIB == {str(lib)!r}
        w = synth.WORKLOADS["tiny32"]
        intr = synth.intrinsics(w)
        gt = synth.ground_truth_pose(w, 0)
        poses = synth.perturb_poses(gt, 3, 20, 0.1, 0)
        pix = synth.pixel_batch(0, 0, 3, 40, w.width, w.height)
        obs = np.random.default_rng(0).uniform(0, 1, (32, 32, 3)).astype(np.float32)
        for kw in [dict(), dict(sh_dir_grad=1, loss_type=6, loss_param=0.01),
                   dict(march_mode=1, step=math.sqrt(3) / 96, max_samples=300, t_stop=5e-2,
                        occ_res=16, density_bias=2.5, loss_type=1,
                        occ_bits=synth.occupancy_pattern("sphere", 16))]:
            of = O.OracleField(synth.field_spec(w, synth.make_field(w, 0), **kw))
            out = of.render_loss_grad(poses, pix, obs, intr, per_sample=True, threads=2)
            off, t, _, delta = out["march"]
            jobs = [(r // 40, pix.ravel()[r], off[r], off[r + 1] - off[r], delta[r],
                     int(out["stop"][r]) - 1 if out["stop"][r] > 1 else -1, (1, -1, 0), 3)
                    for r in range(120) if off[r + 1] > off[r]]
            of.shade_ray_jobs(poses, 40, obs, intr, t, np.array(jobs, dtype=O.RAY_JOB), 0.05,
                              threads=2)
            of.build_occupancy(8, 0.5, threads=2)
        mom = np.zeros((3, 6), np.float32)
        O.step_momentum(poses, mom, np.ones((3, 6), np.float32), 1e-2, 0.9)
        for rep in (0, 1):
            O.step_adam(poses, np.zeros((3, O.ADAM_STATE), np.float32),
                        np.ones((3, 6), np.float32), 5, 5e-3, 3e-3, decay_base=0.33,
                        decay_steps=256, representation=rep)
        O.resample(poses, mom, np.array([0.3, np.nan, 0.1], np.float32), 0.34, 0.1, 0.03, 7, 1)
        print("oracle driver done")
        """))
    env = dict(SAN_ENV, LD_PRELOAD=subprocess.run(["gcc", "-print-file-name=libasan.so"],
                                                  capture_output=True, text=True,
                                                  check=True).stdout.strip(),
               PNERF_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, str(script)], capture_output=True, text=True, env=env,
                       timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0 and "oracle driver done" in out and _clean(out), out[-4000:]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_library_host_code_under_sanitizers(tmp_path):
    src = os.path.join(ROOT, "paper_2210_10108_amd", "csrc")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
           "-fno-omit-frame-pointer"]
    procs, objs = [], []
    for name in ("api", "march", "encode", "mlp", "composite", "pose"):
        obj = tmp_path / f"{name}.o"
        objs.append(str(obj))
        procs.append(subprocess.Popen(
            [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Xclang",
             "-target-feature", "-Xclang", "-packed-fp32-ops", "-fno-gpu-rdc", *san, "-I",
             os.path.join(ROOT, "include"), "-c", os.path.join(src, f"{name}.hip"), "-o",
             str(obj)], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
    for p in procs:
        out, _ = p.communicate(timeout=900)
        assert p.returncode == 0, out[-3000:]
    lib = tmp_path / "libpnerf_san.so"
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *san, *objs, "-o",
                    str(lib)], check=True, capture_output=True)
    exe = tmp_path / "host_driver"
    subprocess.run([CLANG, "-g", "-fsanitize=address,undefined", "-I",
                    os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "sanitize", "host_driver.c"), f"-L{tmp_path}",
                    "-lpnerf_san", f"-Wl,-rpath,{tmp_path}", "-o", str(exe)], check=True)
    env = dict(SAN_ENV, HIP_VISIBLE_DEVICES="")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0 and "host driver done" in out and _clean(out), out[-4000:]
