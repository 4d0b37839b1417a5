"""Register budgets of the hot kernels, from the compiler's resource remarks
(host-side compile for gfx950, no GPU): a kernel that spills to scratch or
drops below its intended occupancy runs several times slower without any
change in its results, so parity tests cannot catch it."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2210_10108_amd import build

# kernel (mangled-name fragment) -> minimum waves per SIMD
BUDGET = {
    "encode.hip": {"k_encodeILb0ELb1E": 7},
    # <levels per lane group, (SH direction path,) (keep,) fp16>
    "mlp.hip": {"k_mlp_fwdILi4ELb1ELb0E": 8, "k_mlp_bwdILi4ELb0ELb0E": 7,
                "k_mlp_bwdILi4ELb1ELb0E": 6, "k_ray_bwdILi4ELb0ELb0ELb0E": 4,
                "k_mlp_fwdILi4ELb1ELb1E": 8, "k_mlp_bwdILi4ELb0ELb1E": 8,
                "k_mlp_bwdILi4ELb1ELb1E": 6},
}


def remarks(src, tmp_path):
    cmd = [build.HIPCC, *build.FLAGS, "-Rpass-analysis=kernel-resource-usage", "-c",
           os.path.join(build.CSRC, src), "-o", str(tmp_path / "k.o")]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    out, name = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            out[name] = {}
            continue
        m = re.search(r"remark:\s+(ScratchSize \[bytes/lane\]|Occupancy \[waves/SIMD\]): (\d+)", line)
        if m and name:
            out[name][m.group(1).split()[0]] = int(m.group(2))
    return out


@pytest.mark.skipif(not shutil.which(build.HIPCC) and not os.path.exists(build.HIPCC),
                    reason="hipcc not installed")
@pytest.mark.parametrize("src", sorted(BUDGET))
def test_hot_kernels_do_not_spill(src, tmp_path):
    got = remarks(src, tmp_path)
    for frag, min_waves in BUDGET[src].items():
        hits = [n for n in got if frag in n]
        assert hits, (src, frag, sorted(got))
        for n in hits:
            assert got[n].get("ScratchSize") == 0, (n, got[n])
            assert got[n].get("Occupancy", 0) >= min_waves, (n, got[n])


# ------------------------------------------------ MFMA results across branches
def _vregs(spec):
    m = re.match(r"v\[(\d+):(\d+)\]", spec)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", spec)
    return {int(m.group(1))} if m else set()


def unpadded_mfma_reads_after_branches(asm):
    """Conditional branches taken within 6 instructions of an MFMA whose target
    reads that MFMA's destination with a vector instruction before any s_nop.
    The toolchain pads an MFMA result's first vector read with wait states on
    the fall-through path but, as measured, not always on the taken edge of a
    branch: a capped build of the backward network kernel whose join read the
    colour layer's accumulators two instructions after their MFMA gave wrong
    forces, and 16 wait states at the join fixed it."""
    L = asm.splitlines()
    labels = {l.split(":")[0]: i for i, l in enumerate(L) if re.match(r"^\.LBB\w+:", l)}
    found = []
    for i, l in enumerate(L):
        m = re.search(r"s_cbranch_\w+ (\.LBB\w+)", l)
        if not m:
            continue
        dst = set()
        for x in L[max(0, i - 6):i]:
            mm = re.search(r"v_mfma\w* (v\[\d+:\d+\])", x)
            if mm:
                dst |= _vregs(mm.group(1))
        if not dst:
            continue
        for x in L[labels[m.group(1)] + 1:labels[m.group(1)] + 8]:
            x = x.strip()
            if not x or x.startswith((";", "s_nop")):
                break
            if x.startswith("v_") and not x.startswith("v_mfma"):
                ops = re.findall(r"v\[\d+:\d+\]|v\d+\b", x.split(None, 1)[1] if " " in x else "")
                if any(_vregs(o) & dst for o in ops[1:]):
                    found.append((i, l.strip(), x))
    return found


@pytest.mark.skipif(not shutil.which(build.HIPCC) and not os.path.exists(build.HIPCC),
                    reason="hipcc not installed")
@pytest.mark.parametrize("src", ["mlp.hip", "encode.hip", "composite.hip", "march.hip", "pose.hip"])
def test_no_mfma_result_read_unpadded_after_a_branch(src, tmp_path):
    out = tmp_path / "k.s"
    cmd = [build.HIPCC, *build.FLAGS, "--cuda-device-only", "-S", os.path.join(build.CSRC, src),
           "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    asm = out.read_text()
    assert "v_mfma" in asm or src != "mlp.hip"
    assert unpadded_mfma_reads_after_branches(asm) == []


def test_the_branch_scan_finds_an_unpadded_read():
    # a taken branch to a join whose first instruction reads the accumulator
    # written two instructions before it, and the same join padded
    bad = "\n".join(["\tv_mfma_f32_16x16x32_bf16 v[24:27], v[28:31], v[16:19], v[24:27]",
                     "\tv_mfma_f32_16x16x32_bf16 v[28:31], v[28:31], v[32:35], v[40:43]",
                     "\ts_cbranch_vccnz .LBB7_29", "\tv_mov_b32_e32 v1, 0",
                     ".LBB7_29:", "\tv_add_f32_e32 v3, v0, v24"])
    assert len(unpadded_mfma_reads_after_branches(bad)) == 1
    good = bad.replace(".LBB7_29:\n", ".LBB7_29:\n\ts_nop 7\n")
    assert unpadded_mfma_reads_after_branches(good) == []
