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
    "mlp.hip": {"k_mlp_fwdILi4ELb1E": 8, "k_mlp_bwdILi4ELb0E": 8, "k_mlp_bwdILi4ELb1E": 6},
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
