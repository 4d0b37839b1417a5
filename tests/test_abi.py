"""The C-ABI library loads, exports every function include/pnerf.h declares,
matches the binding's struct layouts, and rejects bad arguments on the host
before touching a device.  CPU only (no compute calls)."""
import ctypes as C
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pnerf.h")


@pytest.fixture(scope="module")
def pn():
    from paper_2210_10108_amd import pnerf
    if not os.path.exists(pnerf.LIB_PATH):
        from paper_2210_10108_amd import build
        build.build()
    return pnerf


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pnerf_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported_and_bound(pn):
    names = declared_functions()
    assert len(names) >= 12
    L = pn.lib()
    for n in names:
        assert hasattr(L, n), n
        assert n in pn._SIGS, n
    out = subprocess.run(["nm", "-D", "--defined-only", pn.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (pnerf_\w+)", out))
    assert set(names) <= exported


def test_struct_layouts_match_header(pn, tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(f"""
#include <stddef.h>
#include <stdio.h>
#include "{HEADER}"
#define O(f) printf("%s %zu\\n", #f, offsetof(pnerf_field_params, f))
int main(void) {{
  printf("size %zu\\n", sizeof(pnerf_field_params));
  printf("isize %zu\\n", sizeof(pnerf_intrinsics));
  printf("asize %zu\\n", sizeof(pnerf_adam_params));
  printf("astate %d\\n", PNERF_ADAM_STATE);
  printf("a.decay_base %zu\\n", offsetof(pnerf_adam_params, decay_base));
  printf("a.second_moment %zu\\n", offsetof(pnerf_adam_params, second_moment));
  printf("a.representation %zu\\n", offsetof(pnerf_adam_params, representation));
  O(n_levels); O(level_res); O(table); O(w_color3); O(density_bias); O(aabb_max);
  O(march_mode); O(step); O(t_stop); O(occ_bits); O(occ_threshold); O(background);
  O(loss_type); O(loss_param); O(sh_dir_grad); O(max_workspace_bytes); O(overlap_chunks);
  return 0;
}}""")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True,
                                                 check=True).stdout.splitlines())
    assert int(got["size"]) == C.sizeof(pn.FieldParams)
    assert int(got["isize"]) == C.sizeof(pn.Intrinsics)
    assert int(got["asize"]) == C.sizeof(pn.AdamParams)
    assert int(got["astate"]) == pn.ADAM_STATE
    for k, v in got.items():
        if k in ("size", "isize", "asize", "astate"):
            continue
        if k.startswith("a."):
            assert getattr(pn.AdamParams, k[2:]).offset == int(v), k
            continue
        assert getattr(pn.FieldParams, k).offset == int(v), k


def test_host_validation_rejects_bad_arguments(pn):
    L = pn.lib()
    assert L.pnerf_step_momentum(0, None, None, None, 0.1, 0.9, None) == pn.ERR_INVALID_ARG
    assert b"K=0" in L.pnerf_last_error()
    assert L.pnerf_resample_hypotheses(70000, None, None, 6, None, 0.5, 0.1, 0.1, 1, 0,
                                       None) == pn.ERR_INVALID_ARG
    # scalar arguments are checked before pointers, so NULL pointers isolate them
    assert L.pnerf_resample_hypotheses(4, None, None, 65, None, 0.5, 0.1, 0.1, 1, 0,
                                       None) == pn.ERR_INVALID_ARG
    assert b"state_dim" in L.pnerf_last_error()
    assert L.pnerf_resample_hypotheses(4, None, None, 6, None, 0.5, 0.1, 0.1, 1, 0,
                                       None) == pn.ERR_INVALID_ARG
    assert b"NULL" in L.pnerf_last_error()
    assert L.pnerf_step_adam(4, None, None, None, -1, C.byref(pn.AdamParams()),
                             None) == pn.ERR_INVALID_ARG
    assert b"step" in L.pnerf_last_error()
    for field, bad in [("beta1", 1.0), ("beta2", -0.1), ("eps", 0.0), ("lr_rot", -1e-3),
                       ("lr_trans", float("nan")), ("decay_base", 0.0), ("decay_steps", -1),
                       ("staircase", 2), ("second_moment", 3), ("representation", 2)]:
        p = pn.AdamParams()
        setattr(p, field, bad)
        assert L.pnerf_step_adam(4, None, None, None, 0, C.byref(p), None) == \
            pn.ERR_INVALID_ARG, field
        assert b"NULL" not in L.pnerf_last_error(), field
    assert L.pnerf_step_adam(4, None, None, None, 0, C.byref(pn.AdamParams()),
                             None) == pn.ERR_INVALID_ARG
    assert b"NULL pointer" in L.pnerf_last_error()
    assert L.pnerf_step_adam(4, None, None, None, 0, None, None) == pn.ERR_INVALID_ARG
    assert L.pnerf_render_loss_grad(None, 4, None, 8, None, None, None, None, None,
                                    None) == pn.ERR_INVALID_ARG
    assert L.pnerf_create_field(None, None, None) == pn.ERR_INVALID_ARG
    # unsupported level count is refused before any device call
    p = pn.FieldParams()
    p.n_levels = 5
    p.n_features = 2
    out = C.c_void_p()
    assert L.pnerf_create_field(C.byref(p), None, C.byref(out)) == pn.ERR_NOT_SUPPORTED
    assert b"n_levels" in L.pnerf_last_error()
    p.n_levels = 4
    p.log2_table_size = 30
    assert L.pnerf_create_field(C.byref(p), None, C.byref(out)) == pn.ERR_INVALID_ARG
    p.log2_table_size = 12
    p.param_dtype = 2
    assert L.pnerf_create_field(C.byref(p), None, C.byref(out)) == pn.ERR_INVALID_ARG
    assert b"param_dtype" in L.pnerf_last_error()


def test_product_path_does_not_reference_the_oracle():
    pkg = os.path.join(ROOT, "paper_2210_10108_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, fn)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle\b", text, re.M), fn
                assert "liboracle" not in text and "pnerf_oracle" not in text, fn
