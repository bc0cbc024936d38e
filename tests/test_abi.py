"""The C-ABI library loads, exports what include/gsq.h declares, and validates on the host.

These tests make no compute call: they run without a GPU.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2604_18556_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gsq.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B._LIB_PATH):
        pytest.skip("libgsq.so not built (run __graft_entry__.build())")
    return B.load()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:gsq_status|size_t|const char\*)\s+(gsq_\w+)\s*\(", text, re.M)))


def test_header_declares_the_expected_calls():
    assert set(declared_functions()) == set(B.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", B._LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (gsq_\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_ctypes_structs_match_the_c_layout(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(r'''
#include <stdio.h>
#include <stddef.h>
#include "gsq.h"
int main(void) {
  printf("%zu %zu %zu %zu %zu %zu %zu\n", sizeof(gsq_config), offsetof(gsq_config, seed),
         offsetof(gsq_config, init_noise), offsetof(gsq_config, relaxation), sizeof(gsq_step_params),
         offsetof(gsq_step_params, kappa_next), offsetof(gsq_step_params, samples));
  return 0;
}
''')
    exe = tmp_path / "layout"
    r = subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                        "-I", "/opt/rocm/include", str(src), "-o", str(exe)], capture_output=True, text=True)
    if r.returncode:
        pytest.skip("cannot compile against hip_runtime_api.h: " + r.stderr[-300:])
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()]
    assert vals == [ctypes.sizeof(B.CConfig), B.CConfig.seed.offset, B.CConfig.init_noise.offset,
                    B.CConfig.relaxation.offset, ctypes.sizeof(B.CStepParams),
                    B.CStepParams.kappa_next.offset, B.CStepParams.samples.offset]


def _cfg(**kw):
    base = dict(out_features=8, in_features=256, levels=(-1.5, -0.5, 0.5, 1.5), group_size=128)
    base.update(kw)
    return B.LayerConfig(**base)


def test_packed_size_formula(lib):
    assert B.packed_size(_cfg()) == 8 * 256 * 2 // 8 + 2 * 8 * 2
    assert B.packed_size(_cfg(levels=(-1.0, 0.0, 1.0))) == 8 * 256 * 2 // 8 + 2 * 8 * 2
    assert B.packed_size(_cfg(levels=tuple(range(8)))) == 8 * 256 * 3 // 8 + 2 * 8 * 2
    assert B.packed_size(_cfg(batch=3, layout=B.LAYOUT_SUPERBLOCK, levels=tuple(range(8)))) == 3 * 8 * 110
    assert B.packed_size(_cfg(group_size=100)) == 0
    # local shift over a 16-level (4-bit) grid
    assert B.packed_size(_cfg(levels=tuple(range(16)), relaxation=B.RELAX_SHIFT)) == 8 * 256 * 4 // 8 + 2 * 8 * 2
    # base-3: five codes per byte, the last byte padded
    assert B.packed_size(_cfg(levels=(-1.0, 0.0, 1.0), layout=B.LAYOUT_BASE3)) == -(-8 * 256 // 5) + 2 * 8 * 2
    assert B.packed_size(_cfg(out_features=3, levels=(-1.0, 0.0, 1.0), layout=B.LAYOUT_BASE3,
                              relaxation=B.RELAX_TERNARY)) == -(-3 * 256 // 5) + 2 * 3 * 2


@pytest.mark.parametrize("bad", [
    dict(levels=(0.5, -0.5, 1.5, 2.5)),            # not increasing
    dict(levels=(1.0,)),                           # K < 2
    dict(levels=tuple(range(9))),                  # a full-grid categorical over more than 8
    dict(levels=tuple(range(17)), relaxation=B.RELAX_SHIFT),   # more than 16 grid levels
    dict(levels=tuple(range(16)), relaxation=B.RELAX_SHIFT, layout=B.LAYOUT_SUPERBLOCK),
    dict(levels=(-1.0, 0.0, 2.0), relaxation=B.RELAX_TERNARY),
    dict(levels=(-1.5, -0.5, 0.5, 1.5), relaxation=B.RELAX_TERNARY),
    dict(levels=(-1.5, -0.5, 0.5, 1.5), layout=B.LAYOUT_BASE3),
    dict(relaxation=7),
    dict(layout=3),
    dict(levels=(0.0, 0.0)),                       # not increasing / all zero
    dict(group_size=48),
    dict(in_features=200),                         # not a multiple of the group size
    dict(layout=B.LAYOUT_SUPERBLOCK, in_features=384),
    dict(precision=7),
    dict(out_features=0),
    dict(alpha=float("nan")),
])
def test_invalid_configs_are_rejected_before_any_device_work(lib, bad):
    cfg = _cfg(**{k: v for k, v in bad.items() if k != "levels"})
    c = cfg.to_c()
    if "levels" in bad:
        lv = bad["levels"]
        c.n_levels = len(lv)
        for k, x in enumerate(lv[:B.MAX_LEVELS]):
            c.levels[k] = x
    h = ctypes.c_void_p()
    st = lib.gsq_layer_init(ctypes.byref(c), ctypes.c_void_p(16), 0, ctypes.c_void_p(16), None, None,
                            ctypes.byref(h))
    assert st == B.GSQ_EINVAL and h.value is None
    assert lib.gsq_last_error()


def test_null_handles_and_arguments(lib):
    p = B.StepParams(tau=1.0).to_c()
    assert lib.gsq_step(None, ctypes.byref(p), None, None) == B.GSQ_EINVAL
    assert lib.gsq_harden(None, None, None, None, None) == B.GSQ_EINVAL
    assert lib.gsq_pack(None, None, 0, None) == B.GSQ_EINVAL
    assert lib.gsq_check(None, None) == B.GSQ_EINVAL
    assert lib.gsq_layer_destroy(None) == B.GSQ_OK
    h = ctypes.c_void_p()
    assert lib.gsq_layer_init(None, None, 0, None, None, None, ctypes.byref(h)) == B.GSQ_EINVAL
    c = _cfg().to_c()
    assert lib.gsq_gumbel(ctypes.byref(c), -1, 4, 0, None, None) == B.GSQ_EINVAL
    assert lib.gsq_gumbel(ctypes.byref(c), 0, 0, 0, None, None) == B.GSQ_OK
