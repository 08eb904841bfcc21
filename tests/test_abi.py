"""The C-ABI libraries load and export every function their headers declare (no GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_23286_amd")


def declared_functions(header):
    text = open(os.path.join(ROOT, "include", header)).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(rv[s]?_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


def exported(path):
    lib = ctypes.CDLL(path)
    return lib


@pytest.mark.parametrize("header,lib", [("rv.h", "librv.so"), ("rv_synth.h", "librv_synth.so")])
def test_library_exports_every_declared_symbol(header, lib):
    path = os.path.join(PKG, lib)
    if not os.path.exists(path):
        pytest.fail(f"{lib} is not built (run __graft_entry__.build())")
    names = declared_functions(header)
    assert len(names) >= (16 if header == "rv.h" else 2)
    handle = exported(path)
    missing = [n for n in names if not hasattr(handle, n)]
    assert not missing, f"{lib} lacks {missing}"


def test_headers_compile_as_plain_c(tmp_path):
    """Both headers are C (no C++ or HIP types) and self-contained."""
    import subprocess
    src = tmp_path / "t.c"
    src.write_text('#include "rv.h"\n#include "rv_synth.h"\nint main(void){return RV_OK;}\n')
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    "-c", str(src), "-o", str(tmp_path / "t.o")], check=True)


def test_binding_loads_and_reports_version():
    from paper_2609_23286_amd import rv
    assert "gfx950" in rv.version()


def test_invalid_arguments_are_rejected_before_any_device_work():
    """Argument checks run on the host first, so they need no GPU: each call must
    return RV_ERR_INVALID with a message, and change nothing."""
    from paper_2609_23286_amd import rv
    L = rv.lib()
    h = ctypes.c_void_p()
    assert L.rv_mem_create(16, 128, 0, 10, ctypes.byref(h)) == rv.RV_ERR_INVALID
    assert b"head_dim" in L.rv_last_error()
    assert L.rv_mem_create(0, 64, 0, 10, ctypes.byref(h)) == rv.RV_ERR_INVALID
    assert L.rv_mem_create(16, 64, 11, 10, ctypes.byref(h)) == rv.RV_ERR_INVALID
    vp = ctypes.c_void_p
    assert L.rv_attend_frame(vp(1), vp(1), vp(1), 10, None, None, 0, 0, 16, 32, None, vp(1), vp(1),
                             None, None) == rv.RV_ERR_INVALID
    assert L.rv_attend_frame(vp(1), vp(1), vp(1), -1, None, None, 0, 0, 16, 64, None, vp(1), vp(1),
                             None, None) == rv.RV_ERR_INVALID
    assert L.rv_attend_frame(vp(1), vp(1), vp(1), 10, None, None, 5, 5, 16, 64, None, vp(1), vp(1),
                             None, None) == rv.RV_ERR_INVALID          # memory pointers missing
    assert L.rv_attend_frame(vp(1), vp(1), vp(1), 10, vp(1), vp(1), 6, 5, 16, 64, None, vp(1), vp(1),
                             None, None) == rv.RV_ERR_INVALID          # head stride < mem_len
    bad_q = rv.rv_qsub(3, 3, 0, 2)                                     # 9 tokens, not 10
    assert L.rv_attend_frame(vp(1), vp(1), vp(1), 10, None, None, 0, 0, 16, 64, ctypes.byref(bad_q),
                             vp(1), vp(1), vp(1), None) == rv.RV_ERR_INVALID
    assert b"does not describe" in L.rv_last_error()
    assert L.rv_admit(vp(1), 3, vp(1), vp(1), 10, None, 0, None, None) == rv.RV_ERR_INVALID
    assert L.rv_admit_layers(0, None, None, None, None, 10, None, 1, None, 0, None, None,
                             None) == rv.RV_ERR_INVALID
    assert L.rv_mem_stage(None, 10, None, None, None, None) == rv.RV_ERR_INVALID
    assert L.rv_mem_stage_frame(None, vp(1), vp(1), 10, None) == rv.RV_ERR_INVALID
    assert L.rv_mem_stage_frame(vp(1), None, vp(1), 10, None) == rv.RV_ERR_INVALID
    arr1 = (vp * 1)
    assert L.rv_mem_stage_frames(0, arr1(vp(1)), arr1(vp(1)), arr1(vp(1)), 10, None) == rv.RV_ERR_INVALID
    assert L.rv_mem_stage_frames(1, None, arr1(vp(1)), arr1(vp(1)), 10, None) == rv.RV_ERR_INVALID
    assert L.rv_mem_stage_frames(1, arr1(None), arr1(vp(1)), arr1(vp(1)), 10, None) == rv.RV_ERR_INVALID
    assert L.rv_mem_stage_frames(1, arr1(vp(1)), arr1(None), arr1(vp(1)), 10, None) == rv.RV_ERR_INVALID
    assert L.rv_attend_staged(vp(1), 10, None, None, vp(1), vp(1), None, None) == rv.RV_ERR_INVALID
    assert L.rv_admit_staged_layers(0, None, None, 10, None, 1, None, 0, None, None,
                                    None) == rv.RV_ERR_INVALID
    assert L.rv_mem_save(None, b"/tmp/x") == rv.RV_ERR_INVALID
    assert L.rv_mem_load(None, b"/tmp/x") == rv.RV_ERR_INVALID
    # n_tokens == 0 is a no-op that succeeds without touching the device
    assert L.rv_attend_frame(None, None, None, 0, None, None, 0, 0, 16, 64, None, None, None,
                             None, None) == rv.RV_OK


def test_empty_query_subset_is_accepted_and_returns_a_status():
    """A subset with no window ({0, w, N, 2}: every token special) passes the argument
    checks -- its saliency is the empty sum -- and the call returns a status instead of
    aborting: with no GPU here, the status says the device is unavailable or the library
    is not initialised on it."""
    from paper_2609_23286_amd import rv
    L = rv.lib()
    vp = ctypes.c_void_p
    N = 1041
    empty = rv.rv_qsub(0, 37, N, 2)
    st = L.rv_attend_frame(vp(1), vp(1), vp(1), N, None, None, 0, 0, 16, 64, ctypes.byref(empty), vp(1),
                           vp(1), vp(1), None)
    assert st in (rv.RV_ERR_INVALID, rv.RV_ERR_HIP) and L.rv_last_error()
    assert b"query subset" not in L.rv_last_error()


def test_truncate_checks_its_arguments():
    from paper_2609_23286_amd import rv
    L = rv.lib()
    assert L.rv_mem_truncate(None, 0) == rv.RV_ERR_INVALID
    assert L.rv_reserve_workspace(0, 16, 0, 1) == rv.RV_ERR_INVALID
    assert L.rv_reserve_workspace(1041, 16, -1, 1) == rv.RV_ERR_INVALID
