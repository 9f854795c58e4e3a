"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function the headers under include/ declare (pam_lattice.h, the
filter; pam_probe.h, the benchmark's row-copy probe), and rejects invalid
arguments before touching the device."""
import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


@pytest.fixture(scope="module")
def L():
    from paper_1907_00641_amd import binding

    if not os.path.exists(binding.LIB_PATH):
        from paper_1907_00641_amd.build import build_library

        build_library()
    return binding.lib()


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(pam_[a-z_]+)\s*\(", text)
    return sorted(set(names))


def test_header_declares_the_three_operations():
    names = declared_functions()
    for op in ("pam_lattice_build", "pam_filter_fwd", "pam_filter_bwd"):
        assert op in names


def test_library_exports_every_declared_symbol(L):
    from paper_1907_00641_amd import binding

    names = declared_functions()
    assert set(names) == set(binding.EXPORTS)
    for name in names:
        assert hasattr(L, name), name


def test_status_strings(L):
    from paper_1907_00641_amd import binding as B

    for s in range(7):
        assert B.status_string(s)
    assert B.status_string(B.PAM_OK) == "ok"


def test_kernel_names(L):
    from paper_1907_00641_amd import binding as B

    names = B.pam_kernel_names()
    for k in ("range", "layout", "insert", "compact", "resolve", "scan", "scatter", "tiles",
              "splat", "blur", "slice", "splat_bwd", "slice_bwd"):
        assert k in names


def _build(L, feat, n, d, lat):
    return L.pam_lattice_build(feat, n, d, None, lat)


def test_build_rejects_bad_arguments_on_host(L):
    from paper_1907_00641_amd import binding as B

    h = ctypes.c_void_p(None)
    fake = ctypes.c_void_p(0x1000)
    assert _build(L, fake, 10, 3, None) == B.PAM_ERR_INVALID_ARGUMENT       # lat NULL
    assert _build(L, fake, 10, 0, ctypes.byref(h)) == B.PAM_ERR_INVALID_ARGUMENT
    assert _build(L, fake, 10, 17, ctypes.byref(h)) == B.PAM_ERR_INVALID_ARGUMENT
    assert _build(L, fake, -1, 3, ctypes.byref(h)) == B.PAM_ERR_INVALID_ARGUMENT
    assert _build(L, None, 10, 3, ctypes.byref(h)) == B.PAM_ERR_INVALID_ARGUMENT
    assert _build(L, fake, 1 << 29, 3, ctypes.byref(h)) == B.PAM_ERR_INVALID_ARGUMENT  # n(d+1) >= 2^31
    assert h.value is None  # no handle created on rejected calls
    assert "d must be" in B.last_error() or "n must" in B.last_error()


def test_filter_calls_reject_null_handle(L):
    from paper_1907_00641_amd import binding as B

    fake = ctypes.c_void_p(0x1000)
    assert L.pam_filter_fwd(None, fake, 4, 0, fake, None) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_filter_bwd(None, fake, fake, 4, 0, fake, fake, None) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_lattice_stats(None, None, None) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_lattice_export(None, None, None, None, None) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_lattice_set_capacity(None, 64, 1) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_timing_enable(None, 1) == B.PAM_ERR_INVALID_ARGUMENT
    L.pam_lattice_destroy(None)  # ignored


def test_binding_refuses_to_run_without_library(monkeypatch, tmp_path):
    """The product path has no CPU fallback: a missing library raises."""
    from paper_1907_00641_amd import binding as B

    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        B.lib()


def test_grouped_build_rejects_bad_offsets_on_host(L):
    from paper_1907_00641_amd import binding as B
    import numpy as np

    h = ctypes.c_void_p(None)
    fake = ctypes.c_void_p(0x1000)

    def build(starts, groups=None):
        gs = np.asarray(starts, dtype=np.int64)
        G = len(gs) - 1 if groups is None else groups
        return L.pam_lattice_build_groups(fake, 10, 3, gs.ctypes.data, G, None, ctypes.byref(h))

    assert build([0, 4, 3, 10]) == B.PAM_ERR_INVALID_ARGUMENT   # decreasing
    assert build([1, 4, 10]) == B.PAM_ERR_INVALID_ARGUMENT      # does not start at 0
    assert build([0, 4, 9]) == B.PAM_ERR_INVALID_ARGUMENT       # does not end at n
    assert build([0, 10], groups=0) == B.PAM_ERR_INVALID_ARGUMENT
    assert build([0, 10], groups=B.PAM_MAX_GROUPS + 1) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_lattice_build_groups(fake, 10, 3, None, 2, None, ctypes.byref(h)) == B.PAM_ERR_INVALID_ARGUMENT
    assert h.value is None
    assert L.pam_lattice_export_groups(None, None) == B.PAM_ERR_INVALID_ARGUMENT


def test_log_level_prints_failures(tmp_path):
    """PAM_LOG_LEVEL=2 prints each failure with its message on stderr (host
    only: an argument error needs no GPU)."""
    import subprocess
    import sys

    code = ("import ctypes, sys; sys.path.insert(0, %r); from paper_1907_00641_amd import binding as B; "
            "L = B.lib(); h = ctypes.c_void_p(None); "
            "print(L.pam_lattice_build(None, 10, 3, None, ctypes.byref(h)))") % ROOT
    env = dict(os.environ, PAM_LOG_LEVEL="2")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=120)
    assert r.stdout.strip() == "1", r.stdout + r.stderr
    assert "[pam] error 1: feat is NULL" in r.stderr
    env["PAM_LOG_LEVEL"] = "0"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=120)
    assert "[pam]" not in r.stderr
