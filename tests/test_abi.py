"""The C-ABI library loads and exports every symbol include/dresd.h declares;
argument errors are reported without touching a GPU (CPU only)."""
import ctypes
import os
import re

import pytest

from paper_2502_15572_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dresd.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dresd_[a-z_]+)\s*\(", src)))


def test_header_declares_the_binding_surface():
    assert _declared() == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    for name in _declared():
        assert hasattr(lib, name), name


def test_null_arguments_are_rejected_before_any_device_work():
    lib = _lib.load()
    out = ctypes.c_void_p()
    assert lib.dresd_index_create(None, None, 10, 8, 4, 0, None, ctypes.byref(out)) == _lib.EINVAL
    assert b"NULL" in lib.dresd_last_error()
    assert lib.dresd_search(None, None, 1, 1, None, None, None, None) == _lib.EINVAL
    assert lib.dresd_index_info(None, None, None, None, None) == _lib.EINVAL
    assert lib.dresd_profile_enable(None, 1) == _lib.EINVAL
    assert lib.dresd_profile_read(None, None, None, None) == _lib.EINVAL
    assert lib.dresd_search_plan(None, 1, 1, None, None, None, None) == _lib.EINVAL
    lib.dresd_index_destroy(None)  # ignored


@pytest.mark.parametrize("N,d,L,dt", [(0, 8, 4, 0), (10, 0, 4, 0), (10, 8, 0, 0), (10, 8, 4, 3),
                                      (10, 20000, 4, 0), (10, 8, 5000, 0)])
def test_create_range_checks(N, d, L, dt):
    lib = _lib.load()
    out = ctypes.c_void_p()
    fake = ctypes.c_void_p(16)  # never dereferenced: sizes are checked first
    assert lib.dresd_index_create(fake, fake, N, d, L, dt, None, ctypes.byref(out)) == _lib.EINVAL
    assert out.value is None


def test_last_error_is_thread_local():
    import threading
    lib = _lib.load()
    lib.dresd_search(None, None, 1, 1, None, None, None, None)
    seen = []

    def other():
        seen.append(lib.dresd_last_error())

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen == [b""]
