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
    assert lib.dresd_search_plan(None, 1, 1, None, None, None, None, None) == _lib.EINVAL
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


def test_new_entry_points_reject_bad_arguments_before_device_work():
    """Search variants, the transform, draft assembly, the partitioned index
    and k-means validate their arguments before any HIP call."""
    lib = _lib.load()
    E = _lib.EINVAL
    fake = ctypes.c_void_p(16)  # never dereferenced: arguments are checked first
    out = ctypes.c_void_p()
    assert lib.dresd_search_filtered(None, None, None, 1, 1, None, None, None, None) == E
    # transform: ranges, then null pointers; M = 0 is a no-op
    assert lib.dresd_transform(fake, -1, 4, fake, fake, 1e-5, fake, 2, 1e-12, fake, None) == E
    assert lib.dresd_transform(fake, 1, 0, fake, fake, 1e-5, fake, 2, 1e-12, fake, None) == E
    assert lib.dresd_transform(fake, 1, 4, fake, fake, -1.0, fake, 2, 1e-12, fake, None) == E
    assert lib.dresd_transform(None, 1, 4, None, None, 1e-5, None, 2, 1e-12, None, None) == E
    assert lib.dresd_transform(None, 0, 4, None, None, 1e-5, None, 2, 1e-12, None, None) == 0
    # drafts: B, k, L, length, r ranges; nulls with B > 0; B = 0 is a no-op
    for B, k, L, r, ln in [(-1, 4, 4, 2, 2), (1, 0, 4, 1, 2), (1, 2000, 4, 1, 2), (1, 4, 4, 5, 2),
                           (1, 4, 4, 0, 2), (1, 4, 4, 2, 5), (1, 4, 4, 2, 0), (1, 4, 0, 2, 1)]:
        assert lib.dresd_pack_drafts(fake, B, k, L, r, ln, 0, fake, fake, None) == E, (B, k, L, r)
    assert lib.dresd_pack_drafts(None, 1, 4, 4, 2, 2, 0, None, None, None) == E
    assert lib.dresd_pack_drafts(None, 0, 4, 4, 2, 2, 0, None, None, None) == 0
    # partitioned index
    assert lib.dresd_ivf_create(None, None, 10, 8, 4, 0, None, 2, None, None,
                                ctypes.byref(out)) == E
    for N, d, L, dt, P in [(0, 8, 4, 0, 2), (10, 0, 4, 0, 2), (10, 8, 0, 0, 2), (10, 8, 4, 3, 2),
                           (10, 8, 4, 0, 0), (10, 8, 4, 0, (1 << 24) + 1)]:
        assert lib.dresd_ivf_create(fake, fake, N, d, L, dt, fake, P, fake, None,
                                    ctypes.byref(out)) == E, (N, d, L, dt, P)
        assert out.value is None
    assert lib.dresd_ivf_search(None, None, 1, 1, 1, None, None, None, None) == E
    assert lib.dresd_ivf_search_filtered(None, None, None, 1, 1, 1, None, None, None, None) == E
    assert lib.dresd_ivf_search_probes(None, None, None, 1, None, 1, 1, None, None, None,
                                       None) == E
    assert lib.dresd_ivf_info(None, None, None, None, None, None, None) == E
    assert lib.dresd_ivf_profile_enable(None, 1) == E
    assert lib.dresd_ivf_profile_read(None, None, None, None) == E
    lib.dresd_ivf_destroy(None)  # ignored
    # k-means
    for n, d, dt, P in [(-1, 8, 0, 2), (10, 0, 0, 2), (10, 20000, 0, 2), (10, 8, 3, 2),
                        (10, 8, 0, 0)]:
        assert lib.dresd_kmeans_assign(fake, n, d, dt, fake, P, fake, None, None) == E
        assert lib.dresd_kmeans_update(fake, n, d, dt, fake, P, fake, None, None) == E
    assert lib.dresd_kmeans_assign(None, 10, 8, 0, None, 2, None, None, None) == E
    assert lib.dresd_kmeans_assign(None, 0, 8, 0, None, 2, None, None, None) == 0
    assert lib.dresd_kmeans_update(None, 10, 8, 0, None, 2, None, None, None) == E
    for n, d, dt, P in [(0, 8, 0, 1), (10, 0, 0, 2), (10, 20000, 0, 2), (10, 8, 3, 2),
                        (10, 8, 0, 0), (10, 8, 0, 11)]:
        assert lib.dresd_kmeans_init(fake, n, d, dt, P, 7, fake, None) == E
    assert lib.dresd_kmeans_init(None, 10, 8, 0, 2, 7, fake, None) == E
    assert lib.dresd_kmeans_init(fake, 10, 8, 0, 2, 7, None, None) == E
    # bandwidth probe
    ms = ctypes.c_double()
    assert lib.dresd_bw_probe(None, 1 << 20, 1, 0, ctypes.byref(ms), None) == E
    assert lib.dresd_bw_probe(fake, 1 << 20, 1, 0, None, None) == E
    for nbytes, reps, wg in [((1 << 20) + 1, 1, 0), (1 << 19, 1, 0), (1 << 20, 0, 0),
                             (1 << 20, 1001, 0), (1 << 20, 1, -1)]:
        assert lib.dresd_bw_probe(fake, nbytes, reps, wg, ctypes.byref(ms), None) == E
