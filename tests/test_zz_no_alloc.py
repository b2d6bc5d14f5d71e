"""Allocation-free search (dresd_search_noalloc) through the C ABI: it
returns bit for bit what dresd_search returns on the same index and inputs,
on two calls in a row (the second with a smaller input, so it runs on the
scratch the first left behind); it makes no device allocation (free device
memory unchanged; the library's allocation-failure hook armed at the next
allocation does not stop it); and it rejects a search whose workspace
exceeds the fixed scratch with EINVAL, writing nothing."""
import ctypes
import os

import pytest
import torch

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
P = ctypes.c_void_p
OK, EINVAL = 0, 1
SCRATCH_BYTES = 64 << 20


def say(*a):
    print(*a, flush=True)


def _outs(B, k, L, fill=False):
    mk = torch.full if fill else (lambda shape, v, **kw: torch.empty(shape, **kw))
    return (mk((B, k), -7, dtype=torch.int64, device=DEV),
            mk((B, k), 7.0, dtype=torch.float32, device=DEV),
            mk((B, k, L), -7, dtype=torch.int32, device=DEV))


def _noalloc(lib, ix, q, out):
    idx, score, tok = out
    B, k = idx.shape
    return lib.dresd_search_noalloc(ix._h, P(q.data_ptr()), B, k, P(idx.data_ptr()),
                                    P(score.data_ptr()), P(tok.data_ptr()), None)


def test_noalloc_matches_search(gpu_lib):
    from paper_2502_15572_amd import Index
    gen = torch.Generator(device="cuda").manual_seed(7)
    N, d, L = 200003, 128, 10
    x = torch.randn(N, d, device=DEV, generator=gen)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float16)
    cont = torch.randint(0, 32000, (N, L), device=DEV, generator=gen, dtype=torch.int32)
    q = torch.randn(64, d, device=DEV, generator=gen)
    q = (q / q.norm(dim=1, keepdim=True)).contiguous()
    ix = Index(x, cont)
    # the larger call first, then a smaller one on the scratch it left behind
    cases = [(16, 64), (3, 10)]
    outs = {c: _outs(c[0], c[1], L) for c in cases}
    refs = {}
    for B, k in cases:
        assert ix.plan(B, k)["workspace_bytes"] <= SCRATCH_BYTES
        refs[(B, k)] = [t.clone() for t in ix.search(q[:B].contiguous(), k)]
    torch.cuda.synchronize()
    qs = {c: q[:c[0]].contiguous() for c in cases}
    st = _noalloc(gpu_lib, ix, qs[cases[0]], outs[cases[0]])  # kernels loaded and warm
    assert st == OK, gpu_lib.dresd_last_error()
    torch.cuda.synchronize()
    # no torch work inside the measured window: only the two calls
    free0 = torch.cuda.mem_get_info()[0]
    os.environ["DRESD_FAIL_ALLOC_AT"] = "1"  # any library allocation would now fail
    try:
        for B, k in cases:
            say("noalloc B=%d k=%d" % (B, k))
            st = _noalloc(gpu_lib, ix, qs[(B, k)], outs[(B, k)])
            assert st == OK, gpu_lib.dresd_last_error()
        torch.cuda.synchronize()
    finally:
        os.environ.pop("DRESD_FAIL_ALLOC_AT", None)
    assert torch.cuda.mem_get_info()[0] == free0
    for c in cases:
        for a, b in zip(outs[c], refs[c]):
            assert torch.equal(a, b), c
    # too large for the scratch: rejected before any work
    B, k = 64, 1000
    assert ix.plan(B, k)["workspace_bytes"] > SCRATCH_BYTES
    big = _outs(B, k, L, fill=True)
    st = _noalloc(gpu_lib, ix, q[:B].contiguous(), big)
    torch.cuda.synchronize()
    assert st == EINVAL and b"scratch" in gpu_lib.dresd_last_error()
    assert (big[0] == -7).all() and (big[1] == 7.0).all() and (big[2] == -7).all()
    ix.close()


def test_noalloc_tiled_contraction(gpu_lib):
    """The same contract on the tiled contraction (keys of 2,048 dims, 9-16
    queries, each with a sampled pass): bit-identical to dresd_search on two
    calls in a row, the second smaller, with no device allocation."""
    from paper_2502_15572_amd import Index
    gen = torch.Generator(device="cuda").manual_seed(11)
    N, d, L = 20011, 2048, 4
    x = torch.randn(N, d, device=DEV, generator=gen)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.bfloat16)
    cont = torch.randint(0, 32000, (N, L), device=DEV, generator=gen, dtype=torch.int32)
    q = torch.randn(16, d, device=DEV, generator=gen)
    q = (q / q.norm(dim=1, keepdim=True)).contiguous()
    ix = Index(x, cont)
    cases = [(16, 12), (9, 5)]
    outs = {c: _outs(c[0], c[1], L) for c in cases}
    refs = {}
    for B, k in cases:
        plan = ix.plan(B, k)
        assert plan["scan_kernel"] == "tiled" and plan["sample_passes"] == 1
        assert plan["workspace_bytes"] <= SCRATCH_BYTES
        refs[(B, k)] = [t.clone() for t in ix.search(q[:B].contiguous(), k)]
    torch.cuda.synchronize()
    qs = {c: q[:c[0]].contiguous() for c in cases}
    st = _noalloc(gpu_lib, ix, qs[cases[0]], outs[cases[0]])
    assert st == OK, gpu_lib.dresd_last_error()
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    os.environ["DRESD_FAIL_ALLOC_AT"] = "1"
    try:
        for B, k in cases:
            say("noalloc tiled B=%d k=%d" % (B, k))
            st = _noalloc(gpu_lib, ix, qs[(B, k)], outs[(B, k)])
            assert st == OK, gpu_lib.dresd_last_error()
        torch.cuda.synchronize()
    finally:
        os.environ.pop("DRESD_FAIL_ALLOC_AT", None)
    assert torch.cuda.mem_get_info()[0] == free0
    for c in cases:
        for a, b in zip(outs[c], refs[c]):
            assert torch.equal(a, b), c
    ix.close()


def test_noalloc_wide_batch_takes_shared_key_scan(gpu_lib):
    """1,024-dim keys past 64 queries: dresd_search runs the tiled contraction
    with query groups, whose lists exceed the fixed scratch; the allocation-
    free search runs the shared-key scan instead (a launch per 64 queries)
    and returns bitwise the same results, on two calls in a row, the second
    smaller, with no device allocation."""
    from paper_2502_15572_amd import Index
    gen = torch.Generator(device="cuda").manual_seed(12)
    N, d, L = 20011, 1024, 3
    x = torch.randn(N, d, device=DEV, generator=gen)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float16)
    cont = torch.randint(0, 32000, (N, L), device=DEV, generator=gen, dtype=torch.int32)
    q = torch.randn(130, d, device=DEV, generator=gen)
    q = (q / q.norm(dim=1, keepdim=True)).contiguous()
    ix = Index(x, cont)
    cases = [(130, 16), (100, 10)]
    outs = {c: _outs(c[0], c[1], L) for c in cases}
    refs = {}
    for B, k in cases:
        plan = ix.plan(B, k)
        assert plan["scan_kernel"] == "tiled" and plan["launches"] == 1
        assert plan["workspace_bytes"] > SCRATCH_BYTES
        refs[(B, k)] = [t.clone() for t in ix.search(q[:B].contiguous(), k)]
    torch.cuda.synchronize()
    qs = {c: q[:c[0]].contiguous() for c in cases}
    st = _noalloc(gpu_lib, ix, qs[cases[0]], outs[cases[0]])
    assert st == OK, gpu_lib.dresd_last_error()
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    os.environ["DRESD_FAIL_ALLOC_AT"] = "1"
    try:
        for B, k in cases:
            say("noalloc wide B=%d k=%d" % (B, k))
            st = _noalloc(gpu_lib, ix, qs[(B, k)], outs[(B, k)])
            assert st == OK, gpu_lib.dresd_last_error()
        torch.cuda.synchronize()
    finally:
        os.environ.pop("DRESD_FAIL_ALLOC_AT", None)
    assert torch.cuda.mem_get_info()[0] == free0
    for c in cases:
        for a, b in zip(outs[c], refs[c]):
            assert torch.equal(a, b), c
    ix.close()
