"""Parity at the workloads' full sizes, in the launch configuration bench.py
times (same index build, same plans).

Every query of every batch is compared with the oracle's own exact top-k
over the whole datastore (host copy of the same keys; one batched oracle call
per case, each key row read once for all queries): rules R1-R7, and every
returned score against the operand model (the query as the matrix cores take
it for that batch size) within fp32 accumulation error, and against the
exact score within the documented rounding bound.  Printed per case: the
exact-order rate, max |g - exact| and max |g - model|.
"""
import time

import numpy as np
import pytest
import torch

import oracle
from datagen import WORKLOADS, generate, to_numpy_bits
from parity import TOL, check_batch, check_operand_model

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def built():
    cache = {}

    def get(name, B):
        w = WORKLOADS[name].with_pool(B)  # a pool of at least B distinct queries
        key = (name, w.pool)
        if key not in cache:
            cache.clear()
            torch.cuda.empty_cache()
            from paper_2502_15572_amd import Index
            t = time.time()
            g = generate(w, DEV)
            ix = Index(g["keys"], g["cont"])
            kb, dt = to_numpy_bits(g["keys"])
            cont = g["cont"].cpu().numpy()
            say("built %s in %.1fs" % (name, time.time() - t))
            cache[key] = (w, g, ix, kb, dt, cont)
        return cache[key]

    yield get
    cache.clear()


CASES = [(name, B) for name, w in WORKLOADS.items() for B in w.batches]
# The 1M x 4096 datastore at B = 64: eight 8-query groups in one scan launch
# (their workgroups share each key range through one XCD's L2).
CASES.insert(CASES.index(("hidden1m_d4096_bf16", max(WORKLOADS["hidden1m_d4096_bf16"].batches))) + 1,
             ("hidden1m_d4096_bf16", 64))
# Past one query group of the tiled contraction: 128 bf16 queries over the
# 1M x 4096 datastore (two query groups) and 256 f16 queries over the
# 4M x 1024 one (four), each one pass over the keys.
CASES.insert(CASES.index(("hidden1m_d4096_bf16", 64)) + 1, ("hidden1m_d4096_bf16", 128))
CASES.insert(CASES.index(("pca4m_d1024_f16", max(WORKLOADS["pca4m_d1024_f16"].batches))) + 1,
             ("pca4m_d1024_f16", 256))


@pytest.mark.parametrize("name,B", CASES, ids=["%s-B%d" % c for c in CASES])
def test_fullsize(built, name, B):
    w, g, ix, kb, dt, cont = built(name, B)
    q = g["queries"][:B].contiguous()
    assert q.shape[0] == B
    say("search %s B=%d k=%d plan %s" % (name, B, w.k, ix.plan(B, w.k)))
    idx, score, tok = ix.search(q, w.k)
    torch.cuda.synchronize()
    gi, gs, gt = idx.cpu().numpy(), score.cpu().numpy(), tok.cpu().numpy()
    qn = q.cpu().numpy()
    tol = TOL[dt]
    t = time.time()
    say("  oracle over all %d queries ..." % B)
    o_idx, o_score, _, o_next = oracle.topk(kb, dt, qn, w.k, cont)
    say("  oracle %d queries in %.1fs" % (B, time.time() - t))
    rep = check_batch(gi, gs, gt, o_idx, o_score, o_next,
                      lambda bb, rows: oracle.score_rows(kb, dt, qn[bb], rows), w.N, cont, tol)
    dm_max, mode = 0.0, ""
    for b in range(B):
        dm, _de, mode = check_operand_model(
            gi[b], gs[b], qn[b], B, dt, lambda r: oracle.decode_keys(kb[r], dt),
            lambda qq, r: oracle.score_rows(kb, dt, qq, r))
        dm_max = max(dm_max, dm)
    say("  %s B=%d: exact-order %.3f max|g-exact| %.2e max|g-model| %.2e (%s)"
        % (name, B, rep["exact_order_rate"], rep["max_abs_vs_exact"], dm_max, mode))
