"""Parity at the workloads' full sizes, in the launch configuration bench.py
times (same index build, same plans).

The oracle computes the full top-k for a sample of the batch's queries over
the whole datastore (host copy of the same keys); for every query of the
batch the returned rows are re-scored one by one by the oracle and checked
for order, range, bit-exact tokens and score agreement.
"""
import os
import sys
import time

import numpy as np
import pytest
import torch

import oracle
from datagen import WORKLOADS, generate, to_numpy_bits
from parity import TOL, check_batch, check_query

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
SAMPLED = 2  # queries per batch checked against the oracle's full top-k


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def built():
    cache = {}

    def get(name):
        if name not in cache:
            cache.clear()
            torch.cuda.empty_cache()
            from paper_2502_15572_amd import Index
            w = WORKLOADS[name]
            t = time.time()
            g = generate(w, DEV)
            ix = Index(g["keys"], g["cont"])
            kb, dt = to_numpy_bits(g["keys"])
            cont = g["cont"].cpu().numpy()
            say("built %s in %.1fs" % (name, time.time() - t))
            cache[name] = (w, g, ix, kb, dt, cont)
        return cache[name]

    yield get
    cache.clear()


CASES = [(name, B) for name, w in WORKLOADS.items() for B in w.batches]
# The 1M x 4096 datastore at B = 64: eight 8-query groups in one scan launch
# (their workgroups share each key range through one XCD's L2).
CASES.insert(CASES.index(("hidden1m_d4096_bf16", max(WORKLOADS["hidden1m_d4096_bf16"].batches))) + 1,
             ("hidden1m_d4096_bf16", 64))


@pytest.mark.parametrize("name,B", CASES, ids=["%s-B%d" % c for c in CASES])
def test_fullsize(built, name, B):
    w, g, ix, kb, dt, cont = built(name)
    q = g["queries"][:B].contiguous()
    say("search %s B=%d k=%d" % (name, B, w.k))
    idx, score, tok = ix.search(q, w.k)
    torch.cuda.synchronize()
    gi, gs, gt = idx.cpu().numpy(), score.cpu().numpy(), tok.cpu().numpy()
    qn = q.cpu().numpy()
    tol = TOL[dt]
    # every query: order, range, distinctness, tokens, scores vs exact
    for b in range(B):
        ex = oracle.score_rows(kb, dt, qn[b], gi[b])
        assert np.all(np.diff(gs[b].astype(np.float64)) <= 0)
        assert gi[b].min() >= 0 and gi[b].max() < w.N and np.unique(gi[b]).size == w.k
        assert np.array_equal(gt[b], cont[gi[b]])
        assert np.max(np.abs(gs[b].astype(np.float64) - ex)) <= tol
    # sampled queries: full comparison with the oracle's own top-k
    pick = sorted({0, B - 1})[:SAMPLED]
    t = time.time()
    o_idx, o_score, _, o_next = oracle.topk(kb, dt, qn[pick], w.k, cont)
    say("  oracle %d queries in %.1fs" % (len(pick), time.time() - t))
    rep = check_batch(gi[pick], gs[pick], gt[pick], o_idx, o_score, o_next,
                      lambda bb, rows: oracle.score_rows(kb, dt, qn[pick[bb]], rows), w.N, cont,
                      tol)
    say("  exact-order %.2f max|g-exact| %.2e" % (rep["exact_order_rate"],
                                                   rep["max_abs_vs_exact"]))
