"""Parity of the partitioned search at the full size of the Zipf-clustered
workload (33,554,432 keys x 128 dims f16, k = 100), in the configuration
bench.py measures (nprobe 64 of 16,384 partitions, a 128-query batch).

The partitions are the generator's own: its 16,384 Zipf-sized clusters, with
the unit vectors of their centres as centroids (seeded inputs, no k-means).
The oracle picks each query's probes (exact top-nprobe over the centroids)
and, for sampled queries whose probed set is unique (nprobe-th and next
centroid scores at least 1e-5 apart), computes the exact top-k over the
probed partitions; every query's returned rows are re-scored one by one and
checked for order, range, partition, tokens and scores."""
import time

import numpy as np
import pytest
import torch

import oracle
from datagen import WORKLOADS, generate, to_numpy_bits
from parity import TOL, check_batch

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)


def test_fullsize_partitioned():
    from paper_2502_15572_amd import PartitionedIndex
    w = WORKLOADS["zipf33m_d128_f16"]
    B, k, nprobe, SAMPLED = 128, w.k, 64, 2
    t = time.time()
    g = generate(w, DEV)
    c64 = g["centres"].to(torch.float64)
    cents = (c64 / c64.norm(dim=1, keepdim=True)).to(torch.float32).contiguous()
    assign = g["assign"].to(torch.int32).contiguous()
    P = cents.shape[0]
    ix = PartitionedIndex(g["keys"], g["cont"], cents, assign)
    kb, dt = to_numpy_bits(g["keys"])
    cont = g["cont"].cpu().numpy()
    an = assign.cpu().numpy()
    cn = cents.cpu().numpy()
    say("built partitioned %s (P=%d) in %.1fs" % (w.name, P, time.time() - t))
    q = g["queries"][:B].contiguous()
    idx, score, tok = ix.search(q, k, nprobe)
    torch.cuda.synchronize()
    gi, gs, gt = idx.cpu().numpy(), score.cpu().numpy(), tok.cpu().numpy()
    qn = q.cpu().numpy()
    tol = TOL[dt]
    p_idx, p_sc, _, _ = oracle.topk(cn, "f32", qn, nprobe + 1)
    unique = p_sc[:, nprobe - 1] - p_sc[:, nprobe] >= 1e-5
    say("  %d of %d queries with a unique probed set" % (int(unique.sum()), B))
    assert unique.sum() >= B // 2
    for b in np.nonzero(unique)[0]:
        m = int((gi[b] >= 0).sum())
        rows = gi[b, :m]
        assert np.all(gi[b, m:] == -1) and np.all(np.isinf(gs[b, m:]))
        assert np.unique(rows).size == m and (rows >= 0).all() and (rows < w.N).all()
        assert np.isin(an[rows], p_idx[b, :nprobe]).all()
        assert np.all(np.diff(gs[b, :m].astype(np.float64)) <= 0)
        assert np.array_equal(gt[b, :m], cont[rows])
        ex = oracle.score_rows(kb, dt, qn[b], rows)
        assert np.max(np.abs(gs[b, :m].astype(np.float64) - ex)) <= tol
    pick = [int(b) for b in np.nonzero(unique)[0][:SAMPLED]]
    probes = p_idx[pick, :nprobe].astype(np.int32)
    t = time.time()
    o_idx, o_score, _, o_next = oracle.topk_partitioned(kb, dt, qn[pick], k, an, P, probes, cont)
    say("  oracle %d queries in %.1fs" % (len(pick), time.time() - t))
    sets = [set(r.tolist()) for r in probes]
    rep = check_batch(gi[pick], gs[pick], gt[pick], o_idx, o_score, o_next,
                      lambda bb, rows: oracle.score_rows(kb, dt, qn[pick[bb]], rows), w.N, cont,
                      tol, admitted_b=lambda bb, rows: np.isin(an[rows], list(sets[bb])))
    say("  exact-order %.2f max|g-exact| %.2e" % (rep["exact_order_rate"],
                                                   rep["max_abs_vs_exact"]))
    ix.close()
