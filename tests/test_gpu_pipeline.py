"""One decode step of retrieval on the GPU, Algorithm 1 steps 4-8: hidden
states -> query-side transform (Eq. 1, Section 3.3, Eq. 2) -> next-token-
filtered search (Section 3.5; exact and partitioned) -> draft assembly
(Section 3.6), against the same chain of oracles.

The datastore's keys are the oracle's transform of synthetic hidden states
(rounded to f16), so no oracle input comes from the device.  The device's
queries differ from the oracle's by fp32 rounding (~1e-6), far inside the
2e-3 bound for 16-bit keys; drafts are compared bit for bit for queries whose
device ranking equals the oracle's."""
import numpy as np
import pytest
import torch

import oracle
from parity import TOL, check_batch

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def hidden(rng, n, D, centres):
    a = rng.integers(0, centres.shape[0], n)
    return (centres[a] + 0.4 * rng.standard_normal((n, D))).astype(np.float32)


@pytest.mark.parametrize("mode", ["exact", "partitioned", "token_groups"])
def test_decode_step_chain(gpu_lib, mode):
    partitioned = mode == "partitioned"
    from paper_2502_15572_amd import Index, PartitionedIndex, pack_drafts, transform
    rng = np.random.default_rng(5)
    N, D, l, L, B, k, r = 20000, 256, 64, 6, 12, 40, 8
    centres = rng.standard_normal((50, D)) * 2.0
    xs = hidden(rng, N, D, centres)
    mean = xs.mean(axis=0).astype(np.float32)
    var = xs.var(axis=0).astype(np.float32)
    W = np.linalg.qr(rng.standard_normal((D, D)))[0][:, :l].astype(np.float32)
    keys64 = oracle.transform(xs, mean, var, W)
    keys = keys64.astype(np.float16)
    cont = rng.integers(1, 30, (N, L)).astype(np.int32)
    cont[rng.random((N, L)) < 0.05] = 0  # EOS inside some values
    xq = hidden(rng, B, D, centres)
    q_or = oracle.transform(xq, mean, var, W).astype(np.float32)
    nt = cont[rng.integers(0, N, B), 0].astype(np.int32)
    nt[0] = 10 ** 6  # no value starts with it: an empty draft matrix
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    if partitioned:
        P, S = 40, 12
        x64 = oracle.decode_keys(keys, "f16")
        c = x64[rng.choice(N, P, replace=False)]
        for _ in range(3):
            a, _, _ = oracle.kmeans_assign(x64, c)
            c = oracle.kmeans_update(x64, a, c)
        c32 = c.astype(np.float32)
        a, _, _ = oracle.kmeans_assign(x64, c32.astype(np.float64))
        ix = PartitionedIndex(t(keys), t(cont), t(c32), t(a))
        p_idx, p_sc, _, _ = oracle.topk(c32, "f32", q_or, S + 1)
        sel = np.nonzero(p_sc[:, S - 1] - p_sc[:, S] >= 1e-5)[0]
        probes = p_idx[:, :S].astype(np.int32)
    elif mode == "token_groups":
        ix = PartitionedIndex.by_first_token(t(keys), t(cont))
        sel = np.arange(B)
    else:
        ix = Index(t(keys), t(cont))
        sel = np.arange(B)
    # the device chain, on one stream
    y = transform(t(xq), t(mean), t(var), t(W))
    if partitioned:
        gi, gs, gt = ix.search(y, k, S, next_tok=t(nt))
    elif mode == "token_groups":
        gi, gs, gt = ix.search_next_token(y, t(nt), k)
    else:
        gi, gs, gt = ix.search(y, k, next_tok=t(nt))
    drafts, count = pack_drafts(gt, r, L)
    torch.cuda.synchronize()
    gi, gs, gt = gi.cpu().numpy()[sel], gs.cpu().numpy()[sel], gt.cpu().numpy()[sel]
    drafts, count = drafts.cpu().numpy()[sel], count.cpu().numpy()[sel]
    # the oracle chain
    if partitioned:
        o_idx, o_score, o_tok, o_next = oracle.topk_partitioned(keys, "f16", q_or[sel], k, a, P,
                                                                 probes[sel], cont, next_tok=nt[sel])
        sets = [set(p.tolist()) for p in probes[sel]]
        adm = lambda b, rows: np.isin(a[rows], list(sets[b])) & (cont[rows, 0] == nt[sel][b])
    else:
        o_idx, o_score, o_tok, o_next = oracle.topk(keys, "f16", q_or, k, cont, next_tok=nt)
        adm = None
    if adm is None:
        check_batch(gi, gs, gt, o_idx, o_score, o_next,
                    lambda b, rows: oracle.score_rows(keys, "f16", q_or[sel][b], rows), N, cont,
                    TOL["f16"], next_tok=nt)
    else:
        check_batch(gi, gs, gt, o_idx, o_score, o_next,
                    lambda b, rows: oracle.score_rows(keys, "f16", q_or[sel][b], rows), N, cont,
                    TOL["f16"], admitted_b=adm)
    o_drafts, o_count = oracle.pack_drafts(o_tok, r, L)
    same = [b for b in range(len(sel)) if np.array_equal(gi[b], o_idx[b])]
    assert len(same) >= len(sel) // 2
    for b in same:
        assert np.array_equal(drafts[b], o_drafts[b]) and count[b] == o_count[b]
    if not partitioned:
        assert count[0] == 0 and (drafts[0] == 0).all()
    ix.close()
