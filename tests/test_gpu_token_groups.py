"""Parity of the next-token-filtered search over keys grouped by their value's
first token (DReSD Section 3.5: a draft that does not start with the LLM's
next token is dropped; here the filter is a partitioning, and a query scans
only its next token's partition) against the CPU oracle's filtered exact
top-k.  The scores come from the three-part exact query split at every batch
size, so they are held to the 1e-5 bound.
"""
import json
import os
import sys

import numpy as np
import pytest
import torch

import oracle
from datagen import WORKLOADS, generate, to_numpy_bits
from parity import TOL, check_batch
from test_gpu_filtered import GOLDEN, NO_ROW_TOKEN, mixed_tokens

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
_TD = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_token(keys, cont, queries, next_tok, k, dtype, expect_P=None):
    from paper_2502_15572_amd import PartitionedIndex
    ix = PartitionedIndex.by_first_token(keys.to(DEV), cont.to(DEV))
    P = ix.P
    nt = torch.as_tensor(np.asarray(next_tok, np.int32)).to(DEV)
    idx, score, tok = ix.search_next_token(queries.to(DEV, torch.float32), nt, k)
    torch.cuda.synchronize()
    ix.close()
    if expect_P is not None:
        assert P == expect_P
    kb, dt = to_numpy_bits(keys)
    qn = queries.cpu().numpy().astype(np.float32)
    cn = cont.cpu().numpy()
    o_idx, o_score, _, o_next = oracle.topk(kb, dt, qn, k, cn, next_tok=next_tok)
    rep = check_batch(idx.cpu().numpy(), score.cpu().numpy(), tok.cpu().numpy(), o_idx, o_score,
                      o_next, lambda b, rows: oracle.score_rows(kb, dt, qn[b], rows),
                      kb.shape[0], cn, TOL[dt], next_tok=next_tok)
    assert rep["max_abs_vs_exact"] <= 1e-5, rep
    return rep


TOKEN_CASES = [
    # (workload, reduced N, batches)
    ("zipf33m_d128_f16", 200000 + 11, (1, 4, 37)),
    ("batch10m_d256_f16", 120000 + 9, (1, 64)),
    ("hidden1m_d4096_bf16", 6000 + 5, (1, 20)),
    ("flat16k_d256_f32", 16384, (8,)),
]


@pytest.mark.parametrize("name,N,batches", TOKEN_CASES, ids=[c[0] for c in TOKEN_CASES])
def test_token_groups_match_filtered_oracle(gpu_lib, name, N, batches):
    """Zipf first tokens; per batch the source row's token, a frequent one,
    one held by fewer than k rows and one held by none."""
    w = WORKLOADS[name].scaled(N)
    g = generate(w, "cpu")
    P = int(np.unique(g["cont"][:, 0].numpy()).size)
    for B in batches:
        nt = mixed_tokens(g["cont"], g["query_src"], B, w.k, seed=B + 1)
        say("token groups", name, "N=%d P=%d B=%d k=%d tokens %s" % (N, P, B, w.k, nt[:4].tolist()))
        rep = run_token(g["keys"], g["cont"], g["queries"][:B], nt, w.k, w.dtype, expect_P=P)
        say("  exact-order rate %.3f max|g-exact| %.2e" % (rep["exact_order_rate"],
                                                           rep["max_abs_vs_exact"]))


def test_token_groups_golden(gpu_lib):
    """The hand-derived filtered fixture: every case's indices and scores."""
    g = json.load(open(GOLDEN))
    n = len(g["first_tokens"])
    cont = torch.stack([torch.tensor(g["first_tokens"], dtype=torch.int32),
                        torch.arange(n, dtype=torch.int32) + 100], dim=1)
    q = torch.tensor([g["query"]], dtype=torch.float32)
    from paper_2502_15572_amd import PartitionedIndex
    for dt in ("f32", "f16", "bf16"):
        ix = PartitionedIndex.by_first_token(torch.eye(n, dtype=_TD[dt], device=DEV),
                                             cont.to(DEV))
        for c in g["cases"]:
            say("token golden", dt, c["name"])
            nt = torch.tensor([c["next_tok"]], dtype=torch.int32, device=DEV)
            idx, score, tok = ix.search_next_token(q.to(DEV), nt, c["k"])
            assert idx[0].tolist() == c["idx"], (dt, c["name"], idx[0].tolist())
            want = [float("-inf") if v == "-inf" else float(np.float32(v)) for v in c["score"]]
            assert score[0].cpu().tolist() == want, (dt, c["name"], score[0].tolist())
        ix.close()


def _keys(N, d, dt, seed):
    gen = torch.Generator().manual_seed(seed)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    q = torch.randn(9, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    return x, q, gen


def test_token_groups_extreme_token_values(gpu_lib):
    """First tokens anywhere in int32 (negative, zero, the largest), more
    distinct tokens than the lookup's 1,024 threads, and ragged group sizes."""
    N, d, k = 9001, 64, 12
    x, q, gen = _keys(N, d, "f16", 5)
    pool = torch.tensor([-2**31, -7, -1, 0, 1, 2**31 - 1], dtype=torch.int32)
    first = torch.where(torch.rand(N, generator=gen) < 0.5,
                        pool[torch.randint(0, 6, (N,), generator=gen)],
                        torch.randint(-3000, 3000, (N,), generator=gen, dtype=torch.int32))
    cont = torch.stack([first, torch.arange(N, dtype=torch.int32)], dim=1)
    nt = np.asarray([-2**31, 2**31 - 1, -1, 0, int(first[17]), 2999, -2999, 123456789, -7],
                    np.int32)
    run_token(x, cont, q, nt, k, "f16", expect_P=int(torch.unique(first).numel()))


def test_token_groups_one_token_and_small_groups(gpu_lib):
    """One token for every row (one partition, the unfiltered top-k), and
    groups smaller than k (padded results)."""
    N, d, k = 5003, 128, 40
    x, q, gen = _keys(N, d, "bf16", 6)
    cont = torch.stack([torch.full((N,), 42, dtype=torch.int32),
                        torch.arange(N, dtype=torch.int32)], dim=1)
    run_token(x, cont, q, np.full(9, 42, np.int32), k, "bf16", expect_P=1)
    first = (torch.arange(N, dtype=torch.int32) % 400)  # 12-13 rows per token
    cont = torch.stack([first, torch.arange(N, dtype=torch.int32)], dim=1)
    run_token(x, cont, q, np.asarray([0, 1, 399, 5, 77, 400, NO_ROW_TOKEN, 3, 3], np.int32),
              k, "bf16", expect_P=400)


def test_token_groups_errors_and_empty_batch(gpu_lib):
    from paper_2502_15572_amd import PartitionedIndex, train_partitions
    from paper_2502_15572_amd._lib import DresdError
    N, d = 3000, 64
    x, q, gen = _keys(N, d, "f16", 7)
    cont = torch.randint(0, 50, (N, 2), generator=gen, dtype=torch.int32)
    xt, ct, qt = x.to(DEV), cont.to(DEV), q.to(DEV)
    ix = PartitionedIndex.by_first_token(xt, ct)
    nt = torch.zeros(9, dtype=torch.int32, device=DEV)
    with pytest.raises(DresdError):  # no centroids to probe
        ix.search(qt, 5, 1)
    idx, score, tok = ix.search_next_token(qt[:0], nt[:0], 5)
    assert idx.shape == (0, 5)
    ix.close()
    cents, assign = train_partitions(xt, 8, iters=2, seed=1)
    cix = PartitionedIndex(xt, ct, cents, assign)
    with pytest.raises(DresdError):  # not grouped by first token
        cix.search_next_token(qt, nt, 5)
    cix.close()
