"""Parity of next-token-filtered retrieval (DReSD Section 3.5: drafts that do
not start with the LLM's next token x_{t+1} are dropped; read as
filter-then-select) between the HIP path and the CPU oracle.

Each batch mixes the realistic case (the next token of the query's source
row, so the source row competes), a frequent token, a token matching fewer
rows than k (the result is padded with -1 / -inf / zero tokens) and a token
matching no row.  Covers both scan kernels (single-tile and shared-key) and
the sampled threshold passes.
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

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "filtered_closed_forms.json")
_TD = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
NO_ROW_TOKEN = 1 << 30  # no continuation starts with it


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_filtered(keys, cont, queries, next_tok, k, dtype):
    from paper_2502_15572_amd import Index
    ix = Index(keys.to(DEV), cont.to(DEV))
    nt = torch.as_tensor(np.asarray(next_tok, np.int32)).to(DEV)
    idx, score, tok = ix.search(queries.to(DEV, torch.float32), k, next_tok=nt)
    torch.cuda.synchronize()
    ix.close()
    kb, dt = to_numpy_bits(keys)
    qn = queries.cpu().numpy().astype(np.float32)
    cn = cont.cpu().numpy()
    o_idx, o_score, _, o_next = oracle.topk(kb, dt, qn, k, cn, next_tok=next_tok)
    return check_batch(idx.cpu().numpy(), score.cpu().numpy(), tok.cpu().numpy(), o_idx, o_score,
                       o_next, lambda b, rows: oracle.score_rows(kb, dt, qn[b], rows), kb.shape[0],
                       cn, TOL[dt], next_tok=next_tok)


def mixed_tokens(cont, src, B, k, seed):
    """Per query: its source row's next token, or a frequent one, a rare one
    (fewer than k matching rows) or none at all."""
    c0 = cont[:, 0].numpy()
    vals, counts = np.unique(c0, return_counts=True)
    frequent = int(vals[np.argmax(counts)])
    rare = vals[counts < k]
    rare_tok = int(rare[0]) if rare.size else frequent
    rng = np.random.default_rng(seed)
    out = []
    for b in range(B):
        r = b % 4
        if r == 0:
            out.append(int(c0[int(src[b])]) if int(src[b]) >= 0 else frequent)
        elif r == 1:
            out.append(frequent)
        elif r == 2:
            out.append(rare_tok)
        else:
            out.append(NO_ROW_TOKEN)
    return np.asarray(out, np.int32)


def test_filtered_golden_on_gpu(gpu_lib):
    g = json.load(open(GOLDEN))
    n = len(g["first_tokens"])
    cont = torch.stack([torch.tensor(g["first_tokens"], dtype=torch.int32),
                        torch.arange(n, dtype=torch.int32) + 100], dim=1)
    q = torch.tensor([g["query"]], dtype=torch.float32)
    from paper_2502_15572_amd import Index
    for dt in ("f32", "f16", "bf16"):
        ix = Index(torch.eye(n, dtype=_TD[dt], device=DEV), cont.to(DEV))
        for c in g["cases"]:
            say("filtered golden", dt, c["name"])
            nt = torch.tensor([c["next_tok"]], dtype=torch.int32, device=DEV)
            idx, score, tok = ix.search(q.to(DEV), c["k"], next_tok=nt)
            assert idx[0].tolist() == c["idx"], (dt, c["name"], idx[0].tolist())
            want = [float("-inf") if v == "-inf" else float(np.float32(v)) for v in c["score"]]
            assert score[0].cpu().tolist() == want, (dt, c["name"], score[0].tolist())
            for r, i in enumerate(c["idx"]):
                want_tok = cont[i].tolist() if i >= 0 else [0, 0]
                assert tok[0, r].cpu().tolist() == want_tok
        ix.close()


FILTERED = [
    # (workload, reduced N, batches)
    ("flat16k_d256_f32", 16384, (8,)),
    ("hidden1m_d4096_bf16", 6000 + 5, (1, 4, 20)),
    ("pca4m_d1024_f16", 40000 + 3, (1, 16)),
    ("batch10m_d256_f16", 120000 + 9, (64, 256)),
    ("zipf33m_d128_f16", 200000 + 11, (1, 128)),
]


@pytest.mark.parametrize("name,N,batches", FILTERED, ids=[f[0] for f in FILTERED])
def test_filtered_parity_reduced(gpu_lib, name, N, batches):
    w = WORKLOADS[name].scaled(N)
    g = generate(w, "cpu")
    for B in batches:
        nt = mixed_tokens(g["cont"], g["query_src"], B, w.k, seed=B)
        say("filtered", name, "N=%d B=%d k=%d tokens %s" % (N, B, w.k, nt[:4].tolist()))
        rep = run_filtered(g["keys"], g["cont"], g["queries"][:B], nt, w.k, w.dtype)
        say("  exact-order rate %.3f" % rep["exact_order_rate"])


# Few key blocks per tile (1-4): fewer block loads than the load ring's depth
# follow a wave's copy of the tiles' first tokens before they are read.  With
# about one tile per wave every tile is its wave's first, and in the larger
# case each wave's tiles span several groups of four.
FILTERED_SMALL_TILES = [
    # (dtype, N, d, B, k)
    ("f16", 2000, 128, 3, 10),     # 4 blocks per tile, one tile per wave
    ("f16", 1500, 32, 2, 5),       # 1 block per tile
    ("f32", 1800, 20, 4, 6),       # fp32, 2 blocks per tile
    ("f16", 150000, 32, 1, 20),    # 1 block per tile, ~9 tiles per wave
]


@pytest.mark.parametrize("dt,N,d,B,k", FILTERED_SMALL_TILES,
                         ids=["%s-N%d-d%d-B%d-k%d" % c for c in FILTERED_SMALL_TILES])
def test_filtered_few_blocks_per_tile(gpu_lib, dt, N, d, B, k):
    say("filtered small tiles", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N + d * 13 + B * 7 + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    src = torch.randint(0, N, (B,), generator=gen)
    q = x[src].to(torch.float64) + 0.05 * torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 4, (N, 3), generator=gen, dtype=torch.int32)  # ~1/4 of rows match
    nt = cont[src, 0].numpy().astype(np.int32)
    rep = run_filtered(x, cont, q, nt, k, dt)
    say("  exact-order rate %.3f" % rep["exact_order_rate"])


# 256-dim keys at two to four query tiles: one shared-key wave per workgroup
# holds every query tile and filters each key tile against all of them.
FILTERED_ONE_WAVE = [
    # (dtype, N, d, B, k)
    ("bf16", 9001, 256, 20, 12),   # two-part bf16 queries, three tiles padded to four
    ("f16", 30011, 256, 64, 32),   # four query tiles
]


@pytest.mark.parametrize("dt,N,d,B,k", FILTERED_ONE_WAVE,
                         ids=["%s-N%d-d%d-B%d-k%d" % c for c in FILTERED_ONE_WAVE])
def test_filtered_one_wave_shared_key(gpu_lib, dt, N, d, B, k):
    from paper_2502_15572_amd import Index
    say("filtered one-wave shared-key", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N + d * 19 + B * 5 + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    src = torch.randint(0, N, (B,), generator=gen)
    q = x[src].to(torch.float64) + 0.05 * torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 4, (N, 3), generator=gen, dtype=torch.int32)  # ~1/4 of rows match
    nt = cont[src, 0].numpy().astype(np.int32)
    nt[2::5] = NO_ROW_TOKEN
    ix = Index(x.to(DEV), cont.to(DEV))
    assert ix.plan(B, k)["scan_kernel"] == "shared_key"
    ix.close()
    rep = run_filtered(x, cont, q, nt, k, dt)
    say("  exact-order rate %.3f" % rep["exact_order_rate"])


def test_filtered_all_rows_match_equals_unfiltered(gpu_lib):
    """A token every row starts with filters nothing: same result as the
    unfiltered search, bit for bit (shared-key scan and sampled passes)."""
    say("filtered all-match")
    w = WORKLOADS["batch10m_d256_f16"].scaled(60000)
    g = generate(w, "cpu")
    cont = g["cont"].clone()
    cont[:, 0] = 5
    from paper_2502_15572_amd import Index
    ix = Index(g["keys"].to(DEV), cont.to(DEV))
    q = g["queries"][:100].to(DEV)
    a = ix.search(q, w.k)
    b = ix.search(q, w.k, next_tok=torch.full((100,), 5, dtype=torch.int32, device=DEV))
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    ix.close()


# Keys of more than 1,024 dims at batches of two or more query tiles take the
# tiled contraction; its filtered form tests each panel's rows against the
# slots' next tokens, and its sampled pass (per-tile maxima) skips the rows
# the filter drops.
FILTERED_TILED = [
    # (dtype, N, d, B, k)
    ("bf16", 20000, 4096, 64, 10),   # 8 query tiles, sampled pass at stride 16
    ("f16", 30000, 2048, 40, 16),    # f16, 4 query tiles (8 waves, per-wave copy counts)
    ("bf16", 3001, 1100, 33, 12),    # ragged columns, no sampled pass
    ("f16", 20011, 1024, 200, 12),   # four query groups (8 key tiles per wave)
    ("bf16", 5003, 4096, 100, 10),   # two query groups
    ("f16", 7001, 2048, 256, 64),    # four query groups, three-stage ring (the filter's LDS)
    ("bf16", 4001, 1024, 128, 32),   # 1,024-dim bf16 keys, two query groups
]


@pytest.mark.parametrize("dt,N,d,B,k", FILTERED_TILED,
                         ids=["%s-N%d-d%d-B%d-k%d" % c for c in FILTERED_TILED])
def test_filtered_tiled_contraction(gpu_lib, dt, N, d, B, k):
    from paper_2502_15572_amd import Index
    say("filtered tiled", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N + d * 17 + B * 3 + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    src = torch.randint(0, N, (B,), generator=gen)
    q = x[src].to(torch.float64) + 0.05 * torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 4, (N, 3), generator=gen, dtype=torch.int32)  # ~1/4 of rows match
    nt = cont[src, 0].numpy().astype(np.int32)
    nt[3::4] = NO_ROW_TOKEN
    ix = Index(x.to(DEV), cont.to(DEV))
    assert ix.plan(B, k)["scan_kernel"] == "tiled"
    ix.close()
    rep = run_filtered(x, cont, q, nt, k, dt)
    say("  exact-order rate %.3f" % rep["exact_order_rate"])


def test_filtered_tiled_all_rows_match_equals_unfiltered(gpu_lib):
    """The tiled contraction's filtered form with a token every row starts
    with returns the unfiltered result bit for bit."""
    from paper_2502_15572_amd import Index
    say("filtered tiled all-match")
    gen = torch.Generator().manual_seed(77)
    N, d, B, k = 20000, 4096, 64, 10
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(torch.bfloat16)
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32).to(DEV)
    cont = torch.full((N, 2), 5, dtype=torch.int32)
    ix = Index(x.to(DEV), cont.to(DEV))
    a = ix.search(q, k)
    b = ix.search(q, k, next_tok=torch.full((B,), 5, dtype=torch.int32, device=DEV))
    for u, v in zip(a, b):
        assert torch.equal(u, v)
    ix.close()
