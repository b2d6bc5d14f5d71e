"""Parity of the HIP path (through the C ABI) against the CPU oracle.

Sizes are chosen so the oracle finishes in seconds while the device path
still spans many 16-row tiles, a ragged last tile, several sampled threshold
passes and several waves.  Scores must agree within 1e-5 (fp32 keys) or
2e-3 (16-bit keys); index sets may differ only where the oracle's rank-k and
rank-(k+1) scores are closer than that; tokens must be bit-exact.
"""
import json
import os
import sys

import numpy as np
import pytest
import torch

import oracle
from datagen import WORKLOADS, generate, to_numpy_bits
from parity import TOL, check_batch, check_operand_model

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")
DEV = "cuda:0"
_TD = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_case(gpu_lib, keys, cont, queries, k, dtype, tol=None, strict_report=False, kind=None):
    """Search on the GPU and check against the oracle.  keys/cont/queries are
    torch tensors (any device); `kind`: the scan kernel the plan must pick."""
    from paper_2502_15572_amd import Index
    kd = keys.to(DEV)
    ix = Index(kd, cont.to(DEV))
    q = queries.to(DEV, torch.float32)
    if kind is not None:
        assert ix.plan(q.shape[0], k)["scan_kernel"] == kind
    idx, score, tok = ix.search(q, k)
    torch.cuda.synchronize()
    g_idx, g_score, g_tok = idx.cpu().numpy(), score.cpu().numpy(), tok.cpu().numpy()
    kb, dt = to_numpy_bits(keys)
    qn = queries.cpu().numpy().astype(np.float32)
    cn = cont.cpu().numpy()
    o_idx, o_score, _, o_next = oracle.topk(kb, dt, qn, k, cn)
    rep = check_batch(g_idx, g_score, g_tok, o_idx, o_score, o_next,
                      lambda b, rows: oracle.score_rows(kb, dt, qn[b], rows), kb.shape[0], cn,
                      TOL[dt] if tol is None else tol)
    # every returned score against the documented operand precision
    B = qn.shape[0]
    for b in range(B):
        dm, de, mode = check_operand_model(
            g_idx[b], g_score[b], qn[b], B, dt, lambda r: oracle.decode_keys(kb[r], dt),
            lambda qq, r: oracle.score_rows(kb, dt, qq, r))
        rep["max_abs_vs_model"] = max(rep.get("max_abs_vs_model", 0.0), dm)
        rep["operand"] = mode
    ix.close()
    return rep, (g_idx, g_score, g_tok)


def test_golden_closed_forms_on_gpu(gpu_lib):
    """Hand-derived rankings over a standard-basis datastore, exact equality."""
    cases = json.load(open(GOLDEN))["cases"]
    from paper_2502_15572_amd import Index
    for c in cases:
        for dt in ("f32", "f16", "bf16"):
            say("golden", c["name"], dt)
            keys = torch.eye(c["N"], c["d"], dtype=_TD[dt], device=DEV)
            cont = torch.arange(c["N"] * 3, dtype=torch.int32, device=DEV).view(c["N"], 3)
            q = torch.zeros(1, c["d"], dtype=torch.float32)
            for j, v in c["query"].items():
                q[0, int(j)] = float(np.float32(v))
            ix = Index(keys, cont)
            idx, score, tok = ix.search(q.to(DEV), c["k"])
            assert idx[0].tolist() == c["idx"], (c["name"], dt, idx[0].tolist())
            want = np.asarray(c["score"], np.float32)
            assert np.array_equal(score[0].cpu().numpy(), want), (c["name"], dt, score)
            assert torch.equal(tok[0].cpu(), cont.cpu()[torch.tensor(c["idx"])])
            ix.close()


REDUCED = [
    ("flat16k_d256_f32", 16384, None),
    ("hidden1m_d4096_bf16", 6000 + 5, None),
    ("pca4m_d1024_f16", 40000 + 3, None),
    ("batch10m_d256_f16", 120000 + 9, None),
    ("zipf33m_d128_f16", 200000 + 11, None),
]


@pytest.mark.parametrize("name,N,_", REDUCED, ids=[r[0] for r in REDUCED])
def test_workload_parity_reduced(gpu_lib, name, N, _):
    w = WORKLOADS[name].scaled(N)
    g = generate(w, "cpu")
    for B in w.batches:
        say("parity", name, "N=%d B=%d k=%d" % (N, B, w.k))
        rep, _r = run_case(gpu_lib, g["keys"], g["cont"], g["queries"][:B], w.k, w.dtype)
        say("  exact-order rate %.3f, max |g-exact| %.2e, max |g-model| %.2e (%s)"
            % (rep["exact_order_rate"], rep["max_abs_vs_exact"], rep["max_abs_vs_model"],
               rep["operand"]))
        # split-query paths are within summation error of the oracle
        if w.dtype in ("f32", "bf16") or B <= 4:
            assert rep["max_abs_vs_exact"] <= 1e-5, rep


EDGE = [
    # (dtype, N, d, B, k)
    ("f16", 1, 32, 1, 1),            # one row, one partial tile
    ("f16", 15, 40, 3, 15),          # k == N inside one ragged tile, ragged dims
    ("bf16", 17, 64, 2, 17),         # two tiles, k == N
    ("f32", 33, 20, 5, 7),           # fp32 keys with ragged dims
    ("f16", 1000, 128, 17, 63),      # B past one query tile (single f16 rounding)
    ("f16", 1000, 128, 4, 64),       # largest split batch
    ("f16", 1000, 128, 8, 64),       # rounded queries, one tile
    ("f16", 3000, 1024, 32, 16),     # two query tiles padded into the shared-key scan
    ("bf16", 2000, 256, 7, 12),      # bf16 over two query tiles: shared-key scan
    ("f16", 5000, 64, 16, 65),
    ("bf16", 3000, 96, 9, 100),      # bf16 split over two query tiles
    ("f16", 4096, 128, 64, 128),
    ("f32", 2000, 256, 4, 1),
    ("f16", 70000, 128, 1, 1000),    # large k
    # lists of 129-256 keys ordered by rank when published (up to four keys
    # per lane), and 257-512 winners ordered by rank in the merge
    ("f16", 150000, 128, 2, 200),
    ("f16", 60000, 128, 3, 400),
    ("bf16", 9000, 256, 32, 16),
    # many queries per single-tile launch: up to 16 passing rows of a tile
    # for one query must fit the query's LDS stage
    ("f32", 50, 256, 33, 4),         # fp32, three query tiles
    ("f32", 5000, 64, 100, 20),      # fp32, seven query tiles
    ("f16", 3000, 2048, 40, 10),     # f16 blocks per tile outside the shared-key scan
    ("bf16", 2000, 2048, 64, 8),     # bf16 (three-part queries), sixteen query tiles
    # d = 4096 bf16: 8 queries per single-tile group, several groups per
    # launch (workgroups of one key range placed on one XCD when the ranges
    # are a multiple of 8, else in plain order)
    ("bf16", 20000, 4096, 64, 10),   # 8 groups, one launch, 256 ranges
    ("bf16", 3001, 4096, 70, 12),    # 9 groups: two launches of 5, 47 ranges
    ("f16", 9000, 4096, 19, 40),     # f16 at one column: 3 groups of 6-7
    # the largest d (16384): one query operand nearly fills the LDS, so
    # batches split into groups of one or two queries
    ("bf16", 300, 16384, 1, 5),
    ("f16", 300, 16384, 2, 5),
    ("f32", 200, 16384, 3, 4),
]


@pytest.mark.parametrize("dt,N,d,B,k", EDGE, ids=["%s-N%d-d%d-B%d-k%d" % e for e in EDGE])
def test_edge_shapes(gpu_lib, dt, N, d, B, k):
    say("edge", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N * 7 + d * 3 + B + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 32000, (N, 4), generator=gen, dtype=torch.int32)
    run_case(gpu_lib, x, cont, q, k, dt)


# Batches of several 16-column query tiles take the shared-key scan (queries
# in registers, keys staged through LDS): cover every (query tiles per wave,
# blocks per key tile) class it has, ragged batches and dims, fewer key tiles
# than workgroups, k = 1 and large k (list cuts), and both key types.
MQ_EDGE = [
    # (dtype, N, d, B, k)
    ("f16", 777, 128, 50, 10),        # 49 tiles: fewer tiles than workgroups
    ("f16", 9999, 128, 64, 1),        # k = 1
    ("f16", 12345, 100, 256, 50),     # ragged dims, 4 tiles per wave, 4 blocks per tile
    ("f16", 20011, 512, 100, 32),     # 16 blocks per tile
    ("f16", 30001, 1024, 64, 16),     # 32 blocks per tile
    ("bf16", 15013, 256, 64, 40),     # three-part bf16 queries, 4 tiles per wave
    ("bf16", 7001, 128, 13, 9),       # smallest bf16 batch that fills 4 query tiles
    ("f16", 40009, 256, 200, 1000),   # large k: lists cut to k many times
    ("f16", 100, 128, 40, 100),       # k == N: every row returned, in order
    ("bf16", 999, 64, 8, 999),        # k == N, two padded query tiles
    ("f16", 5000, 128, 600, 20),      # three groups of 256 queries
    ("f16", 90001, 128, 24, 300),     # published lists past 256 keys, 300 winners
    # 256-dim keys at 2-4 query tiles: one wave per workgroup holds the batch
    ("f16", 30011, 256, 64, 32),      # four query tiles
    ("f16", 5003, 256, 20, 7),        # two query tiles padded to four
    ("bf16", 8191, 256, 32, 16),      # bf16 two-part queries, four tiles
    ("f16", 300, 256, 48, 100),       # 19 key tiles, fewer than workgroups; k near N
]


@pytest.mark.parametrize("dt,N,d,B,k", MQ_EDGE, ids=["%s-N%d-d%d-B%d-k%d" % e for e in MQ_EDGE])
def test_shared_key_scan_shapes(gpu_lib, dt, N, d, B, k):
    say("shared-key", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N * 5 + d * 11 + B + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 32000, (N, 3), generator=gen, dtype=torch.int32)
    run_case(gpu_lib, x, cont, q, k, dt)


# Keys of more than 1,024 dims at batches of two or more query tiles take the
# tiled contraction (key and query blocks both streamed through LDS): the
# smallest padded batch, ragged dims and column counts just past the
# shared-key scan's, f16 and bf16 operand layouts, fewer key tiles than one
# panel, k == N, large k (the shallower LDS rings), and batches split over
# several launches.
TC_EDGE = [
    # (dtype, N, d, B, k)
    ("bf16", 5003, 4096, 9, 10),      # two query tiles padded to four
    ("bf16", 4099, 1050, 33, 20),     # 33 columns, the last ragged; eight query tiles
    ("f16", 7001, 1600, 64, 5),       # f16, four query tiles of 16 queries
    ("bf16", 2000, 4096, 64, 1000),   # large k: three- and four-stage rings
    ("bf16", 100, 4096, 40, 100),     # 7 key tiles (less than a panel), k == N
    ("f16", 33000, 2048, 130, 16),    # three launches of 43-44 queries
    ("bf16", 16411, 4096, 17, 64),
    # sampled threshold passes (per-tile maxima) at strides 64, 16 and 4
    ("bf16", 40000, 1100, 20, 2),     # stride 64, 35 columns (ragged)
    ("f16", 30000, 2048, 64, 4),      # stride 64
    ("bf16", 20000, 4096, 64, 10),    # stride 16
    ("bf16", 6000, 2048, 50, 16),     # stride 4
    ("bf16", 256003, 1100, 20, 1000),  # stride 4 at large k: the shallow rings of both passes
]


@pytest.mark.parametrize("dt,N,d,B,k", TC_EDGE, ids=["%s-N%d-d%d-B%d-k%d" % e for e in TC_EDGE])
def test_tiled_contraction_shapes(gpu_lib, dt, N, d, B, k):
    say("tiled", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N * 3 + d * 13 + B + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 32000, (N, 3), generator=gen, dtype=torch.int32)
    rep, _r = run_case(gpu_lib, x, cont, q, k, dt, kind="tiled")
    say("  max |g-exact| %.2e, max |g-model| %.2e (%s)"
        % (rep["max_abs_vs_exact"], rep["max_abs_vs_model"], rep["operand"]))


TC_GROUPS = [
    # (dtype, N, d, B, k, launches): batches past one query group of waves
    ("f16", 20011, 1024, 130, 16, 1),   # four query groups, the last past the batch
    ("f16", 9001, 1024, 256, 32, 1),    # four query groups, all full
    ("f16", 12007, 1024, 100, 10, 1),   # two query groups
    ("f16", 6007, 2048, 256, 100, 1),   # four query groups at larger lists
    ("f16", 100, 1024, 200, 50, 1),     # 7 key tiles, less than a 16-tile panel
    ("bf16", 9001, 1024, 40, 16, 1),    # 1,024 dims, one group of 8 query tiles
    ("bf16", 7001, 1024, 128, 8, 1),    # two query groups of 8 tiles
    ("bf16", 5003, 4096, 100, 10, 1),   # two query groups
    ("bf16", 3001, 4096, 256, 10, 2),   # two launches of 128 queries
    ("f16", 4001, 1024, 256, 1000, 4),  # lists too large for query groups: one group per launch
]


@pytest.mark.parametrize("dt,N,d,B,k,nl", TC_GROUPS,
                         ids=["%s-N%d-d%d-B%d-k%d" % e[:5] for e in TC_GROUPS])
def test_tiled_contraction_query_groups(gpu_lib, dt, N, d, B, k, nl):
    from paper_2502_15572_amd import Index
    say("tiled groups", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N * 7 + d + B * 5 + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 32000, (N, 2), generator=gen, dtype=torch.int32)
    ix = Index(x.to(DEV), cont.to(DEV))
    assert ix.plan(B, k)["launches"] == nl
    ix.close()
    run_case(gpu_lib, x, cont, q, k, dt, kind="tiled")


def _random_group_cases(n, seed):
    """Seeded random shapes past one query group: dims from 1,024 (1,024-dim
    keys take the contraction past 64 f16 / 32 bf16 queries), 33-256
    queries, k from 1 to 128."""
    import random
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        dt = rng.choice(["bf16", "f16"])
        d = rng.choice([1024, 1056, 2048, 3000, 4096])
        B = rng.randint(33 if (dt == "bf16" and d == 1024) else 65, 256)
        k = rng.choice([1, 7, 16, 50, 128])
        N = rng.randint(max(k, 500), 20000)
        if N * d * B <= 3e9:
            out.append((dt, N, d, B, k))
    return out


TC_GROUPS_RANDOM = _random_group_cases(8, 77)


@pytest.mark.parametrize("dt,N,d,B,k", TC_GROUPS_RANDOM,
                         ids=["%s-N%d-d%d-B%d-k%d" % e for e in TC_GROUPS_RANDOM])
def test_tiled_contraction_random_groups(gpu_lib, dt, N, d, B, k):
    say("tiled random groups", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N * 5 + d + B + k * 3)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 32000, (N, 2), generator=gen, dtype=torch.int32)
    run_case(gpu_lib, x, cont, q, k, dt, kind="tiled")


def _random_tiled_cases(n, seed):
    """Seeded random shapes for the tiled contraction: dims past 1,024 (ragged
    column counts included), 9-140 queries (one to three launches), k from 1
    to 257, and as many rows as keep the oracle to a few seconds."""
    import random
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        dt = rng.choice(["bf16", "f16"])
        d = rng.choice([1056, 1200, 1536, 2048, 2500, 3072, 4096])
        B = rng.randint(9 if dt == "bf16" else 17, 140)
        k = rng.choice([1, 3, 10, 33, 100, 257])
        N = rng.randint(max(k, 300), 30000)
        if N * d * B <= 2.5e9:
            out.append((dt, N, d, B, k))
    return out


TC_RANDOM = _random_tiled_cases(8, 2025)


@pytest.mark.parametrize("dt,N,d,B,k", TC_RANDOM, ids=["%s-N%d-d%d-B%d-k%d" % e for e in TC_RANDOM])
def test_tiled_contraction_random_shapes(gpu_lib, dt, N, d, B, k):
    say("tiled random", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N + d + B * 31 + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 32000, (N, 2), generator=gen, dtype=torch.int32)
    run_case(gpu_lib, x, cont, q, k, dt, kind="tiled")


def _random_ladder_cases(n, seed):
    """Seeded random shapes for the shared-key scan with two or three
    sampled passes, so that a pass starts from the previous one's
    speculative key: the dense ladder (B*k >= 8192: strides 256 and 16,
    and 4096 once the datastore has 16,384 tiles) and the sparse one
    (strides 4096 and 64, at least 16,384 tiles), ragged row counts, f16 and
    bf16, k up to 250."""
    import random
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        dt = rng.choice(["f16", "bf16"])
        dense = len(out) % 2 == 0
        if dense:
            d = [256, 512, 128, 256][len(out) // 2 % 4]
            B = rng.randint(64, 256 if dt == "f16" else 128)
            k = rng.choice([32, 64, 100, 250])
            if B * k < 8192:
                continue
            N = rng.randint(1024 * 16, 300000)
            if k > (N // 16 // 256) * 4:
                continue
        else:
            d = 128
            B = rng.randint(17, 60)
            k = rng.choice([5, 10, 16, 20])
            if B * k >= 8192:
                continue
            N = rng.randint(16384 * 16 + 1, 330000)
        if N * d * B <= 6e9:
            out.append((dt, N, d, B, k))
    return out


LADDER_RANDOM = _random_ladder_cases(8, 77)


@pytest.mark.parametrize("dt,N,d,B,k", LADDER_RANDOM,
                         ids=["%s-N%d-d%d-B%d-k%d" % e for e in LADDER_RANDOM])
def test_shared_key_sampled_ladders(gpu_lib, dt, N, d, B, k):
    say("ladder random", dt, N, d, B, k)
    gen = torch.Generator().manual_seed(N + d * 7 + B * 13 + k)
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(_TD[dt])
    src = torch.randint(0, N, (B,), generator=gen)
    q = x[src].to(torch.float64) + 0.3 * torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 32000, (N, 2), generator=gen, dtype=torch.int32)
    from paper_2502_15572_amd import Index
    ix = Index(x.to(DEV), cont.to(DEV))
    pl = ix.plan(B, k)
    ix.close()
    say("  plan", pl)
    assert pl["scan_kernel"] == "shared_key" and pl["sample_passes"] >= 2, pl
    run_case(gpu_lib, x, cont, q, k, dt)


def test_grouped_launch_matches_split_batches(gpu_lib):
    """A batch whose single-tile groups share one launch returns, bit for
    bit, what the same queries return as separate batches of one group each
    (the answer is unique: every key names its row)."""
    say("grouped vs split")
    gen = torch.Generator().manual_seed(4096)
    N, d, B, k = 20011, 4096, 40, 16
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(torch.bfloat16)
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 32000, (N, 2), generator=gen, dtype=torch.int32)
    from paper_2502_15572_amd import Index
    ix = Index(x.to(DEV), cont.to(DEV))
    qd = q.to(DEV)
    whole = ix.search(qd, k)
    parts = [ix.search(qd[b:b + 8].contiguous(), k) for b in range(0, B, 8)]
    torch.cuda.synchronize()
    for i, w in enumerate(whole):
        assert torch.equal(w, torch.cat([p[i] for p in parts]))
    ix.close()


def test_shared_key_scan_all_scores_equal(gpu_lib):
    """Every key identical: every score passes every float threshold, so the
    candidate buffers overflow on every tile; the result must still be the
    k lowest rows."""
    say("all-equal")
    gen = torch.Generator().manual_seed(11)
    N, d, B, k = 5003, 128, 64, 20
    v = torch.randn(d, generator=gen, dtype=torch.float64)
    x = (v / v.norm()).to(torch.float16).expand(N, d).contiguous()
    q = torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.arange(N * 2, dtype=torch.int32).view(N, 2)
    rep, (gi, gs, gt) = run_case(gpu_lib, x, cont, q, k, "f16")
    assert (gi == np.arange(k)[None, :]).all()


@pytest.mark.parametrize("period", [256, 4096])
def test_sampled_pass_fallback_to_exact_bound(gpu_lib, period):
    """Each sampled pass after the first starts from a speculative key (the
    j-th best of the sparser sample, j < k).  Here every high-scoring row
    lies in tiles at multiples of `period`, i.e. inside the sparser samples
    only, so the denser passes find fewer than k keys at or above that key
    (the last pass at period 256; both at 4096) and have to keep the exact
    bound they started from.  The result must still be the exact top-k."""
    say("sampled fallback", period)
    N, d, B, k = 61441 * 16, 128, 128, 64  # 3 sampled passes: 4096 holds 16 tiles = 4k rows
    gen = torch.Generator().manual_seed(period)
    u = torch.randn(d, generator=gen, dtype=torch.float64)
    u = u / u.norm()
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    tile = torch.arange(N) // 16
    high = tile % period == 0
    x[high] = u + 0.03 * x[high]
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).to(torch.float16)
    q = u + 0.03 * torch.randn(B, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    # every high row outscores every other row, for every query
    sc = x.float() @ q.T
    assert sc[high].min() > sc[~high].max() + 0.1
    assert int(high.sum()) >= k
    del sc
    cont = torch.randint(0, 32000, (N, 2), generator=gen, dtype=torch.int32)
    from paper_2502_15572_amd import Index
    ix = Index(x.to(DEV), cont.to(DEV))
    pl = ix.plan(B, k)
    ix.close()
    assert pl["scan_kernel"] == "shared_key" and pl["sample_passes"] == 3, pl
    rep, (gi, _, _) = run_case(gpu_lib, x, cont, q, k, "f16")
    assert high[torch.from_numpy(gi).flatten()].all()


def test_all_negative_scores_never_return_padding(gpu_lib):
    """Keys in one half-space, queries in the other: every score is negative,
    so zero-scoring padding rows of the last tile would win if not masked."""
    say("all-negative")
    gen = torch.Generator().manual_seed(3)
    N, d = 1003, 64
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x[:, 0] = x[:, 0].abs() + 1.0
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float16)
    q = torch.zeros(4, d)
    q[:, 0] = -1.0
    cont = torch.arange(N * 2, dtype=torch.int32).view(N, 2)
    rep, (gi, gs, gt) = run_case(gpu_lib, x, cont, q, 20, "f16")
    assert (gs < 0).all() and (gi < N).all()


def test_duplicates_resolve_to_lowest_index(gpu_lib):
    say("duplicates")
    w = WORKLOADS["zipf33m_d128_f16"].scaled(30000)
    g = generate(w, "cpu", planted_duplicates=20)
    rows = [t for _, t in g["duplicates"]]
    q = g["keys"][rows].to(torch.float32)
    rep, (gi, gs, gt) = run_case(gpu_lib, g["keys"], g["cont"], q, 5, "f16")
    for r, (s, t) in enumerate(g["duplicates"]):
        assert gi[r, 0] == s and gi[r, 1] == t and gs[r, 0] == gs[r, 1]


def test_self_retrieval_fp32(gpu_lib):
    """A query equal to an fp32 row returns that row first with score 1 +- 1e-6."""
    say("self-retrieval")
    w = WORKLOADS["flat16k_d256_f32"]
    g = generate(w, "cpu", with_queries=False)
    rows = torch.arange(0, w.N, 61)
    from paper_2502_15572_amd import Index
    ix = Index(g["keys"].to(DEV), g["cont"].to(DEV))
    idx, score, _ = ix.search(g["keys"][rows].to(DEV), 3)
    assert torch.equal(idx[:, 0].cpu(), rows)
    assert float((score[:, 0].double() - 1).abs().max()) <= 1e-6
    ix.close()


def test_determinism_and_stream_reuse(gpu_lib):
    say("determinism")
    w = WORKLOADS["batch10m_d256_f16"].scaled(150000)
    g = generate(w, "cpu")
    from paper_2502_15572_amd import Index
    ix = Index(g["keys"].to(DEV), g["cont"].to(DEV))
    q = g["queries"][:64].to(DEV)
    ref = ix.search(q, w.k)
    s = torch.cuda.Stream()
    for rep in range(5):
        with torch.cuda.stream(s):
            out = ix.search(q, w.k, stream=s)
        s.synchronize()
        for a, b in zip(ref, out):
            assert torch.equal(a, b)
    # a different batch shape in between must not disturb the next result
    ix.search(g["queries"][:3].to(DEV), 7)
    again = ix.search(q, w.k)
    for a, b in zip(ref, again):
        assert torch.equal(a, b)
    ix.close()


def test_argument_errors_on_device(gpu_lib):
    from paper_2502_15572_amd import DresdError, Index
    keys = torch.randn(100, 32, device=DEV).half()
    cont = torch.zeros(100, 2, dtype=torch.int32, device=DEV)
    ix = Index(keys, cont)
    q = torch.randn(2, 32, device=DEV)
    for bad_k in (0, 101, 2000):
        with pytest.raises(DresdError) as e:
            ix.search(q, bad_k)
        assert e.value.status == 1
    out = ix.search(q[:0], 5)  # B == 0 is a no-op
    assert out[0].shape == (0, 5)
    ix.close()


def test_longest_values(gpu_lib):
    """L = 4096 tokens per value (the largest): gathered bit for bit."""
    say("max L")
    gen = torch.Generator().manual_seed(17)
    N, d, L = 200, 64, 4096
    x = torch.randn(N, d, generator=gen, dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float16)
    q = torch.randn(3, d, generator=gen, dtype=torch.float64)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.float32)
    cont = torch.randint(0, 2 ** 31 - 1, (N, L), generator=gen, dtype=torch.int32)
    run_case(gpu_lib, x, cont, q, 7, "f16")
