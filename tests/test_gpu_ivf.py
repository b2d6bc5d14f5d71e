"""Parity of the partitioned (inverted-file) search on the GPU with the
oracle's exact top-k over the probed partitions, by the padded-subset rules
of ``parity.py`` (scores within 1e-5 for fp32 keys, 2e-3 for 16-bit keys;
index sets equal up to near-ties at rank k; tokens bit-exact; every returned
row from a probed partition; padding exactly where the oracle pads).

Inputs: reduced Zipf-clustered and isotropic workloads; partitions from a few
oracle k-means steps (fp64) started from seeded rows, assignments by the
oracle, probes either chosen by the oracle (exact top-nprobe over the
centroids; only queries whose nprobe-th and next centroid scores differ by
at least 1e-5, so the probed set is unique) or seeded random lists with
repeats and out-of-range ids.  Edge cases: every partition probed (equals the
exact search), fewer probed rows than k, empty partitions, k = 1024, one
query and many, d spanning several blocks with a ragged tail."""
import sys

import dataclasses

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
    sys.stdout.flush()


def partitions(kb, dt, P, seed, iters=3):
    """Oracle spherical k-means: centroids [P, d] f32, assignment [N] int32."""
    x = oracle.decode_keys(kb, dt)
    rng = np.random.default_rng(seed)
    c = x[rng.choice(x.shape[0], P, replace=False)]
    for _ in range(iters):
        a, _, _ = oracle.kmeans_assign(x, c)
        c = oracle.kmeans_update(x, a, c)
    c32 = c.astype(np.float32)
    a, _, _ = oracle.kmeans_assign(x, c32.astype(np.float64))
    return c32, a


def make(name, n, P, seed=0):
    w = WORKLOADS[name].scaled(n)
    g = generate(w, "cpu", seed=seed)
    keys, cont, q = g["keys"], g["cont"], g["queries"]
    kb, dt = to_numpy_bits(keys)
    c, a = partitions(kb, dt, P, seed + 1)
    return keys, cont, q, kb, dt, c, a


def check(g, kb, dt, qn, cn, a, probes, k, P, next_tok=None):
    g_idx, g_score, g_tok = (t.cpu().numpy() for t in g)
    o_idx, o_score, _, o_next = oracle.topk_partitioned(kb, dt, qn, k, a, P, probes, cn,
                                                        next_tok=next_tok)
    sets = [set(int(p) for p in row if 0 <= p < P) for row in probes]

    def admitted(b, rows):
        ok = np.isin(a[rows], list(sets[b]))
        if next_tok is not None:
            ok &= cn[rows, 0] == next_tok[b]
        return ok
    return check_batch(g_idx, g_score, g_tok, o_idx, o_score, o_next,
                       lambda b, rows: oracle.score_rows(kb, dt, qn[b], rows), kb.shape[0], cn,
                       TOL[dt], admitted_b=admitted)


CASES = [
    # workload, rows, partitions, batch, k, probes per query
    ("zipf33m_d128_f16", 30000 + 7, 64, 8, 100, 6),
    ("batch10m_d256_f16", 20000 + 3, 50, 33, 32, 4),
    ("hidden1m_d4096_bf16", 3000 + 5, 12, 4, 10, 3),
    ("flat16k_d256_f32", 16384, 40, 8, 10, 5),
]


@pytest.mark.parametrize("name,n,P,B,k,S", CASES, ids=[c[0] for c in CASES])
def test_ivf_search_probes_random(gpu_lib, name, n, P, B, k, S):
    from paper_2502_15572_amd import PartitionedIndex
    say("ivf probes", name, n, P, B, k, S)
    keys, cont, q, kb, dt, c, a = make(name, n, P)
    rng = np.random.default_rng(7)
    probes = rng.integers(-2, P + 2, (B, S)).astype(np.int32)
    probes[:, -1] = probes[:, 0]  # a repeat in every list
    ix = PartitionedIndex(keys.to(DEV), cont.to(DEV), torch.from_numpy(c).to(DEV),
                          torch.from_numpy(a).to(DEV))
    qd = q[:B].to(DEV)
    g = ix.search_probes(qd, torch.from_numpy(probes).to(DEV), k)
    torch.cuda.synchronize()
    check(g, kb, dt, q[:B].numpy(), cont.numpy(), a, probes, k, P)
    # deterministic
    g2 = ix.search_probes(qd, torch.from_numpy(probes).to(DEV), k)
    assert all(torch.equal(x, y) for x, y in zip(g, g2))
    ix.close()


@pytest.mark.parametrize("name,n,P,B,k,S", CASES, ids=[c[0] for c in CASES])
def test_ivf_search_oracle_probes(gpu_lib, name, n, P, B, k, S):
    """Internal probing (exact top-nprobe over the centroids) against the
    oracle's probes, on queries whose probed set is unique."""
    from paper_2502_15572_amd import PartitionedIndex
    say("ivf search", name, n, P, B, k, S)
    keys, cont, q, kb, dt, c, a = make(name, n, P)
    qn = q[:B].numpy()
    p_idx, p_sc, _, _ = oracle.topk(c, "f32", qn, min(S + 1, P))
    unique = (p_sc[:, S - 1] - p_sc[:, S] >= 1e-5) if S < P else np.ones(B, bool)
    assert unique.mean() >= 0.5
    probes = p_idx[:, :S].astype(np.int32)
    ix = PartitionedIndex(keys.to(DEV), cont.to(DEV), torch.from_numpy(c).to(DEV),
                          torch.from_numpy(a).to(DEV))
    g = ix.search(q[:B].to(DEV), k, S)
    torch.cuda.synchronize()
    sel = np.nonzero(unique)[0]
    gs = tuple(t[torch.from_numpy(sel)] for t in g)
    check(gs, kb, dt, qn[sel], cont.numpy(), a, probes[sel], k, P)
    ix.close()


# Internal probing (the exact search over the centroid index) at more shapes:
# centroid sets past one workgroup's 512 rows with a ragged end, 1, 64 and 65
# probes, and dims that are not a multiple of 4.
PROBE_CASES = [
    # workload, rows, partitions, batch, k, probes per query, dims (0: the workload's)
    ("zipf33m_d128_f16", 20000 + 11, 1500, 6, 50, 64, 0),
    ("zipf33m_d128_f16", 20000 + 11, 1500, 6, 50, 1, 0),
    ("zipf33m_d128_f16", 20000 + 11, 1500, 6, 50, 65, 0),
    ("batch10m_d256_f16", 9000 + 1, 700, 5, 20, 17, 50),
]


@pytest.mark.parametrize("name,n,P,B,k,S,d", PROBE_CASES,
                         ids=["P%d-S%d-d%d" % (c[2], c[5], c[6]) for c in PROBE_CASES])
def test_ivf_probe_paths(gpu_lib, name, n, P, B, k, S, d):
    from paper_2502_15572_amd import PartitionedIndex
    say("ivf probe path", name, n, P, B, k, S, d)
    w = WORKLOADS[name].scaled(n)
    if d:
        w = dataclasses.replace(w, d=d)
    g = generate(w, "cpu", seed=3)
    keys, cont, q = g["keys"], g["cont"], g["queries"]
    kb, dt = to_numpy_bits(keys)
    c, a = partitions(kb, dt, P, 4, iters=1)
    qn = q[:B].numpy()
    p_idx, p_sc, _, _ = oracle.topk(c, "f32", qn, S + 1)
    unique = p_sc[:, S - 1] - p_sc[:, S] >= 1e-5
    assert unique.mean() >= 0.5
    ix = PartitionedIndex(keys.to(DEV), cont.to(DEV), torch.from_numpy(c).to(DEV),
                          torch.from_numpy(a).to(DEV))
    for rep in range(2):  # the second search reuses the index's probe buffers
        res = ix.search(q[:B].to(DEV), k, S)
        torch.cuda.synchronize()
        sel = np.nonzero(unique)[0]
        gs = tuple(t[torch.from_numpy(sel)] for t in res)
        check(gs, kb, dt, qn[sel], cont.numpy(), a, p_idx[sel, :S].astype(np.int32), k, P)
    ix.close()


def test_ivf_all_partitions_is_exact_search(gpu_lib):
    """Probing every partition returns the exact search's answer."""
    from paper_2502_15572_amd import PartitionedIndex
    from parity import check_batch as cb
    keys, cont, q, kb, dt, c, a = make("zipf33m_d128_f16", 12000 + 1, 20)
    say("ivf all partitions")
    ix = PartitionedIndex(keys.to(DEV), cont.to(DEV), torch.from_numpy(c).to(DEV),
                          torch.from_numpy(a).to(DEV))
    qn = q[:16].numpy()
    g = ix.search(q[:16].to(DEV), 50, 20)
    torch.cuda.synchronize()
    o_idx, o_score, _, o_next = oracle.topk(kb, dt, qn, 50, cont.numpy())
    cb(*(t.cpu().numpy() for t in g), o_idx, o_score, o_next,
       lambda b, rows: oracle.score_rows(kb, dt, qn[b], rows), kb.shape[0], cont.numpy(), TOL[dt])
    ix.close()


def test_ivf_edges(gpu_lib):
    """Fewer probed rows than k (padding), empty partitions, k = 1024, one
    query, an all-invalid probe list, ragged d."""
    from paper_2502_15572_amd import PartitionedIndex
    rng = np.random.default_rng(11)
    N, d, P = 5000, 100, 30
    x = rng.standard_normal((N, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    keys = torch.from_numpy(x.astype(np.float16))
    kb, dt = to_numpy_bits(keys)
    cont = torch.from_numpy(rng.integers(0, 1000, (N, 4)).astype(np.int32))
    # skewed assignment with empty partitions 3, 17, 29 and a one-row partition 5
    a = rng.integers(0, P, N).astype(np.int32)
    a[np.isin(a, [3, 17, 29])] = 0
    a[a == 5] = 6
    a[123] = 5
    c = rng.standard_normal((P, d))
    c = (c / np.linalg.norm(c, axis=1, keepdims=True)).astype(np.float32)
    ix = PartitionedIndex(keys.to(DEV), cont.to(DEV), torch.from_numpy(c).to(DEV),
                          torch.from_numpy(a).to(DEV))
    info = ix.info()
    assert info["P"] == P and info["N"] == N
    q = rng.standard_normal((5, d))
    q = (q / np.linalg.norm(q, axis=1, keepdims=True)).astype(np.float32)
    probes = np.array([[5, 3, -1], [3, 17, 29], [5, 5, 6], [0, 1, 2], [99, -7, 4]], np.int32)
    for k in (1, 7, 300, 1024):
        say("ivf edges k", k)
        g = ix.search_probes(torch.from_numpy(q).to(DEV), torch.from_numpy(probes).to(DEV), k)
        torch.cuda.synchronize()
        check(g, kb, dt, q, cont.numpy(), a, probes, k, P)
        if k >= 2:
            assert g[0][1, 0].item() == -1  # only empty partitions probed
            assert g[0][0, 0].item() == 123 and g[0][0, 1].item() == -1
    g = ix.search_probes(torch.from_numpy(q[:1]).to(DEV), torch.from_numpy(probes[3:4]).to(DEV), 5)
    torch.cuda.synchronize()
    check(g, kb, dt, q[:1], cont.numpy(), a, probes[3:4], 5, P)
    ix.close()


@pytest.mark.parametrize("name,n,P,B,k,S", CASES[:3], ids=[c[0] for c in CASES[:3]])
def test_ivf_filtered(gpu_lib, name, n, P, B, k, S):
    """Next-token filter over the probed partitions (Section 3.5): each
    query's next token is its source row's first token, a frequent token, or
    one that starts no value; caller probes and internal probing."""
    from paper_2502_15572_amd import PartitionedIndex
    say("ivf filtered", name, n, P, B, k, S)
    keys, cont, q, kb, dt, c, a = make(name, n, P)
    g = generate(WORKLOADS[name].scaled(n), "cpu", seed=0)
    cn = cont.numpy()
    src = g["query_src"][:B].numpy()
    freq = int(np.bincount(cn[:, 0]).argmax())
    nt = np.where(src >= 0, cn[np.maximum(src, 0), 0], freq).astype(np.int32)
    nt[1] = freq
    nt[2] = 10 ** 6
    qn = q[:B].numpy()
    ix = PartitionedIndex(keys.to(DEV), cont.to(DEV), torch.from_numpy(c).to(DEV),
                          torch.from_numpy(a).to(DEV))
    rng = np.random.default_rng(3)
    probes = rng.integers(0, P, (B, S)).astype(np.int32)
    ntd = torch.from_numpy(nt).to(DEV)
    gq = ix.search_probes(q[:B].to(DEV), torch.from_numpy(probes).to(DEV), k, next_tok=ntd)
    torch.cuda.synchronize()
    check(gq, kb, dt, qn, cn, a, probes, k, P, next_tok=nt)
    assert (gq[0][2] == -1).all()
    # internal probing, on queries whose probed set is unique
    p_idx, p_sc, _, _ = oracle.topk(c, "f32", qn, min(S + 1, P))
    unique = p_sc[:, S - 1] - p_sc[:, S] >= 1e-5
    gs = ix.search(q[:B].to(DEV), k, S, next_tok=ntd)
    torch.cuda.synchronize()
    sel = np.nonzero(unique)[0]
    check(tuple(t[torch.from_numpy(sel)] for t in gs), kb, dt, qn[sel], cn, a,
          p_idx[sel, :S].astype(np.int32), k, P, next_tok=nt[sel])
    ix.close()
