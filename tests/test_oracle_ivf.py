"""Pins of the partitioned-search and spherical k-means oracles.

The partitioned search is the exact top-k over the rows of the probed
partitions.  It is pinned by its reductions to the exact search (one
partition; every partition probed), by a brute force written out here in fp64
with numpy's lexsort (tiny inputs: repeated and out-of-range probes, empty
probe sets, fewer admitted rows than k), by a closed form on the identity
datastore, and by a planted mistake (a dropped probe) that the reduction pin
catches.  k-means is pinned by closed forms (symmetric pairs, separated
clusters), ties, empty and zero-sum partitions, a pure-Python brute force,
and the monotone objective of spherical k-means."""
import math

import numpy as np
import pytest

import oracle


def unit_rows(rng, n, d, dtype="f32"):
    x = rng.standard_normal((n, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    if dtype == "f16":
        return x.astype(np.float16)
    return x.astype(np.float32)


def brute_partitioned(keys64, q, k, assign, probes, P, L=None, cont=None):
    B = q.shape[0]
    idx = np.full((B, k), -1, np.int64)
    sc = np.full((B, k), -np.inf, np.float32)
    for b in range(B):
        ps = {int(p) for p in probes[b] if 0 <= p < P}
        rows = np.array([i for i in range(keys64.shape[0]) if int(assign[i]) in ps], np.int64)
        if rows.size == 0:
            continue
        s = (keys64[rows] @ q[b].astype(np.float64)).astype(np.float32)
        order = np.lexsort((rows, -s.astype(np.float64)))[:k]
        idx[b, :order.size] = rows[order]
        sc[b, :order.size] = s[order]
    return idx, sc


def test_one_partition_is_the_exact_search():
    rng = np.random.default_rng(0)
    x = unit_rows(rng, 500, 24)
    q = unit_rows(rng, 6, 24)
    cont = rng.integers(0, 100, (500, 3)).astype(np.int32)
    want = oracle.topk(x, "f32", q, 20, cont)
    got = oracle.topk_partitioned(x, "f32", q, 20, np.zeros(500, np.int32), 1,
                                  np.zeros((6, 1), np.int32), cont)
    for w, g in zip(want, got):
        assert np.array_equal(w, g, equal_nan=True)


def test_all_partitions_probed_is_the_exact_search():
    rng = np.random.default_rng(1)
    x = unit_rows(rng, 700, 16, "f16")
    q = unit_rows(rng, 5, 16)
    assign = rng.integers(0, 7, 700).astype(np.int32)
    probes = np.array([rng.permutation(7) for _ in range(5)], np.int32)
    want = oracle.topk(x, "f16", q, 30)
    got = oracle.topk_partitioned(x, "f16", q, 30, assign, 7, probes)
    assert np.array_equal(want[0], got[0]) and np.array_equal(want[1], got[1])
    with oracle.mutation(9):  # a dropped probe is caught by this pin
        bad = oracle.topk_partitioned(x, "f16", q, 30, assign, 7, probes)
    assert not np.array_equal(want[0], bad[0])


@pytest.mark.parametrize("seed", [2, 3, 4])
def test_partitioned_brute_force(seed):
    rng = np.random.default_rng(seed)
    N, d, P, k = 90, 8, 6, 12
    x = unit_rows(rng, N, d)
    # a repeated row makes equal scores, broken by the lower row
    x[40] = x[7]
    assign = rng.integers(0, P, N).astype(np.int32)
    assign[40] = assign[7]
    q = unit_rows(rng, 5, d)
    q[4] = x[7]
    probes = np.array([[0, 1, -1], [2, 2, 2], [7, -5, 99], [5, 3, 0], [assign[7], 1, 1]],
                      np.int32)
    cont = np.arange(N * 2, dtype=np.int32).reshape(N, 2)
    idx, sc, tok, nxt = oracle.topk_partitioned(x, "f32", q, k, assign, P, probes, cont)
    bi, bs = brute_partitioned(x.astype(np.float64), q, k, assign, probes, P)
    assert np.array_equal(idx, bi)
    assert np.array_equal(sc, bs)
    # gathered tokens decode back to the row; padding is zero
    for b in range(5):
        for r in range(k):
            want = cont[idx[b, r]] if idx[b, r] >= 0 else np.zeros(2, np.int32)
            assert np.array_equal(tok[b, r], want)
    # query 2 probes nothing valid: every rank is padding, no next score
    assert (idx[2] == -1).all() and np.isinf(sc[2]).all() and math.isnan(nxt[2])
    # query 4 is row 7 itself: rank 1 is row 7, then its copy row 40
    assert idx[4, 0] == 7 and idx[4, 1] == 40 and sc[4, 0] == sc[4, 1]


def test_partitioned_identity_closed_form():
    # keys e_0..e_15; row i in partition i % 4; query (e_1 + e_2) / sqrt 2
    N = d = 16
    x = np.eye(N, dtype=np.float32)
    assign = (np.arange(N) % 4).astype(np.int32)
    q = np.zeros((2, d), np.float32)
    q[:, 1] = q[:, 2] = 1 / np.sqrt(2)
    idx, sc, _, _ = oracle.topk_partitioned(x, "f32", q, 4, assign, 4,
                                            np.array([[1], [2, ]], np.int32).reshape(2, 1))
    s = np.float32(1 / np.sqrt(2))
    # partition 1 = rows 1, 5, 9, 13: row 1 scores 1/sqrt2, the rest 0
    assert idx[0].tolist() == [1, 5, 9, 13] and sc[0].tolist() == [s, 0, 0, 0]
    assert idx[1].tolist() == [2, 6, 10, 14] and sc[1].tolist() == [s, 0, 0, 0]
    idx, sc, _, _ = oracle.topk_partitioned(x, "f32", q, 3, assign, 4, np.array([[2, 1]] * 2))
    assert idx[0].tolist() == [1, 2, 5] and sc[0].tolist() == [s, s, 0]


def test_kmeans_assign_brute_force_and_ties():
    rng = np.random.default_rng(5)
    x = oracle.decode_keys(unit_rows(rng, 40, 6, "f16"), "f16")
    c = unit_rows(rng, 5, 6).astype(np.float64)
    c[3] = c[1]  # duplicate centroid: its rows go to the lower id
    a, best, _ = oracle.kmeans_assign(x, c)
    for i in range(40):
        s = [sum(float(x[i, j]) * float(c[p, j]) for j in range(6)) for p in range(5)]
        m = max(s)
        assert a[i] == min(p for p in range(5) if s[p] == m)
        assert best[i] == pytest.approx(m, abs=1e-15)
    assert 3 not in a.tolist()


def test_kmeans_update_closed_forms():
    t = 0.3
    x = np.array([[math.cos(t), math.sin(t)], [math.cos(t), -math.sin(t)],
                  [0.0, 1.0], [0.0, -1.0]])
    old = np.array([[0.6, 0.8], [0.0, 1.0], [-1.0, 0.0]])
    # partition 0: a symmetric pair -> (1, 0); partition 1: x and -x (zero
    # sum) -> unchanged; partition 2: empty -> unchanged
    c = oracle.kmeans_update(x, [0, 0, 1, 1], old)
    assert np.allclose(c[0], [1.0, 0.0], atol=1e-15)
    assert np.array_equal(c[1], old[1]) and np.array_equal(c[2], old[2])
    # one row: its centroid is the row itself
    c = oracle.kmeans_update(x[:1], [2], old)
    assert np.allclose(c[2], x[0], atol=1e-15) and np.array_equal(c[:2], old[:2])


def test_kmeans_separated_clusters_and_monotone_objective():
    rng = np.random.default_rng(6)
    d, P = 32, 8
    centres = unit_rows(rng, P, d).astype(np.float64)
    lab = rng.integers(0, P, 2000)
    x = centres[lab] + 0.05 * rng.standard_normal((2000, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    # start from one row of every cluster: one step recovers the labels
    init = np.stack([x[np.nonzero(lab == p)[0][0]] for p in range(P)])
    a, _, _ = oracle.kmeans_assign(x, init)
    assert np.array_equal(a, lab)
    c = oracle.kmeans_update(x, a, init)
    mean_dir = np.stack([x[lab == p].sum(0) for p in range(P)])
    mean_dir /= np.linalg.norm(mean_dir, axis=1, keepdims=True)
    assert np.allclose(c, mean_dir, atol=1e-12)
    # random start on unstructured data: the objective never decreases
    y = rng.standard_normal((1500, 16))
    y /= np.linalg.norm(y, axis=1, keepdims=True)
    c = y[rng.choice(1500, 20, replace=False)]
    prev = -np.inf
    for _ in range(8):
        a, _, _ = oracle.kmeans_assign(y, c)
        c = oracle.kmeans_update(y, a, c)
        obj = oracle.kmeans_objective(y, c)
        assert obj >= prev - 1e-9
        prev = obj


def test_splitmix64_published_outputs():
    # outputs of the generator's published reference implementation: from
    # state 0, and from state 1234567 (the sequence its authors' test prints)
    assert oracle.splitmix64(0, 3) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4,
                                       0x06C45D188009454F]
    assert oracle.splitmix64(1234567, 5) == [6457827717110365317, 3203168211198807973,
                                             9817491932198370423, 4593380528125082431,
                                             16408922859458223821]


def test_kmeans_init_picks_and_units():
    rng = np.random.default_rng(8)
    x = rng.standard_normal((23, 5))
    x[4] = 0.0
    o = oracle.splitmix64(9, 1)[0] % 23
    for P in (1, 2, 5, 7, 22, 23):
        pick, c = oracle.kmeans_init(x, P, 9)
        # brute force of the definition: offset, then floor(j n / P) steps
        assert pick.tolist() == [(o + math.floor(j * 23 / P)) % 23 for j in range(P)]
        assert len(set(pick.tolist())) == P and pick[0] == o
        for j, r in enumerate(pick):
            nrm = math.sqrt(sum(float(v) ** 2 for v in x[r]))
            want = x[r] / nrm if nrm > 0 else np.zeros(5)
            assert np.allclose(c[j], want, atol=1e-15)
    # P = n takes every row once; seeds move the offset
    pick, _ = oracle.kmeans_init(x, 23, 9)
    assert sorted(pick.tolist()) == list(range(23))
    assert len({int(oracle.kmeans_init(x, 3, s)[0][0]) for s in range(10)}) > 1
    with pytest.raises(ValueError):
        oracle.kmeans_init(x, 24, 0)


def test_partitioned_filtered_reductions_and_brute_force():
    """With the next-token filter: every partition probed is the filtered
    exact search; a tiny brute force of filter-and-probe; one token that no
    probed row starts with pads every rank."""
    rng = np.random.default_rng(9)
    N, d, P, k = 400, 12, 5, 15
    x = unit_rows(rng, N, d)
    cont = rng.integers(0, 4, (N, 3)).astype(np.int32)
    assign = rng.integers(0, P, N).astype(np.int32)
    q = unit_rows(rng, 4, d)
    nt = np.array([0, 1, 3, 7], np.int32)
    allp = np.tile(np.arange(P, dtype=np.int32), (4, 1))
    want = oracle.topk(x, "f32", q, k, cont, next_tok=nt)
    got = oracle.topk_partitioned(x, "f32", q, k, assign, P, allp, cont, next_tok=nt)
    for w, g in zip(want, got):
        assert np.array_equal(w, g, equal_nan=True)
    probes = np.array([[0, 2], [1, 1], [4, -1], [0, 3]], np.int32)
    idx, sc, _, _ = oracle.topk_partitioned(x, "f32", q, k, assign, P, probes, cont, next_tok=nt)
    x64 = x.astype(np.float64)
    for b in range(4):
        ps = {int(p) for p in probes[b] if 0 <= p < P}
        rows = np.array([i for i in range(N) if assign[i] in ps and cont[i, 0] == nt[b]], np.int64)
        s = (x64[rows] @ q[b].astype(np.float64)).astype(np.float32) if rows.size else \
            np.zeros(0, np.float32)
        order = np.lexsort((rows, -s.astype(np.float64)))[:k]
        m = order.size
        assert np.array_equal(idx[b, :m], rows[order]) and np.array_equal(sc[b, :m], s[order])
        assert (idx[b, m:] == -1).all() and np.isinf(sc[b, m:]).all()
    assert (idx[3] == -1).all()  # token 7 starts no value
