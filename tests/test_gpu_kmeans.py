"""Parity of the GPU spherical k-means steps with the fp64 oracle.

Assignment: where the oracle's best and second-best centroid differ by at
least tol the GPU picks the same centroid; elsewhere its pick scores within
tol of the best (exact scores from the oracle); its reported score is within
tol of the best.  tol = (d + 2) 2^-24 bounds an fp32 sum of d exact products
of unit vectors.  Exact ties (duplicate centroids) go to the lower id.
Seeding: centroids within 6e-8 of the oracle's picks made unit (one fp32
rounding of each element), a zero row giving a zero centroid.  Update: given
the oracle's assignment, centroids within 1e-6 of the oracle's
(2^-30 fixed-point sums), counts exact, bitwise deterministic, empty and
zero-sum partitions unchanged.  Training: the objective never decreases, and
the trained partitions give a partitioned search whose every row comes from a
probed partition, with high recall against the exact search."""
import sys

import numpy as np
import pytest
import torch

import oracle
from datagen import WORKLOADS, generate, to_numpy_bits

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
_TD = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def unit(rng, n, d):
    x = rng.standard_normal((n, d))
    return x / np.linalg.norm(x, axis=1, keepdims=True)


def as_keys(x64, dt):
    return torch.from_numpy(x64.astype(np.float32)).to(_TD[dt])


SHAPES = [
    # dtype, n, d, P
    ("f32", 1, 16, 1),         # one row, one centroid
    ("bf16", 70, 16384, 3),    # the largest d, a ragged row tile
    ("f16", 1000 + 3, 100, 70),
    ("bf16", 2000 + 1, 300, 64),
    ("f32", 777, 64, 5),
    ("f16", 5000, 128, 257),
    ("bf16", 64, 2048, 130),
]


@pytest.mark.parametrize("dt,n,d,P", SHAPES, ids=["%s-n%d-d%d-P%d" % s for s in SHAPES])
def test_kmeans_assign(gpu_lib, dt, n, d, P):
    from paper_2502_15572_amd import kmeans_assign
    say("kmeans assign", dt, n, d, P)
    rng = np.random.default_rng(n + d + P)
    keys = as_keys(unit(rng, n, d), dt)
    c = unit(rng, P, d).astype(np.float32)
    tie = P >= 4  # P // 2 differs from 1
    if tie:
        c[P // 2] = c[1]  # an exact tie: its rows go to id 1
    a, sc = kmeans_assign(keys.to(DEV), torch.from_numpy(c).to(DEV), with_score=True)
    torch.cuda.synchronize()
    a, sc = a.cpu().numpy(), sc.cpu().numpy()
    kb, _ = to_numpy_bits(keys)
    x = oracle.decode_keys(kb, dt)
    oa, ob, S = oracle.kmeans_assign(x, c.astype(np.float64))
    tol = (d + 2) * 2.0 ** -24
    srt = np.sort(S, axis=1)
    gap = srt[:, -1] - srt[:, -2] if P > 1 else np.full(n, np.inf)
    clear = gap >= tol
    assert np.array_equal(a[clear], oa[clear])
    assert np.all((a >= 0) & (a < P))
    assert np.all(S[np.arange(n), a] >= ob - tol)
    assert np.all(np.abs(sc - ob) <= tol)
    if tie:
        assert not np.any(a == P // 2)


@pytest.mark.parametrize("dt,n,d,P", SHAPES, ids=["%s-n%d-d%d-P%d" % s for s in SHAPES])
def test_kmeans_update(gpu_lib, dt, n, d, P):
    from paper_2502_15572_amd import kmeans_update
    say("kmeans update", dt, n, d, P)
    rng = np.random.default_rng(2 * n + d)
    x64 = unit(rng, n, d)
    planted = n >= 2 and P >= 5
    if planted:
        x64[1] = -x64[0]
    keys = as_keys(x64, dt)
    kb, _ = to_numpy_bits(keys)
    x = oracle.decode_keys(kb, dt)
    old = unit(rng, P, d).astype(np.float32)
    a = rng.integers(0, P, n).astype(np.int32)
    if planted:
        a[a == 2] = 3          # partition 2 is empty
        a[a == 0] = 4
        a[0] = a[1] = 0        # partition 0 holds x and -x: zero sum
    want = oracle.kmeans_update(x, a, old.astype(np.float64))
    cg = torch.from_numpy(old).to(DEV)
    counts = kmeans_update(keys.to(DEV), torch.from_numpy(a).to(DEV), cg)
    torch.cuda.synchronize()
    got = cg.cpu().numpy()
    assert np.array_equal(counts.cpu().numpy(), np.bincount(a, minlength=P))
    if planted:
        assert np.array_equal(got[0], old[0]) and np.array_equal(got[2], old[2])
    assert np.max(np.abs(got - want)) <= 1e-6
    cg2 = torch.from_numpy(old).to(DEV)
    kmeans_update(keys.to(DEV), torch.from_numpy(a).to(DEV), cg2)
    assert torch.equal(cg, cg2)


@pytest.mark.parametrize("dt,n,d,P,seed", [
    ("f32", 37, 5, 1, 0), ("f16", 1000, 128, 64, 5), ("bf16", 999, 130, 999, 2 ** 64 - 1),
    ("f16", 4097, 67, 300, 12345)])
def test_kmeans_init_matches_oracle(gpu_lib, dt, n, d, P, seed):
    from paper_2502_15572_amd import kmeans_init
    say("kmeans init %s n=%d d=%d P=%d seed=%d" % (dt, n, d, P, seed))
    rng = np.random.default_rng(n + d)
    keys = as_keys(unit(rng, n, d), dt)
    pick, _ = oracle.kmeans_init(np.ones((n, 1)), P, seed)
    if P > 3:
        keys[int(pick[3])] = 0  # a zero row gives a zero centroid
    kb, kdt = to_numpy_bits(keys)
    x = oracle.decode_keys(kb, kdt)
    pick, want = oracle.kmeans_init(x, P, seed)
    xd = keys.to(DEV)
    got = kmeans_init(xd, P, seed)
    torch.cuda.synchronize()
    got = got.cpu().numpy().astype(np.float64)
    # one fp32 rounding of each element of a unit vector: within 2^-25 (+ slack)
    assert np.max(np.abs(got - want)) <= 6e-8
    zero = ~np.any(x[pick] != 0, axis=1)
    assert zero.sum() == (1 if P > 3 else 0)
    assert np.array_equal(got[zero], np.zeros_like(got[zero]))


def test_train_partitions_and_search(gpu_lib):
    from paper_2502_15572_amd import PartitionedIndex, kmeans_assign, train_partitions
    say("train partitions")
    w = WORKLOADS["zipf33m_d128_f16"].scaled(40000)
    g = generate(w, "cpu", seed=3)
    keys, cont, q = g["keys"], g["cont"], g["queries"][:32]
    kd = keys.to(DEV)
    P = 64
    kb, dt = to_numpy_bits(keys)
    x = oracle.decode_keys(kb, dt)
    prev = -np.inf
    for iters in (0, 1, 2, 4, 8):
        c, a = train_partitions(kd, P, iters=iters, seed=5)
        obj = oracle.kmeans_objective(x, c.cpu().numpy().astype(np.float64))
        # each fp32 pick is within (d + 2) 2^-24 of the best; centroids within 1e-6
        assert obj >= prev - 2e-5 * x.shape[0]
        prev = obj
    assert torch.equal(a, kmeans_assign(kd, c))
    ix = PartitionedIndex(kd, cont.to(DEV), c, a)
    k, nprobe = 20, 16
    gi, gs, gt = ix.search(q.to(DEV), k, nprobe)
    torch.cuda.synchronize()
    gi = gi.cpu().numpy()
    o_idx, _, _, _ = oracle.topk(kb, dt, q.numpy(), k)
    recall = np.mean([len(set(gi[b]) & set(o_idx[b])) / k for b in range(len(q))])
    say("recall@%d with %d of %d partitions: %.3f" % (k, nprobe, P, recall))
    assert recall >= 0.9
    # every row from one of the query's probed partitions (queries whose
    # probed set is unique: nprobe-th and next centroid 1e-5 apart)
    pc, ps, _, _ = oracle.topk(c.cpu().numpy(), "f32", q.numpy(), nprobe + 1)
    an = a.cpu().numpy()
    checked = 0
    for b in range(len(q)):
        if ps[b, nprobe - 1] - ps[b, nprobe] < 1e-5:
            continue
        rows = gi[b][gi[b] >= 0]
        assert np.isin(an[rows], pc[b, :nprobe]).all()
        checked += 1
    assert checked >= len(q) // 2
    ix.close()


def test_kmeans_update_on_two_streams(gpu_lib):
    """k-means updates issued back to back on two streams (each with its own
    library buffer of sums): every result equals the one computed alone."""
    from paper_2502_15572_amd import kmeans_update
    rng = np.random.default_rng(31)
    data = []
    for n, d, P in ((20000, 128, 300), (15000, 128, 200)):
        keys = as_keys(unit(rng, n, d), "f16").to(DEV)
        a = torch.from_numpy(rng.integers(0, P, n).astype(np.int32)).to(DEV)
        c0 = torch.from_numpy(unit(rng, P, d).astype(np.float32)).to(DEV)
        ref = c0.clone()
        kmeans_update(keys, a, ref)
        data.append((keys, a, c0, ref))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[], []]
    for _ in range(6):
        for i, s in enumerate(streams):
            keys, a, c0, _ = data[i]
            with torch.cuda.stream(s):
                c = c0.clone()
                kmeans_update(keys, a, c, stream=s)
                outs[i].append(c)
    torch.cuda.synchronize()
    for i in range(2):
        for c in outs[i]:
            assert torch.equal(c, data[i][3])
