"""Parity of the GPU query-side transform (Algorithm 1 steps 4-6: Eq. 1
z-score, Section 3.3 projection, Eq. 2 L2) with the fp64 oracle.

Tolerance, derived from the arithmetic (fp32, unit roundoff u = 2^-24): the
projection is a length-D sum of products computed in some order in fp32, so
each unnormalised output element is within (D + 10) u sum_j |z_j W_jk| of the
exact value (z itself carries a few roundings); normalisation adds about
(l + 10) u relative to each element.  The bound is computed per element."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
U = 2.0 ** -24


def make_case(M, D, l, seed):
    rng = np.random.default_rng(seed)
    sample = rng.standard_normal((2048, D)) * rng.uniform(0.1, 3.0, D) + rng.standard_normal(D)
    mean = sample.mean(axis=0)
    var = sample.var(axis=0)
    Q, _ = np.linalg.qr(rng.standard_normal((D, max(l, 1))))
    W = Q[:, :l] if Q.shape[1] >= l else rng.standard_normal((D, l)) / np.sqrt(D)
    x = rng.standard_normal((M, D)) * rng.uniform(0.1, 3.0, D) + mean
    f = lambda a: np.ascontiguousarray(a, np.float32)
    return f(x), f(mean), f(var), f(W)


def bound(x, mean, var, W, eps_z, y_exact):
    z = (x.astype(np.float64) - mean) / np.sqrt(var.astype(np.float64) + eps_z)
    v = z @ W.astype(np.float64)
    nrm = np.maximum(np.linalg.norm(v, axis=1, keepdims=True), 1e-30)
    D, l = W.shape
    return U * ((D + 10) * (np.abs(z) @ np.abs(W.astype(np.float64))) / nrm
                + (l + 10) * np.abs(y_exact)) + 1e-30


def run(x, mean, var, W, eps_z=1e-5, eps_n=1e-12):
    from paper_2502_15572_amd import transform
    t = lambda a: torch.from_numpy(a).to(DEV)
    y = transform(t(x), t(mean), t(var), t(W), eps_z, eps_n)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


SHAPES = [
    # (M, D, l): decode-step queries at the paper's reductions, ragged tiles,
    # tiny, and a datastore-sized pass
    (1, 4096, 64),
    (16, 4096, 256),
    (257, 1000, 130),
    (3, 17, 5),
    (300, 4096, 1024),
    (20000, 512, 128),
    # datastore-sized passes take 128-row tiles: ragged rows, dims and
    # columns, and dims that are not a multiple of 4 (scalar staging)
    (1500, 1000, 130),
    (1100, 999, 70),
]


@pytest.mark.parametrize("M,D,l", SHAPES, ids=["M%d-D%d-l%d" % s for s in SHAPES])
def test_transform_parity(gpu_lib, M, D, l):
    print("transform", M, D, l, flush=True)
    x, mean, var, W = make_case(M, D, l, seed=M + D + l)
    want = oracle.transform(x, mean, var, W, 1e-5, 1e-12)
    got = run(x, mean, var, W)
    err = np.abs(got - want)
    tol = bound(x, mean, var, W, 1e-5, want)
    assert np.all(err <= tol), (float(err.max()), float((err / tol).max()))
    assert np.allclose(np.linalg.norm(got, axis=1), 1.0, atol=1e-5)
    print("  max |gpu - oracle| %.2e, max err/bound %.3f" % (err.max(), (err / tol).max()),
          flush=True)


def test_transform_zero_row_and_zero_variance(gpu_lib):
    """x == mean gives 0 (Eq. 2's eps, no NaN); a zero-variance dim is scaled
    by 1/sqrt(eps) (Eq. 1's eps)."""
    D, l = 40, 8
    x, mean, var, W = make_case(4, D, l, seed=7)
    x[0] = mean
    var[3] = 0.0
    got = run(x, mean, var, W, eps_z=0.25)
    want = oracle.transform(x, mean, var, W, 0.25, 1e-12)
    assert np.array_equal(got[0], np.zeros(l))
    tol = bound(x, mean, var, W, 0.25, want)
    assert np.all(np.abs(got - want) <= tol)


def test_transform_feeds_search(gpu_lib):
    """Transformed datastore rows as keys and a transformed row as the query:
    the row's own key ranks first (self-retrieval through the whole chain)."""
    from paper_2502_15572_amd import Index, transform
    D, l, N = 256, 64, 5000
    x, mean, var, W = make_case(N, D, l, seed=11)
    t = lambda a: torch.from_numpy(a).to(DEV)
    keys = transform(t(x), t(mean), t(var), t(W))
    ix = Index(keys, torch.arange(N, dtype=torch.int32, device=DEV).view(N, 1))
    rows = torch.tensor([5, 999, 4321], device=DEV)
    q = transform(t(x)[rows], t(mean), t(var), t(W))
    idx, score, tok = ix.search(q, 3)
    assert idx[:, 0].tolist() == rows.tolist()
    assert torch.equal(tok[:, 0, 0].long(), rows)
    ix.close()


def test_transform_argument_errors(gpu_lib):
    from paper_2502_15572_amd import _lib
    lib = _lib.load()
    assert lib.dresd_transform(None, 1, 4, None, None, 1e-5, None, 2, 1e-12, None, None) == 1
    assert lib.dresd_transform(None, 0, 4, None, None, 1e-5, None, 2, 1e-12, None, None) == 0
    assert lib.dresd_transform(None, 0, 0, None, None, 1e-5, None, 2, 1e-12, None, None) == 1
    assert lib.dresd_transform(None, 0, 4, None, None, -1.0, None, 2, 1e-12, None, None) == 1


def test_transform_on_two_streams(gpu_lib):
    """Transforms with split partial sums issued back to back on two streams
    (each stream has its own library buffer): every result equals the one
    computed alone, bit for bit."""
    from paper_2502_15572_amd import transform
    t = lambda a: torch.from_numpy(a).to(DEV)
    cases = [make_case(16, 4096, 256, 21), make_case(8, 4096, 512, 22)]
    args = [tuple(t(a) for a in c) for c in cases]
    refs = [transform(*a) for a in args]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[], []]
    torch.cuda.synchronize()
    for _ in range(8):
        for i, s in enumerate(streams):
            with torch.cuda.stream(s):
                outs[i].append(transform(*args[i], stream=s))
    torch.cuda.synchronize()
    for i in range(2):
        for y in outs[i]:
            assert torch.equal(y, refs[i])
