"""The seeded generators follow their recipe (CPU only)."""
import math

import numpy as np
import torch

from datagen import WORKLOADS, generate
from datagen.workloads import expected_cos_perturbed, zipf_mass


def test_deterministic_and_chunk_independent():
    w = WORKLOADS["zipf33m_d128_f16"].scaled(70000)   # spans two noise chunks
    a = generate(w, "cpu")
    b = generate(w, "cpu")
    assert torch.equal(a["keys"].view(torch.int16), b["keys"].view(torch.int16))
    assert torch.equal(a["cont"], b["cont"]) and torch.equal(a["queries"], b["queries"])
    # per-chunk generators: a smaller datastore's continuations are a prefix
    small = generate(w.scaled(1000), "cpu", with_queries=False)
    assert torch.equal(small["cont"], a["cont"][:1000])


def test_norms_and_shapes():
    for name, w in WORKLOADS.items():
        ws = w.scaled(3000)
        g = generate(ws, "cpu")
        k = g["keys"]
        assert tuple(k.shape) == (ws.N, ws.d)
        n = k.to(torch.float64).norm(dim=1)
        bound = {"f32": 1e-6, "f16": 2e-3, "bf16": 8e-3}[ws.dtype]
        assert float((n - 1).abs().max()) < bound
        q = g["queries"]
        assert q.dtype == torch.float32 and tuple(q.shape) == (ws.pool, ws.d)
        assert float((q.to(torch.float64).norm(dim=1) - 1).abs().max()) < 1e-6
        assert g["cont"].dtype == torch.int32 and tuple(g["cont"].shape) == (ws.N, ws.L)
        assert int(g["cont"].min()) >= 0 and int(g["cont"].max()) < ws.vocab


def test_token_zipf_mass():
    w = WORKLOADS["flat16k_d256_f32"]
    g = generate(w, "cpu", with_queries=False)
    p0 = float((g["cont"] == 0).double().mean())
    want = zipf_mass(w.vocab, w.token_zipf, 1)
    assert abs(p0 - want) < 4 * math.sqrt(want * (1 - want) / g["cont"].numel())


def test_cluster_zipf_mass():
    w = WORKLOADS["zipf33m_d128_f16"].scaled(200000)
    g = generate(w, "cpu", with_queries=False)
    top = float((g["assign"] == 0).double().mean())
    want = zipf_mass(w.clusters, w.cluster_zipf, 1)
    assert abs(top - want) < 4 * math.sqrt(want * (1 - want) / w.N)


def test_perturbed_query_cosine():
    w = WORKLOADS["batch10m_d256_f16"].scaled(5000)
    g = generate(w, "cpu")
    src = g["query_src"]
    cos = (g["queries"].double() * g["keys"][src].double()).sum(1)
    want = expected_cos_perturbed(w.d, w.query_noise)
    assert abs(float(cos.mean()) - want) < 0.05


def test_mixed_queries_interleave():
    w = WORKLOADS["pca4m_d1024_f16"].scaled(4000)
    g = generate(w, "cpu")
    kinds = g["query_kind"].tolist()
    assert kinds[0::2] == [0] * (w.pool // 2) and kinds[1::2] == [1] * (w.pool // 2)
    assert all(s >= 0 for s in g["query_src"][0::2].tolist())


def test_pool_grows_to_the_batch():
    # a batch larger than the workload's query pool takes a pool of that many
    # distinct queries (the bench never repeats or drops queries in a batch)
    w = WORKLOADS["pca4m_d1024_f16"].scaled(2000)
    assert w.with_pool(w.pool) is w and w.with_pool(1) is w
    big = w.with_pool(256)
    assert big.pool == 256 and big.N == w.N and big.d == w.d
    q = generate(big, "cpu")["queries"]
    assert tuple(q.shape) == (256, w.d)
    assert torch.unique(q, dim=0).shape[0] == 256
