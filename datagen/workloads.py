"""Workload definitions and seeded generators.

Stand-ins for the paper's datastores (Section 4.2, Table 1: 19M-57.2M keys
built from Llama2 hidden states, reduced by PCA to 32-128 dimensions,
Section 5.2).  The datasets and weights are not available, so keys are drawn
from Gaussian clusters, L2-normalised (Section 3.4, Eq. 2) and rounded to the
storage type; values are next-token sequences drawn from a Zipf law over a
32,000-token vocabulary (Section 3.5: each key maps to its next N tokens).

Recipe (per workload, fixed seed):
  * centres c_m ~ N(0, I_d), m < M;
  * cluster id a_i uniform over M, or truncated Zipf(s) over ranks 1..M;
  * isotropic:   x_i = c_{a_i} + sigma * eps_i;
    anisotropic: x_i = c_{a_i} + s_{a_i} (.) eps_i with per-cluster,
                 per-dimension scales s_{m,j} = 10^{U(-1,0)} in [0.1, 1];
  * x_i normalised in fp64, then rounded to f32 / f16 / bf16 (not
    renormalised after rounding);
  * continuations: i.i.d. truncated Zipf(1.1) over ranks 1..V, token = rank-1;
  * queries: "perturbed" = normalize(x_hat_src + 0.1 * eps) for a uniformly
    drawn source row (kept fp32); "fresh" = normalize(c_m + s_m (.) eps) with m
    drawn from the cluster-assignment law; "mixed" interleaves them
    (even = perturbed, odd = fresh).

Each random component has its own generator seeded from (seed, workload id,
component, chunk), so results do not depend on the chunk size used to build
them, only on the device the generator runs on (torch's CPU and GPU
generators are different streams).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int
    N: int
    d: int
    dtype: str           # "f32" | "f16" | "bf16"
    clusters: int
    aniso: bool
    k: int
    batches: tuple
    pool: int
    query_kind: str      # "perturbed" | "mixed"
    sigma: float = 0.3   # isotropic within-cluster std
    cluster_zipf: float | None = None
    L: int = 10
    vocab: int = 32000
    token_zipf: float = 1.1
    query_noise: float = 0.1

    def scaled(self, N: int) -> "Workload":
        """Same recipe at a different datastore size (for fast parity runs)."""
        return dataclasses.replace(self, N=int(N))

    def with_pool(self, n: int) -> "Workload":
        """Same recipe with a query pool of at least n queries (a batch larger
        than the pool takes a larger one; smaller batches keep the pool)."""
        return self if n <= self.pool else dataclasses.replace(self, pool=int(n))

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def key_bytes(self) -> int:
        return self.N * self.d * self.elem_bytes


WORKLOADS = {
    w.name: w
    for w in [
        Workload("flat16k_d256_f32", 0, 16384, 256, "f32", 64, False, 10, (8,), 8, "perturbed"),
        Workload("hidden1m_d4096_bf16", 1, 1 << 20, 4096, "bf16", 1024, True, 10, (1, 4), 64,
                 "perturbed"),
        Workload("pca4m_d1024_f16", 2, 1 << 22, 1024, "f16", 4096, True, 16, (1, 16), 64, "mixed"),
        Workload("batch10m_d256_f16", 3, 10_000_000, 256, "f16", 8192, True, 32, (64, 256), 256,
                 "perturbed"),
        Workload("zipf33m_d128_f16", 4, 1 << 25, 128, "f16", 16384, True, 100, (1, 128), 128,
                 "perturbed", cluster_zipf=1.2),
    ]
}

_TORCH_DTYPE = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
_CHUNK = 1 << 16   # rows per noise generator


def _gen(device, seed: int, wid: int, comp: int, chunk: int = 0) -> torch.Generator:
    g = torch.Generator(device=device)
    # A fixed mixing of the four integers into one 63-bit seed.
    s = (((seed * 1_000_003 + wid) * 1_000_033 + comp) * 1_000_037 + chunk) & ((1 << 63) - 1)
    g.manual_seed(s)
    return g


def _zipf_cdf(n: int, s: float, device) -> torch.Tensor:
    r = torch.arange(1, n + 1, dtype=torch.float64, device=device)
    w = r.pow(-s)
    c = torch.cumsum(w, 0)
    return c / c[-1]


def _zipf_draw(cdf: torch.Tensor, count: int, g: torch.Generator) -> torch.Tensor:
    u = torch.rand(count, dtype=torch.float64, device=cdf.device, generator=g)
    idx = torch.searchsorted(cdf, u)
    return idx.clamp_(max=cdf.numel() - 1)


def _assign(w: Workload, count: int, g: torch.Generator, device) -> torch.Tensor:
    if w.cluster_zipf is None:
        return torch.randint(0, w.clusters, (count,), generator=g, device=device)
    return _zipf_draw(_zipf_cdf(w.clusters, w.cluster_zipf, device), count, g)


def _normalize64(x: torch.Tensor) -> torch.Tensor:
    x = x.to(torch.float64)
    return x / x.norm(dim=1, keepdim=True)


def generate(w: Workload, device="cpu", seed: int = 0, with_queries: bool = True,
             planted_duplicates: int = 0):
    """Build keys [N,d] (storage dtype), continuations [N,L] int32 and a
    query pool [pool,d] fp32 on ``device``.

    ``planted_duplicates`` > 0 copies that many random earlier rows over later
    rows (used by tie-break tests; the duplicate pairs are returned).
    """
    device = torch.device(device)
    N, d = w.N, w.d
    centres = torch.randn(w.clusters, d, generator=_gen(device, seed, w.wid, 0), device=device,
                          dtype=torch.float32)
    scales = None
    if w.aniso:
        u = torch.rand(w.clusters, d, generator=_gen(device, seed, w.wid, 1), device=device,
                       dtype=torch.float32)
        scales = torch.pow(10.0, -u)
    assign = _assign(w, N, _gen(device, seed, w.wid, 2), device)
    keys = torch.empty(N, d, dtype=_TORCH_DTYPE[w.dtype], device=device)
    for c0 in range(0, N, _CHUNK):
        c1 = min(N, c0 + _CHUNK)
        eps = torch.randn(c1 - c0, d, generator=_gen(device, seed, w.wid, 3, c0 // _CHUNK),
                          device=device, dtype=torch.float32)
        a = assign[c0:c1]
        if w.aniso:
            x = centres[a].to(torch.float64) + scales[a].to(torch.float64) * eps.to(torch.float64)
        else:
            x = centres[a].to(torch.float64) + w.sigma * eps.to(torch.float64)
        keys[c0:c1] = _normalize64(x).to(torch.float32).to(keys.dtype)
        del eps, x
    dups = []
    if planted_duplicates:
        # sources in the lower half, copies in the upper half, so no copy
        # is itself overwritten later
        g = _gen(device, seed, w.wid, 7)
        half = N // 2
        dst = half + torch.randperm(N - half, generator=g, device=device)[:planted_duplicates]
        srcs = torch.randint(0, half, (dst.numel(),), generator=g, device=device)
        keys[dst] = keys[srcs]
        dups = list(zip(srcs.tolist(), dst.tolist()))
    tcdf = _zipf_cdf(w.vocab, w.token_zipf, device)
    cont = torch.empty(N, w.L, dtype=torch.int32, device=device)
    for c0 in range(0, N, _CHUNK):
        c1 = min(N, c0 + _CHUNK)
        t = _zipf_draw(tcdf, (c1 - c0) * w.L, _gen(device, seed, w.wid, 4, c0 // _CHUNK))
        cont[c0:c1] = t.view(c1 - c0, w.L).to(torch.int32)
    out = {"keys": keys, "cont": cont, "assign": assign, "centres": centres, "duplicates": dups}
    if with_queries:
        out.update(_queries(w, keys, centres, scales, device, seed))
    return out


def _queries(w: Workload, keys, centres, scales, device, seed):
    P = w.pool
    gs = _gen(device, seed, w.wid, 5)
    gn = _gen(device, seed, w.wid, 6)
    src = torch.randint(0, w.N, (P,), generator=gs, device=device)
    noise = torch.randn(P, w.d, generator=gn, device=device, dtype=torch.float32).to(torch.float64)
    pert = _normalize64(keys[src].to(torch.float64) + w.query_noise * noise)
    kinds = torch.zeros(P, dtype=torch.int8, device=device)
    q = pert
    if w.query_kind == "mixed":
        m = _assign(w, P, _gen(device, seed, w.wid, 8), device)
        eps = torch.randn(P, w.d, generator=_gen(device, seed, w.wid, 9), device=device,
                          dtype=torch.float32).to(torch.float64)
        base = centres[m].to(torch.float64)
        fresh = base + (scales[m].to(torch.float64) * eps if w.aniso else w.sigma * eps)
        fresh = _normalize64(fresh)
        odd = torch.arange(P, device=device) % 2 == 1
        q = torch.where(odd[:, None], fresh, pert)
        kinds = odd.to(torch.int8)
        src = torch.where(odd, torch.full_like(src, -1), src)
    return {"queries": q.to(torch.float32).contiguous(), "query_src": src, "query_kind": kinds}


def to_numpy_bits(keys: torch.Tensor) -> tuple[np.ndarray, str]:
    """Host copy of the keys in the form the oracle takes (bits for 16-bit types)."""
    k = keys.detach().cpu().contiguous()
    if k.dtype == torch.float32:
        return k.numpy(), "f32"
    if k.dtype == torch.float16:
        return k.view(torch.int16).numpy().view(np.uint16), "f16"
    if k.dtype == torch.bfloat16:
        return k.view(torch.int16).numpy().view(np.uint16), "bf16"
    raise TypeError(keys.dtype)


def zipf_mass(n: int, s: float, rank: int) -> float:
    """Probability of ``rank`` under truncated Zipf(s) on 1..n (for tests)."""
    h = sum(r ** -s for r in range(1, n + 1))
    return rank ** -s / h


def expected_cos_perturbed(d: int, noise: float) -> float:
    """E[cos(x, normalize(x + noise*eps))] ~ 1/sqrt(1 + d*noise^2) for unit x."""
    return 1.0 / math.sqrt(1.0 + d * noise * noise)
