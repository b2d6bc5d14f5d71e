"""CPU oracle for DReSD's dense retrieval step -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it; the product path fails loudly when its HIP extension
is missing instead of falling back here.

The arithmetic lives in ``dresd_oracle.c`` (plain C, fp64 accumulation,
rounded once to fp32; ranking by score descending then lowest row index).
It follows DReSD Section 3.5, Eq. 3 (cosine similarity argmax over a
key -> next-tokens store) with unit-norm keys and queries (Section 3.4,
Eq. 2), generalised to the k best keys that batch verification consumes
(Section 3.6); ``topk(..., next_tok=...)`` adds the next-token filter of
Section 3.5 (only rows whose value starts with the query's next token
compete); ``topk_partitioned`` is the partitioned (inverted-file) reading
of the paper's approximate search: the exact k best rows among the
partitions each query probes.  This module marshals numpy arrays into that
library (building it with gcc when it is missing) and holds the fp64 numpy
oracles of the steps around the search: the query-side transform (Eqs. 1-2,
Section 3.3), spherical k-means (the partitioning of the partitioned search)
and draft assembly (Section 3.6).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dresd_oracle.c")
_LIB = os.path.join(_HERE, "libdresd_oracle.so")
_lock = threading.Lock()
_lib = None

DTYPE_CODES = {"f32": 0, "f16": 1, "bf16": 2}


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O3", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-Wall", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_LIB)
            P = ctypes.c_void_p
            lib.oracle_topk.argtypes = [P, ctypes.c_int, ctypes.c_int64, ctypes.c_int32,
                                        P, ctypes.c_int32, ctypes.c_int32, P, ctypes.c_int32,
                                        P, P, P, P, ctypes.c_int32]
            lib.oracle_topk.restype = ctypes.c_int
            lib.oracle_topk_filtered.argtypes = [P, ctypes.c_int, ctypes.c_int64, ctypes.c_int32,
                                                 P, ctypes.c_int32, ctypes.c_int32, P,
                                                 ctypes.c_int32, P, P, P, P, P, ctypes.c_int32]
            lib.oracle_topk_filtered.restype = ctypes.c_int
            I32 = ctypes.c_int32
            lib.oracle_topk_partitioned.argtypes = [P, ctypes.c_int, ctypes.c_int64, I32, P, I32,
                                                    I32, P, I32, P, I32, P, I32, P, P, P, P, P,
                                                    I32]
            lib.oracle_topk_partitioned.restype = ctypes.c_int
            lib.oracle_score_rows.argtypes = [P, ctypes.c_int, ctypes.c_int64, ctypes.c_int32,
                                              P, P, ctypes.c_int64, P]
            lib.oracle_score_rows.restype = ctypes.c_int
            lib.oracle_set_mutation.argtypes = [ctypes.c_int]
            lib.oracle_set_mutation.restype = None
            _lib = lib
    return _lib


def _emb_bits(emb: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        if emb.dtype != np.float32:
            raise TypeError("f32 keys must be a float32 array")
    elif dtype == "f16":
        if emb.dtype not in (np.float16, np.uint16):
            raise TypeError("f16 keys must be float16 (or their uint16 bits)")
    elif dtype == "bf16":
        if emb.dtype != np.uint16:
            raise TypeError("bf16 keys must be passed as their uint16 bits")
    else:
        raise ValueError("unknown key dtype %r" % dtype)
    if emb.ndim != 2:
        raise ValueError("keys must be [N, d]")
    return np.ascontiguousarray(emb)


def topk(emb: np.ndarray, dtype: str, queries: np.ndarray, k: int,
         cont: np.ndarray | None = None, threads: int = 0, next_tok=None):
    """Exact top-k by inner product.

    Returns ``(idx[B,k] int64, score[B,k] f32, tokens[B,k,L] int32 or None,
    next_score[B] f32)`` where ``next_score`` is the (k+1)-th best score
    (NaN when there is none).  With ``next_tok`` ([B] ints) only rows whose
    continuation starts with that query's next token compete (Section 3.5);
    ranks past the matching rows hold index -1, score -inf and zero tokens.
    """
    e = _emb_bits(emb, dtype)
    q = np.ascontiguousarray(queries, dtype=np.float32)
    if q.ndim != 2 or q.shape[1] != e.shape[1]:
        raise ValueError("queries must be [B, d]")
    N, d = e.shape
    B = q.shape[0]
    if not (1 <= k <= N):
        raise ValueError("need 1 <= k <= N")
    idx = np.empty((B, k), np.int64)
    score = np.empty((B, k), np.float32)
    nxt = np.empty((B,), np.float32)
    tok = None
    L = 0
    cptr = None
    if cont is not None:
        c = np.ascontiguousarray(cont, dtype=np.int32)
        if c.ndim != 2 or c.shape[0] != N:
            raise ValueError("continuations must be [N, L]")
        L = c.shape[1]
        tok = np.empty((B, k, L), np.int32)
        cptr = c.ctypes.data
    lib = _load()
    tptr = tok.ctypes.data if tok is not None else None
    if next_tok is None:
        rc = lib.oracle_topk(e.ctypes.data, DTYPE_CODES[dtype], N, d, q.ctypes.data, B, k,
                             cptr, L, idx.ctypes.data, score.ctypes.data, tptr,
                             nxt.ctypes.data, int(threads))
    else:
        nt = np.ascontiguousarray(next_tok, dtype=np.int32).reshape(-1)
        if nt.shape[0] != B or cont is None or L < 1:
            raise ValueError("next_tok needs one token per query and continuations")
        rc = lib.oracle_topk_filtered(e.ctypes.data, DTYPE_CODES[dtype], N, d, q.ctypes.data,
                                      B, k, cptr, L, nt.ctypes.data, idx.ctypes.data,
                                      score.ctypes.data, tptr, nxt.ctypes.data, int(threads))
    if rc != 0:
        raise RuntimeError("oracle top-k failed")
    return idx, score, tok, nxt


def topk_partitioned(emb: np.ndarray, dtype: str, queries: np.ndarray, k: int,
                     assign, P: int, probes, cont: np.ndarray | None = None, threads: int = 0,
                     next_tok=None):
    """Partitioned retrieval (the approximate search of Section 3.5, read as
    an inverted file): row i belongs to partition ``assign[i]`` in [0, P);
    query b returns the exact k best rows among the partitions listed in
    ``probes[b]`` (entries outside [0, P) ignored, repeats counted once) --
    with ``next_tok`` only those whose value starts with the query's next
    token (Section 3.5's filter).  Same outputs and padding as
    ``topk(..., next_tok=...)``."""
    e = _emb_bits(emb, dtype)
    q = np.ascontiguousarray(queries, dtype=np.float32)
    if q.ndim != 2 or q.shape[1] != e.shape[1]:
        raise ValueError("queries must be [B, d]")
    N, d = e.shape
    B = q.shape[0]
    if not (1 <= k <= N):
        raise ValueError("need 1 <= k <= N")
    a = np.ascontiguousarray(assign, dtype=np.int32).reshape(-1)
    if a.shape[0] != N:
        raise ValueError("assign must hold one partition per row")
    pr = np.ascontiguousarray(probes, dtype=np.int32)
    if pr.ndim != 2 or pr.shape[0] != B:
        raise ValueError("probes must be [B, S]")
    idx = np.empty((B, k), np.int64)
    score = np.empty((B, k), np.float32)
    nxt = np.empty((B,), np.float32)
    tok, L, cptr = None, 0, None
    if cont is not None:
        c = np.ascontiguousarray(cont, dtype=np.int32)
        if c.ndim != 2 or c.shape[0] != N:
            raise ValueError("continuations must be [N, L]")
        L = c.shape[1]
        tok = np.empty((B, k, L), np.int32)
        cptr = c.ctypes.data
    ntp = None
    if next_tok is not None:
        nt = np.ascontiguousarray(next_tok, dtype=np.int32).reshape(-1)
        if nt.shape[0] != B or cont is None or L < 1:
            raise ValueError("next_tok needs one token per query and continuations")
        ntp = nt.ctypes.data
    rc = _load().oracle_topk_partitioned(
        e.ctypes.data, DTYPE_CODES[dtype], N, d, q.ctypes.data, B, k, cptr, L, a.ctypes.data,
        int(P), pr.ctypes.data, pr.shape[1], ntp, idx.ctypes.data, score.ctypes.data,
        tok.ctypes.data if tok is not None else None, nxt.ctypes.data, int(threads))
    if rc != 0:
        raise RuntimeError("oracle partitioned top-k failed (assignment out of range?)")
    return idx, score, tok, nxt


def decode_keys(emb: np.ndarray, dtype: str) -> np.ndarray:
    """Key rows as float64 (exact for f32, f16 and bf16 bits)."""
    e = _emb_bits(emb, dtype)
    if dtype == "bf16":
        return (e.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if dtype == "f16" and e.dtype == np.uint16:
        return e.view(np.float16).astype(np.float64)
    return e.astype(np.float64)


def kmeans_assign(x: np.ndarray, centroids: np.ndarray):
    """Assignment step of spherical k-means, the partitioning behind the
    partitioned search: each row goes to the centroid with the largest inner
    product (cosine for unit rows, Eq. 3), ties to the lowest centroid id.
    x [n, d] float64 (``decode_keys``), centroids [P, d]; returns
    (assign [n] int32, best score [n] float64, all scores [n, P] float64)."""
    s = np.asarray(x, np.float64) @ np.asarray(centroids, np.float64).T
    a = np.argmax(s, axis=1)  # first maximum = lowest id
    return a.astype(np.int32), s[np.arange(s.shape[0]), a], s


def kmeans_update(x: np.ndarray, assign, centroids: np.ndarray) -> np.ndarray:
    """Update step of spherical k-means: each centroid becomes the unit
    vector along the sum of its rows; a partition with no rows (or a zero
    sum) keeps its previous centroid.  Returns [P, d] float64."""
    x = np.asarray(x, np.float64)
    c = np.array(centroids, np.float64)
    a = np.asarray(assign).reshape(-1)
    P = c.shape[0]
    if a.shape[0] != x.shape[0] or (a.size and (a.min() < 0 or a.max() >= P)):
        raise ValueError("assign must hold one partition in [0, P) per row")
    sums = np.zeros_like(c)
    np.add.at(sums, a, x)
    n = np.sqrt(np.sum(sums * sums, axis=1))
    ok = n > 0
    c[ok] = sums[ok] / n[ok, None]
    return c


def splitmix64(state: int, count: int) -> list:
    """The first ``count`` outputs of SplitMix64 (Steele, Lea and Flood,
    "Fast splittable pseudorandom number generators", OOPSLA 2014) from
    ``state``: add the golden-ratio increment, then two xor-shift-multiply
    rounds and a final xor-shift.  The seeded source of k-means seeding."""
    m = (1 << 64) - 1
    out = []
    for _ in range(count):
        state = (state + 0x9E3779B97F4A7C15) & m
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
        out.append(z ^ (z >> 31))
    return out


def kmeans_init(x: np.ndarray, P: int, seed: int):
    """Starting centroids of spherical k-means: P distinct rows spread
    evenly through the row order from a seeded offset o (the first SplitMix64
    output from ``seed``, mod n), row (o + floor(j n / P)) mod n for
    centroid j, each scaled to unit length (a zero row stays zero).
    Returns (picked rows [P] int64, centroids [P, d] float64)."""
    x = np.asarray(x, np.float64)
    n = x.shape[0]
    if not 1 <= P <= n:
        raise ValueError("need 1 <= P <= n")
    o = splitmix64(seed, 1)[0] % n
    pick = np.array([(o + (j * n) // P) % n for j in range(P)], np.int64)
    rows = x[pick]
    nrm = np.sqrt(np.sum(rows * rows, axis=1))
    c = np.zeros_like(rows)
    ok = nrm > 0
    c[ok] = rows[ok] / nrm[ok, None]
    return pick, c


def kmeans_objective(x: np.ndarray, centroids: np.ndarray) -> float:
    """Sum over rows of the best inner product with a centroid: the quantity
    spherical k-means never decreases."""
    return float(np.sum(np.max(np.asarray(x, np.float64) @ np.asarray(centroids, np.float64).T,
                               axis=1)))


def score_rows(emb: np.ndarray, dtype: str, query: np.ndarray, rows) -> np.ndarray:
    """Oracle scores of the given rows for one query (fp32)."""
    e = _emb_bits(emb, dtype)
    q = np.ascontiguousarray(query, dtype=np.float32).reshape(-1)
    r = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1)
    out = np.empty(r.shape, np.float32)
    rc = _load().oracle_score_rows(e.ctypes.data, DTYPE_CODES[dtype], e.shape[0], e.shape[1],
                                   q.ctypes.data, r.ctypes.data, r.size, out.ctypes.data)
    if rc != 0:
        raise RuntimeError("oracle_score_rows failed (row out of range?)")
    return out


class mutation:
    """Context manager that plants a numbered mistake in the oracle (CPU tests only)."""

    def __init__(self, m: int):
        self.m = m

    def __enter__(self):
        _load().oracle_set_mutation(self.m)
        return self

    def __exit__(self, *exc):
        _load().oracle_set_mutation(0)
        return False


def transform(x: np.ndarray, mean: np.ndarray, var: np.ndarray, W: np.ndarray,
              eps_z: float = 1e-5, eps_n: float = 1e-12) -> np.ndarray:
    """Query-side transform of Algorithm 1 steps 4-6, in fp64, in the paper's
    order: z-score normalisation with the datastore's per-dimension mean and
    variance (Section 3.2, Eq. 1: (v - E[V]) / sqrt(Var[V] + eps)), projection
    onto the first l principal components (Section 3.3: v W_l), and L2
    normalisation (Section 3.4, Eq. 2: v_l / max(||v_l||_2, eps)).

    x [M, D], mean [D], var [D], W [D, l]; returns [M, l] float64.
    """
    x = np.asarray(x, np.float64)
    mu = np.asarray(mean, np.float64)
    vr = np.asarray(var, np.float64)
    Wl = np.asarray(W, np.float64)
    if x.ndim != 2 or Wl.ndim != 2 or Wl.shape[0] != x.shape[1]:
        raise ValueError("x must be [M, D] and W [D, l]")
    if mu.shape != (x.shape[1],) or vr.shape != (x.shape[1],):
        raise ValueError("mean and var must be [D]")
    z = (x - mu) / np.sqrt(vr + eps_z)                                   # Eq. 1
    v = z @ Wl                                                           # Section 3.3
    n = np.sqrt(np.sum(v * v, axis=1, keepdims=True))
    return v / np.maximum(n, eps_n)                                      # Eq. 2


def pack_drafts(tokens: np.ndarray, r: int, length: int, eos: int = 0):
    """Draft assembly for batch verification (Section 3.6): drafts are rows of
    a [r, length] matrix padded with the EOS id.

    For each query, walk its retrieved continuations in rank order; a draft is
    the first ``length`` tokens with every token after the first EOS replaced
    by EOS (the sequence has ended); drafts that start with EOS (nothing to
    propose, e.g. the padding ranks of a filtered search) and drafts equal to
    an earlier one are dropped; the first ``r`` remaining drafts fill the rows
    and missing rows are all EOS.

    tokens [B, k, L] int; returns (drafts [B, r, length] int32, count [B] int32).
    """
    t = np.asarray(tokens)
    B, k, L = t.shape
    if not (1 <= length <= L) or r < 1:
        raise ValueError("need 1 <= length <= L and r >= 1")
    out = np.full((B, r, length), eos, np.int32)
    cnt = np.zeros(B, np.int32)
    for b in range(B):
        kept = []
        for rank in range(k):
            d = []
            ended = False
            for j in range(length):
                v = int(t[b, rank, j])
                if ended:
                    v = eos
                elif v == eos:
                    ended = True
                d.append(v)
            if d[0] == eos or d in kept:
                continue
            kept.append(d)
            if len(kept) == r:
                break
        for i, d in enumerate(kept):
            out[b, i] = d
        cnt[b] = len(kept)
    return out, cnt
