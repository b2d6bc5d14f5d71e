"""MI355X-native exact dense retrieval for DReSD (Dense Retrieval for
Speculative Decoding): a datastore of L2-normalised token embeddings mapped to
their next tokens (Section 3.5), searched by inner product (Eq. 3 with unit
norms) for the k best keys whose continuations become drafts (Section 3.6).

The search runs in hand-written gfx950 HIP kernels behind the C ABI of
``include/dresd.h``; this module only passes torch device pointers and the
current stream to it.
"""
from __future__ import annotations

import ctypes

from . import _lib
from ._lib import DresdError, K_MAX  # noqa: F401

__all__ = ["Index", "PartitionedIndex", "DresdError", "K_MAX", "transform", "pack_drafts",
           "kmeans_assign", "kmeans_update", "kmeans_init", "train_partitions", "bw_probe"]

_DTYPES = None


def _dtype_code(t):
    import torch
    global _DTYPES
    if _DTYPES is None:
        _DTYPES = {torch.float32: _lib.F32, torch.float16: _lib.F16, torch.bfloat16: _lib.BF16}
    if t.dtype not in _DTYPES:
        raise TypeError("keys must be float32, float16 or bfloat16, not %s" % t.dtype)
    return _DTYPES[t.dtype]


def _stream_handle(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


# dresd_search_plan's scan kinds
SCAN_KINDS = {0: "single_tile", 1: "shared_key", 2: "single_tile_grouped", 3: "tiled"}


class Index:
    """An exact inner-product index over ``keys[N, d]`` with values ``cont[N, L]``.

    Both tensors must be contiguous and on the current GPU; they are copied
    into library-owned memory, so they may be freed after construction.
    """

    def __init__(self, keys, cont, stream=None):
        import torch
        if not (keys.is_cuda and cont.is_cuda):
            raise ValueError("keys and continuations must be GPU tensors")
        if keys.dim() != 2 or cont.dim() != 2 or cont.shape[0] != keys.shape[0]:
            raise ValueError("keys must be [N, d] and continuations [N, L]")
        if cont.dtype != torch.int32:
            raise TypeError("continuations must be int32")
        keys = keys.contiguous()
        cont = cont.contiguous()
        self._lib = _lib.load()
        self._h = ctypes.c_void_p()
        self.N, self.d = int(keys.shape[0]), int(keys.shape[1])
        self.L = int(cont.shape[1])
        self.device = keys.device
        _lib.check(self._lib.dresd_index_create(
            ctypes.c_void_p(keys.data_ptr()), ctypes.c_void_p(cont.data_ptr()), self.N, self.d,
            self.L, _dtype_code(keys), _stream_handle(stream), ctypes.byref(self._h)))

    def search(self, queries, k: int, tokens: bool = True, out=None, stream=None, next_tok=None):
        """Top-k by inner product.  Returns ``(idx int64[B,k], score f32[B,k],
        tokens int32[B,k,L] or None)``.  With ``next_tok`` (int32 GPU tensor
        [B]) only rows whose continuation starts with the query's next token
        compete (Section 3.5); ranks past the matching rows hold idx -1,
        score -inf and zero tokens."""
        import torch
        if not queries.is_cuda or queries.dtype != torch.float32:
            raise TypeError("queries must be a float32 GPU tensor")
        if queries.dim() != 2 or queries.shape[1] != self.d:
            raise ValueError("queries must be [B, %d]" % self.d)
        q = queries.contiguous()
        B = int(q.shape[0])
        if next_tok is not None:
            if not next_tok.is_cuda or next_tok.dtype != torch.int32 or next_tok.numel() != B:
                raise TypeError("next_tok must be an int32 GPU tensor with one token per query")
            next_tok = next_tok.contiguous()
        if out is None:
            idx = torch.empty((B, k), dtype=torch.int64, device=q.device)
            score = torch.empty((B, k), dtype=torch.float32, device=q.device)
            tok = torch.empty((B, k, self.L), dtype=torch.int32, device=q.device) if tokens else None
        else:
            idx, score, tok = out
        tptr = ctypes.c_void_p(tok.data_ptr()) if tok is not None else None
        if next_tok is None:
            _lib.check(self._lib.dresd_search(
                self._h, ctypes.c_void_p(q.data_ptr()), B, int(k),
                ctypes.c_void_p(idx.data_ptr()), ctypes.c_void_p(score.data_ptr()), tptr,
                _stream_handle(stream)))
        else:
            _lib.check(self._lib.dresd_search_filtered(
                self._h, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(next_tok.data_ptr()), B,
                int(k), ctypes.c_void_p(idx.data_ptr()), ctypes.c_void_p(score.data_ptr()), tptr,
                _stream_handle(stream)))
        return idx, score, tok

    def plan(self, B: int, k: int):
        sp, w, ws = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64()
        kind, nl = ctypes.c_int32(), ctypes.c_int32()
        _lib.check(self._lib.dresd_search_plan(self._h, int(B), int(k), ctypes.byref(sp),
                                               ctypes.byref(w), ctypes.byref(ws),
                                               ctypes.byref(kind), ctypes.byref(nl)))
        return {"sample_passes": sp.value, "scan_waves": w.value, "workspace_bytes": ws.value,
                "scan_kernel": SCAN_KINDS[kind.value], "launches": nl.value}

    def profile(self, on: bool = True):
        _lib.check(self._lib.dresd_profile_enable(self._h, 1 if on else 0))

    def profile_read(self):
        a, b, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
        _lib.check(self._lib.dresd_profile_read(self._h, ctypes.byref(a), ctypes.byref(b),
                                                ctypes.byref(n)))
        return {"scan_ms": a.value, "search_ms": b.value, "searches": n.value}

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            self._lib.dresd_index_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _search_out(B, k, L, tokens, device, out):
    import torch
    if out is not None:
        return out
    idx = torch.empty((B, k), dtype=torch.int64, device=device)
    score = torch.empty((B, k), dtype=torch.float32, device=device)
    tok = torch.empty((B, k, L), dtype=torch.int32, device=device) if tokens else None
    return idx, score, tok


class PartitionedIndex:
    """Partitioned (approximate) inner-product index: ``keys[N, d]`` with
    values ``cont[N, L]``, grouped into the partitions ``assign[N]`` (int32 in
    [0, P)) whose unit centroids are ``centroids[P, d]`` (float32).  A search
    probes the ``nprobe`` partitions with the best centroids and returns the
    exact top-k over their keys (the paper's approximate search, Section 3.5,
    read as an inverted file).  Everything is copied at construction."""

    def __init__(self, keys, cont, centroids, assign, stream=None):
        import torch
        for t in (keys, cont, centroids, assign):
            if not t.is_cuda:
                raise ValueError("all inputs must be GPU tensors")
        if keys.dim() != 2 or cont.dim() != 2 or cont.shape[0] != keys.shape[0]:
            raise ValueError("keys must be [N, d] and continuations [N, L]")
        if centroids.dtype != torch.float32 or centroids.dim() != 2 or \
                centroids.shape[1] != keys.shape[1]:
            raise TypeError("centroids must be float32 [P, d]")
        if cont.dtype != torch.int32 or assign.dtype != torch.int32 or \
                assign.numel() != keys.shape[0]:
            raise TypeError("continuations and assign must be int32; assign holds one id per key")
        keys, cont = keys.contiguous(), cont.contiguous()
        centroids, assign = centroids.contiguous(), assign.contiguous()
        self._lib = _lib.load()
        self._h = ctypes.c_void_p()
        self.N, self.d = int(keys.shape[0]), int(keys.shape[1])
        self.L = int(cont.shape[1])
        self.P = int(centroids.shape[0])
        _lib.check(self._lib.dresd_ivf_create(
            ctypes.c_void_p(keys.data_ptr()), ctypes.c_void_p(cont.data_ptr()), self.N, self.d,
            self.L, _dtype_code(keys), ctypes.c_void_p(centroids.data_ptr()), self.P,
            ctypes.c_void_p(assign.data_ptr()), _stream_handle(stream), ctypes.byref(self._h)))

    @classmethod
    def by_first_token(cls, keys, cont, stream=None):
        """Keys grouped by the first token of their continuation (one
        partition per distinct first token, in ascending token order, no
        centroids), for ``search_next_token``.  Copies everything."""
        import torch
        for t in (keys, cont):
            if not t.is_cuda:
                raise ValueError("all inputs must be GPU tensors")
        if keys.dim() != 2 or cont.dim() != 2 or cont.shape[0] != keys.shape[0]:
            raise ValueError("keys must be [N, d] and continuations [N, L]")
        if cont.dtype != torch.int32:
            raise TypeError("continuations must be int32")
        keys, cont = keys.contiguous(), cont.contiguous()
        self = cls.__new__(cls)
        self._lib = _lib.load()
        self._h = ctypes.c_void_p()
        self.N, self.d = int(keys.shape[0]), int(keys.shape[1])
        self.L = int(cont.shape[1])
        _lib.check(self._lib.dresd_ivf_create_by_token(
            ctypes.c_void_p(keys.data_ptr()), ctypes.c_void_p(cont.data_ptr()), self.N, self.d,
            self.L, _dtype_code(keys), _stream_handle(stream), ctypes.byref(self._h)))
        self.P = self.info()["P"]
        return self

    def search_next_token(self, queries, next_tok, k: int, tokens: bool = True, out=None,
                          stream=None):
        """Next-token-filtered exact top-k (the result of ``Index.search``
        with ``next_tok``) over an index from ``by_first_token``: each query
        scans only the keys whose continuation starts with its next token
        (``next_tok``, int32 GPU tensor [B])."""
        q = self._check_q(queries)
        B = int(q.shape[0])
        nt = self._next_tok(next_tok, B)
        if nt is None:
            raise TypeError("next_tok is required")
        idx, score, tok = _search_out(B, k, self.L, tokens, q.device, out)
        _lib.check(self._lib.dresd_ivf_search_next_token(
            self._h, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(nt.data_ptr()), B, int(k),
            ctypes.c_void_p(idx.data_ptr()), ctypes.c_void_p(score.data_ptr()),
            ctypes.c_void_p(tok.data_ptr()) if tok is not None else None, _stream_handle(stream)))
        return idx, score, tok

    def _check_q(self, queries):
        import torch
        if not queries.is_cuda or queries.dtype != torch.float32:
            raise TypeError("queries must be a float32 GPU tensor")
        if queries.dim() != 2 or queries.shape[1] != self.d:
            raise ValueError("queries must be [B, %d]" % self.d)
        return queries.contiguous()

    @staticmethod
    def _next_tok(next_tok, B):
        import torch
        if next_tok is None:
            return None
        if not next_tok.is_cuda or next_tok.dtype != torch.int32 or next_tok.numel() != B:
            raise TypeError("next_tok must be an int32 GPU tensor with one token per query")
        return next_tok.contiguous()

    def search(self, queries, k: int, nprobe: int, tokens: bool = True, out=None, stream=None,
               next_tok=None):
        """Top-k over the keys of the ``nprobe`` best partitions (with
        ``next_tok``, int32 GPU tensor [B], only keys whose continuation starts
        with the query's next token).  Returns ``(idx, score, tokens)`` as
        ``Index.search``; ranks past the admitted keys hold idx -1, score -inf
        and zero tokens."""
        q = self._check_q(queries)
        B = int(q.shape[0])
        nt = self._next_tok(next_tok, B)
        idx, score, tok = _search_out(B, k, self.L, tokens, q.device, out)
        args = (ctypes.c_void_p(idx.data_ptr()), ctypes.c_void_p(score.data_ptr()),
                ctypes.c_void_p(tok.data_ptr()) if tok is not None else None,
                _stream_handle(stream))
        if nt is None:
            _lib.check(self._lib.dresd_ivf_search(
                self._h, ctypes.c_void_p(q.data_ptr()), B, int(k), int(nprobe), *args))
        else:
            _lib.check(self._lib.dresd_ivf_search_filtered(
                self._h, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(nt.data_ptr()), B, int(k),
                int(nprobe), *args))
        return idx, score, tok

    def search_probes(self, queries, probes, k: int, tokens: bool = True, out=None, stream=None,
                      next_tok=None):
        """Top-k over the keys of the partitions in ``probes`` (int32 GPU
        tensor [B, S]; ids outside [0, P) ignored, repeats counted once),
        optionally next-token filtered."""
        import torch
        q = self._check_q(queries)
        B = int(q.shape[0])
        if not probes.is_cuda or probes.dtype != torch.int32 or probes.dim() != 2 or \
                probes.shape[0] != B:
            raise TypeError("probes must be an int32 GPU tensor [B, S]")
        pr = probes.contiguous()
        nt = self._next_tok(next_tok, B)
        idx, score, tok = _search_out(B, k, self.L, tokens, q.device, out)
        _lib.check(self._lib.dresd_ivf_search_probes(
            self._h, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(pr.data_ptr()),
            int(pr.shape[1]), ctypes.c_void_p(nt.data_ptr()) if nt is not None else None, B,
            int(k), ctypes.c_void_p(idx.data_ptr()), ctypes.c_void_p(score.data_ptr()),
            ctypes.c_void_p(tok.data_ptr()) if tok is not None else None, _stream_handle(stream)))
        return idx, score, tok

    def info(self):
        N, d, L, dt, P, T = (ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32(),
                             ctypes.c_int32(), ctypes.c_int64())
        _lib.check(self._lib.dresd_ivf_info(self._h, ctypes.byref(N), ctypes.byref(d),
                                            ctypes.byref(L), ctypes.byref(dt), ctypes.byref(P),
                                            ctypes.byref(T)))
        return {"N": N.value, "d": d.value, "L": L.value, "dtype": dt.value, "P": P.value,
                "tiles": T.value}

    def profile(self, on: bool = True):
        _lib.check(self._lib.dresd_ivf_profile_enable(self._h, 1 if on else 0))

    def profile_read(self):
        a, b, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
        _lib.check(self._lib.dresd_ivf_profile_read(self._h, ctypes.byref(a), ctypes.byref(b),
                                                    ctypes.byref(n)))
        return {"scan_ms": a.value, "search_ms": b.value, "searches": n.value}

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            self._lib.dresd_ivf_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def transform(x, mean, var, W, eps_z: float = 1e-5, eps_n: float = 1e-12, out=None, stream=None):
    """Query-side transform of Algorithm 1 steps 4-6 on the GPU: z-score
    normalisation (Eq. 1), projection onto the principal components W
    ([D, l], Section 3.3) and L2 normalisation (Eq. 2).  All tensors are
    float32 on the GPU; returns y [M, l]."""
    import torch
    for name, t in (("x", x), ("mean", mean), ("var", var), ("W", W)):
        if not t.is_cuda or t.dtype != torch.float32:
            raise TypeError("%s must be a float32 GPU tensor" % name)
    if x.dim() != 2 or W.dim() != 2 or W.shape[0] != x.shape[1]:
        raise ValueError("x must be [M, D] and W [D, l]")
    M, D = int(x.shape[0]), int(x.shape[1])
    l = int(W.shape[1])
    if mean.numel() != D or var.numel() != D:
        raise ValueError("mean and var must hold D values")
    x, mean, var, W = x.contiguous(), mean.contiguous(), var.contiguous(), W.contiguous()
    y = torch.empty((M, l), dtype=torch.float32, device=x.device) if out is None else out
    lib = _lib.load()
    _lib.check(lib.dresd_transform(ctypes.c_void_p(x.data_ptr()), M, D,
                                   ctypes.c_void_p(mean.data_ptr()),
                                   ctypes.c_void_p(var.data_ptr()), float(eps_z),
                                   ctypes.c_void_p(W.data_ptr()), l, float(eps_n),
                                   ctypes.c_void_p(y.data_ptr()), _stream_handle(stream)))
    return y


def pack_drafts(tokens, r: int, length: int, eos: int = 0, out=None, stream=None):
    """Draft assembly for batch verification (Section 3.6) on the GPU: tokens
    [B, k, L] int32 (from ``Index.search``) -> (drafts [B, r, length] int32,
    count [B] int32): EOS-padded rows, drafts starting with EOS and repeats
    dropped in rank order."""
    import torch
    if not tokens.is_cuda or tokens.dtype != torch.int32 or tokens.dim() != 3:
        raise TypeError("tokens must be an int32 GPU tensor [B, k, L]")
    B, k, L = (int(s) for s in tokens.shape)
    t = tokens.contiguous()
    if out is None:
        drafts = torch.empty((B, r, length), dtype=torch.int32, device=t.device)
        count = torch.empty((B,), dtype=torch.int32, device=t.device)
    else:
        drafts, count = out
    lib = _lib.load()
    _lib.check(lib.dresd_pack_drafts(ctypes.c_void_p(t.data_ptr()), B, k, L, int(r), int(length),
                                     int(eos), ctypes.c_void_p(drafts.data_ptr()),
                                     ctypes.c_void_p(count.data_ptr()), _stream_handle(stream)))
    return drafts, count


def _rows(x):
    if not x.is_cuda or x.dim() != 2:
        raise TypeError("rows must be a GPU tensor [n, d]")
    return x.contiguous()


def kmeans_assign(x, centroids, with_score: bool = False, stream=None):
    """Nearest centroid by inner product for every row of ``x`` ([n, d],
    float32/float16/bfloat16 on the GPU; ``centroids`` float32 [P, d]), ties
    to the lower id.  Returns assign int32 [n] (and the fp32 scores)."""
    import torch
    x = _rows(x)
    c = centroids.contiguous()
    if c.dtype != torch.float32 or c.dim() != 2 or c.shape[1] != x.shape[1]:
        raise TypeError("centroids must be float32 [P, d]")
    n, d = int(x.shape[0]), int(x.shape[1])
    a = torch.empty((n,), dtype=torch.int32, device=x.device)
    sc = torch.empty((n,), dtype=torch.float32, device=x.device) if with_score else None
    _lib.check(_lib.load().dresd_kmeans_assign(
        ctypes.c_void_p(x.data_ptr()), n, d, _dtype_code(x), ctypes.c_void_p(c.data_ptr()),
        int(c.shape[0]), ctypes.c_void_p(a.data_ptr()),
        ctypes.c_void_p(sc.data_ptr()) if sc is not None else None, _stream_handle(stream)))
    return (a, sc) if with_score else a


def kmeans_update(x, assign, centroids, stream=None):
    """Spherical k-means update in place: each centroid (float32 [P, d],
    contiguous) becomes the unit vector along the sum of its rows (unchanged
    without rows).  Returns the rows per centroid (int32 [P])."""
    import torch
    x = _rows(x)
    if not centroids.is_contiguous() or centroids.dtype != torch.float32:
        raise TypeError("centroids must be a contiguous float32 tensor [P, d]")
    if assign.dtype != torch.int32 or assign.numel() != x.shape[0]:
        raise TypeError("assign must be int32 with one entry per row")
    a = assign.contiguous()
    P = int(centroids.shape[0])
    counts = torch.empty((P,), dtype=torch.int32, device=x.device)
    _lib.check(_lib.load().dresd_kmeans_update(
        ctypes.c_void_p(x.data_ptr()), int(x.shape[0]), int(x.shape[1]), _dtype_code(x),
        ctypes.c_void_p(a.data_ptr()), P, ctypes.c_void_p(centroids.data_ptr()),
        ctypes.c_void_p(counts.data_ptr()), _stream_handle(stream)))
    return counts


def kmeans_init(x, P: int, seed: int = 0, stream=None):
    """Starting centroids of spherical k-means (float32 [P, d]): P distinct
    rows of ``x`` at even spacing through the row order from an offset drawn
    from ``seed`` (SplitMix64), each scaled to unit length."""
    import torch
    x = _rows(x)
    n, d = int(x.shape[0]), int(x.shape[1])
    if not (1 <= P <= n):
        raise ValueError("need 1 <= P <= n")
    if not (0 <= seed < 1 << 64):
        raise ValueError("seed must be in [0, 2^64)")
    centroids = torch.empty((P, d), dtype=torch.float32, device=x.device)
    _lib.check(_lib.load().dresd_kmeans_init(
        ctypes.c_void_p(x.data_ptr()), n, d, _dtype_code(x), P, seed,
        ctypes.c_void_p(centroids.data_ptr()), _stream_handle(stream)))
    return centroids


def train_partitions(x, P: int, iters: int = 10, seed: int = 0, stream=None):
    """Spherical k-means on the GPU: P centroids started by kmeans_init, then
    ``iters`` assign + update steps.  Returns (centroids float32 [P, d],
    assign int32 [n])."""
    x = _rows(x)
    centroids = kmeans_init(x, P, seed, stream)
    for _ in range(iters):
        assign = kmeans_assign(x, centroids, stream=stream)
        kmeans_update(x, assign, centroids, stream)
    return centroids, kmeans_assign(x, centroids, stream=stream)


def bw_probe(buf, reps: int = 10, workgroups: int = 0, stream=None) -> float:
    """Achievable HBM read bandwidth with the scans' access pattern: reads
    every byte of the GPU tensor ``buf`` (contents irrelevant; whole 1 KiB
    blocks, at least 1 MiB) ``reps`` times after one untimed pass with
    ``workgroups`` workgroups (0: four per compute unit).  Returns GB/s."""
    if not buf.is_cuda:
        raise ValueError("buf must be a GPU tensor")
    nbytes = buf.numel() * buf.element_size() // 1024 * 1024
    lib = _lib.load()
    ms = ctypes.c_double()
    _lib.check(lib.dresd_bw_probe(ctypes.c_void_p(buf.data_ptr()), nbytes, int(reps),
                                  int(workgroups), ctypes.byref(ms), _stream_handle(stream)))
    return nbytes / (ms.value * 1e-3) / 1e9
