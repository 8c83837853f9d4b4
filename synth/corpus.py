"""Synthetic codebooks and CSR document batches (seeded, deterministic).

Conventions (one reading each of what the workload description leaves open):

* Codebook row ``f`` of configuration ``c`` is
  ``default_rng([seed, c, 1, f]).random(N, dtype=float32)``.  numpy's float32
  path returns ``k * 2**-24`` with integer ``0 <= k < 2**24``, so every weight
  is exactly representable in fp32 and fp64 and each row can be regenerated on
  its own (the oracle never needs a device copy).
* Term frequencies follow a truncated Zipf law, ``p(r) ~ r**-s`` for ranks
  ``r = 1..F``, and feature id ``r - 1`` (ids ordered by descending
  frequency, the relabelling the paper keeps as its substrate).
* "Drawn without replacement" is successive sampling proportional to weight:
  i.i.d. draws with the first occurrence of each feature kept until the
  document holds its target count.  Documents that need very many draws (a
  target close to the support size) are completed with the equivalent
  exponential-race construction over their support.
* ``Poisson(mean, min 1)`` is ``max(1, k)``; ``lognormal(median m, sigma s,
  clipped lo..hi)`` is ``clip(rint(m * exp(s * Z)), lo, hi)``; every target is
  further clipped to the size of the document's support.
* Topic workload: each of the topics owns a uniformly random subset of the
  vocabulary in random rank order with Zipf(s) over rank; a document mixes
  1..3 distinct topics with equal weight; each draw picks one of its topics
  uniformly, then a feature from that topic's law.
* Streams: codebook rows ``[seed, c, 1, f]``, batch ``b`` of documents
  ``[seed, c, 2, b]``, topic subsets ``[seed, c, 3]``.

Documents are returned as CSR with int32 ``indptr``/``indices`` and strictly
ascending indices within each row.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Optional, Sequence, Tuple

import numpy as np


@dataclass(frozen=True)
class Config:
    key: int
    name: str
    N: int                 # neurons (map side squared)
    F: int                 # vocabulary size
    docs: int              # documents in one full pass
    batch: int             # documents per CSR batch
    nnz: Tuple             # ("poisson", mean) or ("lognormal", median, sigma, lo, hi)
    zipf_s: float = 1.1
    topics: int = 0        # 0 = one global Zipf law over F
    topic_size: int = 0
    topics_per_doc: Tuple[int, int] = (1, 3)


CONFIGS = {
    1: Config(1, "map32x32-F2048-10k", 1024, 2048, 10_000, 10_000, ("poisson", 20.0)),
    2: Config(2, "map128x128-F20000-1M", 16384, 20_000, 1_000_000, 65_536, ("poisson", 80.0)),
    3: Config(3, "map256x256-F20000-4M", 65536, 20_000, 4_000_000, 1_048_576,
              ("lognormal", 70.0, 0.6, 1, 2000)),
    4: Config(4, "map512x512-F20000-2M", 262144, 20_000, 2_000_000, 1_048_576, ("poisson", 80.0)),
    5: Config(5, "map512x512-F20000-26.9M-topics", 262144, 20_000, 26_900_000, 1_000_000,
              ("lognormal", 80.0, 0.7, 1, 4000), topics=256, topic_size=2000),
}


def _cfg(cfg) -> Config:
    return cfg if isinstance(cfg, Config) else CONFIGS[int(cfg)]


def batch_sizes(cfg) -> list:
    """Document counts of the batches of one full pass (last one ragged)."""
    c = _cfg(cfg)
    full, rest = divmod(c.docs, c.batch)
    return [c.batch] * full + ([rest] if rest else [])


# ----------------------------------------------------------------------------
# Codebook
# ----------------------------------------------------------------------------

def codebook_rows(cfg, rows: Sequence[int], seed: int = 0, N: Optional[int] = None) -> np.ndarray:
    """Rows ``rows`` of the codebook as float32 [len(rows), N]."""
    c = _cfg(cfg)
    n = c.N if N is None else int(N)
    out = np.empty((len(rows), n), np.float32)
    for i, f in enumerate(rows):
        np.random.default_rng([seed, c.key, 1, int(f)]).random(n, dtype=np.float32, out=out[i])
    return out


def codebook(cfg, seed: int = 0, ldw: Optional[int] = None, N: Optional[int] = None,
             F: Optional[int] = None, out: Optional[np.ndarray] = None,
             threads: Optional[int] = None) -> np.ndarray:
    """Feature-major codebook W[F][ldw] (float32); columns N..ldw-1 are zero.

    ``out`` may be any writable float32 array of shape [F, ldw] (for example a
    pinned host tensor's numpy view); rows are filled by a thread pool.
    """
    c = _cfg(cfg)
    n = c.N if N is None else int(N)
    f_count = c.F if F is None else int(F)
    ld = n if ldw is None else int(ldw)
    if ld < n:
        raise ValueError("ldw < N")
    if out is None:
        out = np.empty((f_count, ld), np.float32)
    if out.shape != (f_count, ld) or out.dtype != np.float32:
        raise ValueError("out has the wrong shape or dtype")

    def fill(f: int) -> None:
        np.random.default_rng([seed, c.key, 1, f]).random(n, dtype=np.float32, out=out[f, :n])
        if ld > n:
            out[f, n:] = 0.0

    nthreads = threads or min(16, os.cpu_count() or 1)
    if nthreads <= 1 or f_count < 64:
        for f in range(f_count):
            fill(f)
    else:
        with ThreadPoolExecutor(nthreads) as ex:
            list(ex.map(fill, range(f_count), chunksize=32))
    return out


# ----------------------------------------------------------------------------
# Documents
# ----------------------------------------------------------------------------

def zipf_cdf(n: int, s: float) -> np.ndarray:
    """CDF of the truncated Zipf law p(r) ~ r**-s over ranks 1..n (float64)."""
    w = np.arange(1, n + 1, dtype=np.float64) ** (-float(s))
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    return cdf


class _ZipfRank:
    """Exact ``searchsorted(cdf, u, side="right")`` through a guide table.

    Bucket ``b = floor(u * 2**20)`` bounds the answer between the ranks of the
    bucket's two edges; a few vectorised steps walk the (short) gap.
    """

    BITS = 20

    def __init__(self, cdf: np.ndarray):
        self.cdf = cdf
        edges = np.arange((1 << self.BITS) + 1, dtype=np.float64) / float(1 << self.BITS)
        g = np.searchsorted(cdf, edges, side="right")
        self.guide = g[:-1].astype(np.int64)
        self.steps = int(np.max(g[1:] - g[:-1]))
        self.n = len(cdf)

    def __call__(self, u: np.ndarray) -> np.ndarray:
        r = self.guide[(u * float(1 << self.BITS)).astype(np.int64)]
        for _ in range(self.steps):
            r += self.cdf[np.minimum(r, self.n - 1)] <= u
        return np.minimum(r, self.n - 1)


def _zipf_pmf(n: int, s: float) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-float(s))
    return w / w.sum()


def topic_subsets(cfg, seed: int = 0) -> np.ndarray:
    """[topics, topic_size] int32: row t lists topic t's features in rank order."""
    c = _cfg(cfg)
    if not c.topics:
        raise ValueError("configuration has no topics")
    rng = np.random.default_rng([seed, c.key, 3])
    out = np.empty((c.topics, c.topic_size), np.int32)
    for t in range(c.topics):
        out[t] = rng.choice(c.F, size=c.topic_size, replace=False)
    return out


def _targets(rng, spec, n: int) -> np.ndarray:
    kind = spec[0]
    if kind == "poisson":
        k = rng.poisson(spec[1], n).astype(np.int64)
        return np.maximum(k, 1)
    if kind == "lognormal":
        med, sig, lo, hi = spec[1:]
        z = rng.standard_normal(n)
        k = np.rint(med * np.exp(sig * z)).astype(np.int64)
        return np.clip(k, lo, hi)
    raise ValueError(f"unknown nnz law {kind!r}")


def _first_distinct(D: np.ndarray, k: np.ndarray):
    """Per row of draws D [c, M]: which draws are the first k[i] distinct values.

    Returns (done [c], keep [c, M] in value-sorted order, values [c, M] sorted
    ascending along each row).  ``keep`` marks, for rows that reached k[i]
    distinct values, exactly the first occurrences of the first k[i] distinct
    values in draw order.
    """
    c, m = D.shape
    if m >= (1 << 16) or (int(D.max(initial=0)) >= (1 << 15)):
        raise ValueError("draw block too large for packed keys")
    pos = np.arange(m, dtype=np.int32)[None, :]
    key = np.sort((D.astype(np.int32) << 16) | pos, axis=1)
    val = key >> 16
    first = np.ones((c, m), dtype=bool)
    first[:, 1:] = val[:, 1:] != val[:, :-1]
    fpos = np.where(first, key & 0xFFFF, np.int32(1 << 30))
    nfirst = np.count_nonzero(first, axis=1)
    done = nfirst >= k
    kk = np.minimum(k, m).astype(np.int64)
    # k-th smallest first-occurrence position of each row
    kth = np.take_along_axis(np.sort(fpos, axis=1), (kk - 1)[:, None], 1)
    keep = first & (fpos <= kth)
    return done, keep, val


def _exp_race(rng, support: np.ndarray, weight: np.ndarray, k: int) -> np.ndarray:
    """k distinct items of ``support`` by successive sampling ~ ``weight``.

    Exponential race: item i gets key E_i / w_i with E_i ~ Exp(1); the k
    smallest keys are, in order, a successive sample proportional to w.
    """
    keys = rng.standard_exponential(len(support)) / weight
    pick = np.argpartition(keys, k - 1)[:k] if k < len(support) else np.arange(len(support))
    return np.sort(support[pick]).astype(np.int32)


def documents(cfg, batch: int = 0, seed: int = 0, n_docs: Optional[int] = None):
    """CSR batch ``batch`` of configuration ``cfg``: (indptr int32[B+1], indices int32[nnz]).

    ``n_docs`` overrides the batch size (a prefix-shaped smaller batch drawn
    from the same stream layout, used by tests).
    """
    c = _cfg(cfg)
    sizes = batch_sizes(c)
    B = sizes[batch] if n_docs is None else int(n_docs)
    rng = np.random.default_rng([seed, c.key, 2, int(batch)])
    k = _targets(rng, c.nnz, B)
    s = c.zipf_s

    if c.topics:
        subsets = topic_subsets(c, seed)
        lo, hi = c.topics_per_doc
        ntop = rng.integers(lo, hi + 1, B)
        # hi distinct topics per document, uniformly without replacement
        # (sequential draws from the remaining topics); the first ntop are used
        doc_topics = np.empty((B, hi), np.int64)
        for j in range(hi):
            t = rng.integers(0, c.topics - j, B)
            taken = np.sort(doc_topics[:, :j], axis=1)
            for q in range(j):
                t += t >= taken[:, q]
            doc_topics[:, j] = t
        zr = _ZipfRank(zipf_cdf(c.topic_size, s))
        pmf = _zipf_pmf(c.topic_size, s)

        def doc_support(d: int) -> np.ndarray:
            return np.unique(subsets[doc_topics[d, :ntop[d]]].reshape(-1))

        # the support has at least topic_size features, so only larger targets
        # can be clipped by it
        for d in np.nonzero(k > c.topic_size)[0]:
            k[d] = min(k[d], doc_support(int(d)).size)

        def draw(docs: np.ndarray, m: int) -> np.ndarray:
            tsel = (rng.random((docs.size, m)) * ntop[docs, None]).astype(np.int64)
            topic = np.take_along_axis(doc_topics[docs].astype(np.int64), tsel, 1)
            rank = zr(rng.random((docs.size, m)))
            return subsets[topic, rank].astype(np.int32)

        def race(d: int) -> np.ndarray:
            t = doc_topics[d, :ntop[d]]
            feats = subsets[t].reshape(-1)
            w = np.tile(pmf, len(t)) / len(t)
            order = np.argsort(feats, kind="stable")
            fs, ws = feats[order], w[order]
            uniq, start = np.unique(fs, return_index=True)
            wsum = np.add.reduceat(ws, start)
            return _exp_race(rng, uniq, wsum, int(k[d]))
    else:
        k = np.minimum(k, c.F)
        zr = _ZipfRank(zipf_cdf(c.F, s))
        pmf = _zipf_pmf(c.F, s)
        ids = np.arange(c.F, dtype=np.int32)

        def draw(docs: np.ndarray, m: int) -> np.ndarray:
            return zr(rng.random((docs.size, m))).astype(np.int32)

        def race(d: int) -> np.ndarray:
            return _exp_race(rng, ids, pmf, int(k[d]))

    indptr = np.zeros(B + 1, np.int64)
    indptr[1:] = np.cumsum(k)
    if indptr[-1] > np.iinfo(np.int32).max:
        raise ValueError("batch too large for int32 CSR")
    indices = np.empty(int(indptr[-1]), np.int32)

    pending = np.arange(B)
    m_scale = 1.0
    rounds = 0
    while pending.size and rounds < 3:
        kk = k[pending]
        m_of = (np.ceil((1.35 * kk + 24) * m_scale / 16.0) * 16).astype(np.int64)
        nxt = []
        for m in np.unique(m_of):
            grp = pending[m_of == m]
            chunk = max(1, (1 << 21) // int(m))
            for a in range(0, grp.size, chunk):
                docs = grp[a:a + chunk]
                D = draw(docs, int(m))
                done, keep, val = _first_distinct(D, k[docs])
                dd = docs[done]
                if dd.size:
                    kp = keep[done]
                    out_pos = indptr[dd][:, None] + np.cumsum(kp, axis=1) - 1
                    indices[out_pos[kp]] = val[done][kp]
                nxt.append(docs[~done])
        pending = np.sort(np.concatenate(nxt)) if nxt else np.empty(0, np.int64)
        m_scale *= 3.0
        rounds += 1
    for d in pending:
        d = int(d)
        indices[indptr[d]:indptr[d + 1]] = race(d)
    return indptr.astype(np.int32), indices
