"""fp64 oracle of the best-matching-unit (BMU) search (test infrastructure).

What the path computes (paper, Section 3 "Background: the design being
tuned"): a self-organizing map is trained by finding, for every document, the
neuron whose weight vector is closest to it -- its best-matching unit -- and
the search is exact (an exact argmin, invariant to how the codebook is
stored).  The codebook is stored feature-major: feature ``v``'s weight for
neuron ``i`` sits at ``W[v*M + i]`` (same section), so the sparse binary
document turns the search into a sparse-dense product over the document's
features.  For a binary document with feature set S the squared Euclidean
distance expands to

    d_j = sum_f (x_f - W[f, j])^2 = |S| + ||w_j||^2 - 2 * sum_{f in S} W[f, j],

and the BMU is argmin_j d_j.  Readings taken where the paper is silent (all
listed with the design notes): ties go to the lowest neuron index; the
returned distance is the full squared distance above (not its square root);
empty documents are allowed (d_j = ||w_j||^2); a document's feature ids are
strictly ascending (the vector is binary).

Every function here is a direct evaluation of a definition, in fp64, with no
blocking or reordering beyond what numpy's own reductions do.  Pins (tests
that tie this module to something other than itself): hand-worked dyadic
examples, the dense brute force ``bmu_search_dense`` in exact rational
arithmetic, the exact integer evaluation ``bmu_search_exact``, and
invariances (document order, feature relabelling, tile size and tile
membership).

``cluster_order`` implements a reading of "tile-membership clustering" (the
paper, Section 4.2, gives the goal -- documents sharing rare descriptors in
the same tile -- but no algorithm); its pins are hand-worked orderings and
the permutation's invariants, so its *quality* is a reading, while its
*definition* is pinned.
"""

from __future__ import annotations

from fractions import Fraction
from typing import Iterable, Optional, Tuple

import numpy as np


def _rows(indptr: np.ndarray, indices: np.ndarray, d: int) -> np.ndarray:
    a, b = int(indptr[d]), int(indptr[d + 1])
    s = np.asarray(indices[a:b], dtype=np.int64)
    if s.size > 1 and not np.all(s[1:] > s[:-1]):
        raise ValueError(f"document {d}: feature ids must be strictly ascending")
    return s


# ----------------------------------------------------------------------------
# Codebook norms ||w_j||^2 (Section 3; the "norms" kernel of Table 4)
# ----------------------------------------------------------------------------

def codebook_norms(W: np.ndarray, N: Optional[int] = None) -> np.ndarray:
    """||w_j||^2 = sum_f W[f, j]^2 in fp64 for j < N (W is [F, ldw])."""
    n = W.shape[1] if N is None else int(N)
    Wd = np.asarray(W[:, :n], dtype=np.float64)
    return np.einsum("fj,fj->j", Wd, Wd)


def codebook_norms_blocks(blocks: Iterable[np.ndarray]) -> np.ndarray:
    """Same definition, accumulated over row blocks of a large codebook."""
    acc = None
    for blk in blocks:
        b = np.asarray(blk, dtype=np.float64)
        part = np.einsum("fj,fj->j", b, b)
        acc = part if acc is None else acc + part
    if acc is None:
        raise ValueError("no rows")
    return acc


# ----------------------------------------------------------------------------
# BMU search (Section 3), direct per-document definition
# ----------------------------------------------------------------------------

def doc_distances(W: np.ndarray, norms: np.ndarray, feats: np.ndarray, N: Optional[int] = None) -> np.ndarray:
    """d_j for one document with feature set ``feats`` (fp64, all j < N)."""
    n = norms.shape[0] if N is None else int(N)
    dot = np.asarray(W[feats, :n], dtype=np.float64).sum(axis=0) if feats.size else np.zeros(n)
    return float(feats.size) + np.asarray(norms[:n], dtype=np.float64) - 2.0 * dot


def bmu_search(W: np.ndarray, indptr: np.ndarray, indices: np.ndarray,
               norms: Optional[np.ndarray] = None, N: Optional[int] = None,
               docs: Optional[Iterable[int]] = None):
    """Exact BMU of each document (or of the documents listed in ``docs``).

    Returns (bmu int64, dist fp64, second int64, dist2 fp64) where ``second``
    is the best neuron other than the BMU (-1 and +inf when N == 1).
    """
    n = W.shape[1] if N is None else int(N)
    if norms is None:
        norms = codebook_norms(W, n)
    doc_list = range(len(indptr) - 1) if docs is None else list(docs)
    m = len(doc_list)
    bmu = np.empty(m, np.int64)
    dist = np.empty(m, np.float64)
    j2 = np.full(m, -1, np.int64)
    d2 = np.full(m, np.inf, np.float64)
    for i, d in enumerate(doc_list):
        dd = doc_distances(W, norms, _rows(indptr, indices, d), n)
        b = int(np.argmin(dd))          # first occurrence: ties -> lowest index
        bmu[i], dist[i] = b, dd[b]
        if n > 1:
            dd[b] = np.inf
            s = int(np.argmin(dd))
            j2[i], d2[i] = s, dd[s]
    return bmu, dist, j2, d2


def bmu_search_dense(W, indptr, indices, N: Optional[int] = None):
    """Brute force in exact rational arithmetic: d_j = sum_f (x_f - W[f,j])^2.

    For tiny inputs only (pure Python).  W entries are converted exactly from
    their binary floating-point values.
    """
    F = W.shape[0]
    n = W.shape[1] if N is None else int(N)
    Wq = [[Fraction(float(W[f, j])) for j in range(n)] for f in range(F)]
    out_b, out_d = [], []
    for d in range(len(indptr) - 1):
        s = set(int(v) for v in indices[int(indptr[d]):int(indptr[d + 1])])
        best = None
        for j in range(n):
            dj = sum(((1 if f in s else 0) - Wq[f][j]) ** 2 for f in range(F))
            if best is None or dj < best[1]:
                best = (j, dj)
        out_b.append(best[0])
        out_d.append(best[1])
    return out_b, out_d


def bmu_search_exact(K: np.ndarray, bits: int, indptr: np.ndarray, indices: np.ndarray,
                     N: Optional[int] = None):
    """Exact integer evaluation for dyadic codebooks W = K * 2**-bits.

    2**(2*bits) * d_j = |S| * 2**(2*bits) + sum_f K[f,j]^2 - 2**(bits+1) * sum_{f in S} K[f,j]
    computed in Python integers (no rounding anywhere).  Returns, per
    document, (bmu, scaled distance, sorted list of all tied minimisers).
    """
    n = K.shape[1] if N is None else int(N)
    Kp = [[int(K[f, j]) for j in range(n)] for f in range(K.shape[0])]
    sq = [sum(Kp[f][j] * Kp[f][j] for f in range(K.shape[0])) for j in range(n)]
    one = 1 << (2 * bits)
    res = []
    for d in range(len(indptr) - 1):
        s = [int(v) for v in indices[int(indptr[d]):int(indptr[d + 1])]]
        vals = []
        for j in range(n):
            dot = sum(Kp[f][j] for f in s)
            vals.append(len(s) * one + sq[j] - (dot << (bits + 1)))
        m = min(vals)
        ties = [j for j, v in enumerate(vals) if v == m]
        res.append((ties[0], m, ties))
    return res


# ----------------------------------------------------------------------------
# Tile plan (Section 4.1): the union of the distinct features of a tile
# ----------------------------------------------------------------------------

def tile_union(indptr: np.ndarray, indices: np.ndarray, T: int, perm: Optional[np.ndarray] = None):
    """Per tile of T consecutive (permuted) documents: sorted union + membership.

    Tile t holds documents perm[t*T : (t+1)*T] (identity when perm is None);
    the last tile may be short.  Returns a list of (features int64[U],
    masks[U]) where bit s of masks[u] is set iff the tile's s-th document
    contains features[u] (uint64 for T <= 64, Python ints beyond).
    """
    B = len(indptr) - 1
    order = np.arange(B) if perm is None else np.asarray(perm, dtype=np.int64)
    out = []
    for t0 in range(0, B, T):
        members = {}
        for s, d in enumerate(order[t0:t0 + T]):
            for f in _rows(indptr, indices, int(d)):
                members[int(f)] = members.get(int(f), 0) | (1 << s)
        feats = np.array(sorted(members), dtype=np.int64)
        masks = np.array([members[int(f)] for f in feats], dtype=np.uint64 if T <= 64 else object)
        out.append((feats, masks))
    return out


def bmu_search_tiled(W: np.ndarray, indptr: np.ndarray, indices: np.ndarray, T: int,
                     perm: Optional[np.ndarray] = None, norms: Optional[np.ndarray] = None,
                     N: Optional[int] = None):
    """The tiled evaluation (Section 4.1): sweep each tile's union once.

    For every tile, each union feature's weight row is read once and added
    to the accumulator of every member document.  Results are mapped back to
    input order.  In fp64 with dyadic weights every sum is exact, so this
    must equal ``bmu_search`` bit for bit, for any T and any perm.
    """
    n = W.shape[1] if N is None else int(N)
    if norms is None:
        norms = codebook_norms(W, n)
    B = len(indptr) - 1
    order = np.arange(B) if perm is None else np.asarray(perm, dtype=np.int64)
    bmu = np.empty(B, np.int64)
    dist = np.empty(B, np.float64)
    for t, (feats, masks) in enumerate(tile_union(indptr, indices, T, perm)):
        docs = order[t * T:(t + 1) * T]
        acc = np.zeros((len(docs), n))
        for f, m in zip(feats, masks):
            row = np.asarray(W[f, :n], dtype=np.float64)
            for s in range(len(docs)):
                if (int(m) >> s) & 1:
                    acc[s] += row
        for s, d in enumerate(docs):
            nnz = int(indptr[d + 1] - indptr[d])
            dd = nnz + np.asarray(norms[:n], dtype=np.float64) - 2.0 * acc[s]
            b = int(np.argmin(dd))
            bmu[d], dist[d] = b, dd[b]
    return bmu, dist


# ----------------------------------------------------------------------------
# Tile-membership clustering (Section 4.2), one reading
# ----------------------------------------------------------------------------

def cluster_order(indptr: np.ndarray, indices: np.ndarray, F: int) -> np.ndarray:
    """Permutation that groups documents sharing their dominant features.

    Reading of "cluster the corpus so that articles sharing descriptors fall
    in the same tile" with no labels: let df(f) be the number of documents
    of the batch containing f; a document's signature is (s1, s2), its two
    features of highest df (ties to the lower feature id; F stands in for a
    missing feature).  Documents are ordered by (s1, s2, input position).
    perm[i] is the input index of the document placed at position i.
    """
    B = len(indptr) - 1
    df = np.zeros(F, np.int64)
    for d in range(B):
        for f in _rows(indptr, indices, d):
            df[f] += 1
    keys = []
    for d in range(B):
        fs = [int(f) for f in _rows(indptr, indices, d)]
        ranked = sorted(fs, key=lambda f: (-df[f], f))
        s1 = ranked[0] if len(ranked) > 0 else F
        s2 = ranked[1] if len(ranked) > 1 else F
        keys.append((s1, s2, d))
    keys.sort()
    return np.array([k[2] for k in keys], dtype=np.int64)


# ----------------------------------------------------------------------------
# Acceptance rule for a device result against this oracle
# ----------------------------------------------------------------------------

def accept_bmu(W: np.ndarray, norms: np.ndarray, feats: np.ndarray, g: int, dist_g: float,
               rel: float = 1e-5, N: Optional[int] = None) -> Tuple[bool, str]:
    """Check one device answer (index g, distance dist_g) for one document.

    Index: g is accepted iff it is the oracle's BMU b, or d[g] <= d[b] * (1 + rel)
    (g lies in the oracle's near-tie band: the top two differ by < rel
    relative).  Distance: |dist_g - d[g]| <= rel * d[g]; when d[g] has
    cancelled to below 1e-3 of its condition scale |S| + ||w_g||^2 + 2|dot_g|,
    the bound is rel times that scale instead.
    """
    n = norms.shape[0] if N is None else int(N)
    dd = doc_distances(W, norms, feats, n)
    if not (0 <= g < n):
        return False, f"index {g} out of range"
    b = int(np.argmin(dd))
    if g != b and not dd[g] <= dd[b] + rel * abs(dd[b]):
        return False, f"index {g} (d={dd[g]!r}) outside near-tie band of bmu {b} (d={dd[b]!r})"
    dot_g = (float(feats.size) + float(norms[g]) - dd[g]) / 2.0
    scale = float(feats.size) + float(norms[g]) + 2.0 * abs(dot_g)
    ref = abs(dd[g]) if abs(dd[g]) >= 1e-3 * scale else scale
    if abs(float(dist_g) - dd[g]) > rel * ref:
        return False, f"distance {dist_g!r} vs oracle {dd[g]!r} (reference {ref!r})"
    return True, ""


def accept_top2(W: np.ndarray, norms: np.ndarray, feats: np.ndarray, g1: int, dist1: float, g2: int,
                dist2: float, rel: float = 1e-5, N: Optional[int] = None) -> Tuple[bool, str]:
    """Check one device answer (best g1, second g2) for one document.

    The second-best unit is the best neuron other than the best one (paper,
    Section 6.2, Table 5: it feeds the topographic error).  g1 must pass
    ``accept_bmu``; g2 must differ from g1 and be the oracle's best neuron
    other than g1, or lie within its near-tie band (rel relative); dist2 is
    checked against d[g2] by the same distance rule as dist1.  With N == 1
    there is no second unit: g2 must be -1 and dist2 +inf.
    """
    n = norms.shape[0] if N is None else int(N)
    ok, why = accept_bmu(W, norms, feats, g1, dist1, rel, n)
    if not ok:
        return False, "first: " + why
    if n == 1:
        if g2 == -1 and np.isinf(dist2) and dist2 > 0:
            return True, ""
        return False, f"N == 1 needs (-1, inf), got ({g2}, {dist2!r})"
    if not (0 <= g2 < n) or g2 == g1:
        return False, f"second index {g2} invalid (first is {g1})"
    dd = doc_distances(W, norms, feats, n)
    rest = dd.copy()
    rest[g1] = np.inf
    s = int(np.argmin(rest))
    if g2 != s and not dd[g2] <= dd[s] + rel * abs(dd[s]):
        return False, f"second {g2} (d={dd[g2]!r}) outside near-tie band of {s} (d={dd[s]!r})"
    dot_g = (float(feats.size) + float(norms[g2]) - dd[g2]) / 2.0
    scale = float(feats.size) + float(norms[g2]) + 2.0 * abs(dot_g)
    ref = abs(dd[g2]) if abs(dd[g2]) >= 1e-3 * scale else scale
    if abs(float(dist2) - dd[g2]) > rel * ref:
        return False, f"second distance {dist2!r} vs oracle {dd[g2]!r} (reference {ref!r})"
    return True, ""

