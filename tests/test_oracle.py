"""Pins of the fp64 oracle against what the mathematics fixes (CPU only).

Each pin ties the oracle to something other than itself: hand-worked exact
values, a dense brute force in rational arithmetic, an exact integer
evaluation, special cases with closed-form answers, and invariances of the
exact argmin (document order, feature relabelling, codebook layout, tile size
and tile membership).
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from conftest import GOLDEN


def _csr(docs):
    indptr = np.zeros(len(docs) + 1, np.int64)
    indptr[1:] = np.cumsum([len(d) for d in docs])
    indices = np.array([f for d in docs for f in d], dtype=np.int64)
    return indptr, indices


def _load(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


def _example_W(ex, ldw=None):
    F, N = ex["F"], ex["N"]
    ld = N if ldw is None else ldw
    W = np.zeros((F, ld), np.float64)
    for j, w in enumerate(ex["neurons"]):
        for f, v in enumerate(w):
            W[f, j] = float(Fraction(v))
    return W


def _random_dyadic(rng, F, N, bits=8):
    return rng.integers(0, 1 << bits, (F, N)).astype(np.float64) / float(1 << bits)


def _random_docs(rng, B, F, mean=4.0, empty_every=0):
    docs = []
    for i in range(B):
        k = min(F, int(rng.poisson(mean)))
        if empty_every and i % empty_every == 0:
            k = 0
        docs.append(sorted(rng.choice(F, k, replace=False).tolist()))
    return docs


# ----------------------------------------------------------------------------
# hand-worked examples
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("ldw_pad", [0, 1])
def test_hand_examples(ldw_pad):
    for ex in _load("hand_examples.json")["examples"]:
        N = ex["N"]
        W = _example_W(ex, ldw=N + ldw_pad)
        norms = oracle.codebook_norms(W, N)
        assert norms.tolist() == [float(Fraction(v)) for v in ex["norms"]]
        indptr, indices = _csr([d["features"] for d in ex["docs"]])
        bmu, dist, j2, d2 = oracle.bmu_search(W, indptr, indices, N=N)
        for i, d in enumerate(ex["docs"]):
            want = [float(Fraction(v)) for v in d["d"]]
            got = oracle.doc_distances(W, norms, np.array(d["features"], np.int64), N)
            assert got.tolist() == want, (ex["name"], i)
            assert bmu[i] == d["bmu"], (ex["name"], i)
            assert dist[i] == want[d["bmu"]]
            rest = sorted((v, j) for j, v in enumerate(want) if j != d["bmu"])
            assert (j2[i], d2[i]) == (rest[0][1], rest[0][0])


def test_hand_examples_match_dense_brute_force():
    for ex in _load("hand_examples.json")["examples"]:
        W = _example_W(ex)
        indptr, indices = _csr([d["features"] for d in ex["docs"]])
        b, dq = oracle.bmu_search_dense(W, indptr, indices)
        assert b == [d["bmu"] for d in ex["docs"]]
        assert dq == [Fraction(d["d"][d["bmu"]]) for d in ex["docs"]]


# ----------------------------------------------------------------------------
# brute force and exact integer evaluation
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_random_tiny_vs_dense_brute_force(seed):
    rng = np.random.default_rng(seed)
    F, N, B = int(rng.integers(1, 11)), int(rng.integers(1, 9)), 25
    W = _random_dyadic(rng, F, N, bits=3)   # coarse grid -> many exact ties
    docs = _random_docs(rng, B, F, mean=F / 3, empty_every=7)
    indptr, indices = _csr(docs)
    b_dense, d_dense = oracle.bmu_search_dense(W, indptr, indices)
    bmu, dist, _, _ = oracle.bmu_search(W, indptr, indices)
    assert bmu.tolist() == b_dense
    assert [Fraction(float(x)) for x in dist] == d_dense


@pytest.mark.parametrize("seed", range(4))
def test_fp64_equals_exact_integer(seed):
    rng = np.random.default_rng(100 + seed)
    F, N, B, bits = 40, 50, 120, 16
    K = rng.integers(0, 1 << bits, (F, N))
    K[:, 7] = K[:, 3]                    # duplicated neuron: an exact tie
    W = K.astype(np.float64) / float(1 << bits)
    docs = _random_docs(rng, B, F, mean=8.0, empty_every=11)
    indptr, indices = _csr(docs)
    exact = oracle.bmu_search_exact(K, bits, indptr, indices)
    bmu, dist, _, _ = oracle.bmu_search(W, indptr, indices)
    for i, (b, scaled, ties) in enumerate(exact):
        assert bmu[i] == ties[0] == b
        assert Fraction(float(dist[i])) == Fraction(scaled, 1 << (2 * bits))


def test_exact_integer_on_generated_24bit_codebook():
    """Generated weights are k * 2**-24; the integer form is exact for them."""
    from synth import codebook_rows, documents
    F, N = 48, 40
    W32 = codebook_rows(1, range(F), N=N)
    K = np.rint(W32.astype(np.float64) * (1 << 24)).astype(np.int64)
    assert np.array_equal(K.astype(np.float64) / (1 << 24), W32.astype(np.float64))
    indptr, indices = documents(1, 0, n_docs=60)
    keep = [[f for f in indices[indptr[d]:indptr[d + 1]] if f < F] for d in range(60)]
    ip, ix = _csr(keep)
    exact = oracle.bmu_search_exact(K, 24, ip, ix)
    bmu, dist, j2, d2 = oracle.bmu_search(W32, ip, ix)
    for i, (b, scaled, ties) in enumerate(exact):
        # fp64 rounds only the ~55-bit norm sums; the argmin is exact unless
        # the true gap is below that rounding, which the int form reports
        gap = (d2[i] - dist[i])
        if gap > 1e-9:
            assert bmu[i] == b
        assert abs(dist[i] - scaled / float(1 << 48)) <= 1e-12 * max(1.0, abs(dist[i]))


# ----------------------------------------------------------------------------
# special cases with closed-form answers
# ----------------------------------------------------------------------------

def test_single_neuron_is_always_bmu():
    rng = np.random.default_rng(3)
    W = _random_dyadic(rng, 9, 1)
    indptr, indices = _csr(_random_docs(rng, 30, 9, empty_every=5))
    bmu, dist, j2, d2 = oracle.bmu_search(W, indptr, indices)
    assert np.all(bmu == 0) and np.all(j2 == -1) and np.all(np.isinf(d2))


def test_empty_document_is_argmin_of_norms():
    rng = np.random.default_rng(4)
    W = _random_dyadic(rng, 12, 33, bits=2)
    norms = oracle.codebook_norms(W)
    indptr, indices = _csr([[], []])
    bmu, dist, _, _ = oracle.bmu_search(W, indptr, indices)
    first = min(range(33), key=lambda j: (norms[j], j))
    assert bmu.tolist() == [first, first]
    assert dist[0] == norms[first]


def test_neuron_equal_to_document_has_zero_distance():
    rng = np.random.default_rng(5)
    F, N = 10, 8
    W = _random_dyadic(rng, F, N) * 0.5 + 0.25
    doc = [1, 4, 7]
    W[:, 5] = 0.0
    W[doc, 5] = 1.0
    indptr, indices = _csr([doc])
    bmu, dist, _, _ = oracle.bmu_search(W, indptr, indices)
    assert bmu[0] == 5 and dist[0] == 0.0
    W[:, 2] = W[:, 5]                       # a lower index ties it
    bmu, dist, _, _ = oracle.bmu_search(W, indptr, indices)
    assert bmu[0] == 2 and dist[0] == 0.0


# ----------------------------------------------------------------------------
# invariances of the exact argmin
# ----------------------------------------------------------------------------

def test_invariant_to_codebook_layout():
    """Neuron-major rows, evaluated in the dense form, give the same answers."""
    rng = np.random.default_rng(6)
    F, N = 14, 21
    W = _random_dyadic(rng, F, N, bits=4)
    Wnm = np.ascontiguousarray(W.T)            # [N][F], neuron-major
    docs = _random_docs(rng, 40, F, mean=5, empty_every=9)
    indptr, indices = _csr(docs)
    bmu, dist, _, _ = oracle.bmu_search(W, indptr, indices)
    for i, d in enumerate(docs):
        x = np.zeros(F)
        x[d] = 1.0
        dd = ((x[None, :] - Wnm) ** 2).sum(axis=1)
        assert bmu[i] == int(np.argmin(dd)) and dist[i] == dd.min()


def test_invariant_to_document_order():
    rng = np.random.default_rng(7)
    W = _random_dyadic(rng, 16, 24, bits=3)
    docs = _random_docs(rng, 50, 16, mean=5)
    p = rng.permutation(50)
    a = oracle.bmu_search(W, *_csr(docs))
    b = oracle.bmu_search(W, *_csr([docs[i] for i in p]))
    for x, y in zip(a, b):
        assert np.array_equal(x[p], y)


def test_invariant_to_feature_relabel():
    rng = np.random.default_rng(8)
    F = 18
    W = _random_dyadic(rng, F, 20, bits=3)
    docs = _random_docs(rng, 40, F, mean=6)
    r = rng.permutation(F)                     # new id of old feature f is r[f]
    W2 = np.empty_like(W)
    W2[r] = W
    docs2 = [sorted(int(r[f]) for f in d) for d in docs]
    a = oracle.bmu_search(W, *_csr(docs))
    b = oracle.bmu_search(W2, *_csr(docs2))
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("T", [1, 2, 3, 4, 8, 16, 64])
def test_tiled_sweep_equals_direct(T):
    rng = np.random.default_rng(9 + T)
    F, N, B = 30, 17, 70
    W = _random_dyadic(rng, F, N, bits=6)
    docs = _random_docs(rng, B, F, mean=6, empty_every=13)
    indptr, indices = _csr(docs)
    bmu, dist, _, _ = oracle.bmu_search(W, indptr, indices)
    perms = [None, rng.permutation(B), oracle.cluster_order(indptr, indices, F)]
    for perm in perms:
        tb, td = oracle.bmu_search_tiled(W, indptr, indices, T, perm=perm)
        assert np.array_equal(tb, bmu) and np.array_equal(td, dist)


def test_tile_union_matches_set_union():
    rng = np.random.default_rng(10)
    F, B = 25, 37
    docs = _random_docs(rng, B, F, mean=5, empty_every=6)
    indptr, indices = _csr(docs)
    for T in (1, 3, 8, 32):
        for perm in (None, rng.permutation(B)):
            order = list(range(B)) if perm is None else list(perm)
            tiles = oracle.tile_union(indptr, indices, T, perm)
            assert len(tiles) == (B + T - 1) // T
            for t, (feats, masks) in enumerate(tiles):
                members = order[t * T:(t + 1) * T]
                want = sorted(set().union(*[set(docs[d]) for d in members]))
                assert feats.tolist() == want
                for f, m in zip(feats, masks):
                    bits = [s for s in range(len(members)) if (int(m) >> s) & 1]
                    assert bits == [s for s, d in enumerate(members) if f in docs[d]]


# ----------------------------------------------------------------------------
# clustering reading
# ----------------------------------------------------------------------------

def test_cluster_order_hand_examples():
    for ex in _load("cluster_examples.json")["examples"]:
        indptr, indices = _csr(ex["docs"])
        perm = oracle.cluster_order(indptr, indices, ex["F"])
        assert perm.tolist() == ex["perm"]


def test_cluster_order_is_a_sorted_permutation():
    rng = np.random.default_rng(11)
    F, B = 40, 300
    docs = _random_docs(rng, B, F, mean=6, empty_every=17)
    indptr, indices = _csr(docs)
    perm = oracle.cluster_order(indptr, indices, F)
    assert sorted(perm.tolist()) == list(range(B))
    df = np.zeros(F, int)
    for d in docs:
        df[d] += 1

    def sig(d):
        r = sorted(docs[d], key=lambda f: (-df[f], f)) + [F, F]
        return (r[0], r[1], d)

    keys = [sig(int(d)) for d in perm]
    assert keys == sorted(keys)


# ----------------------------------------------------------------------------
# norms and acceptance rule
# ----------------------------------------------------------------------------

def test_norms_definition_and_blocks():
    rng = np.random.default_rng(12)
    W = _random_dyadic(rng, 13, 9, bits=5)
    want = [sum(Fraction(float(W[f, j])) ** 2 for f in range(13)) for j in range(9)]
    got = oracle.codebook_norms(W)
    assert [Fraction(float(v)) for v in got] == want
    blocks = oracle.codebook_norms_blocks([W[:5], W[5:6], W[6:]])
    assert np.array_equal(blocks, got)
    assert np.array_equal(oracle.codebook_norms(np.pad(W, ((0, 0), (0, 3))), 9), got)


def test_accept_rule():
    ex = _load("hand_examples.json")["examples"][1]     # B: ties and zeros
    W = _example_W(ex)
    norms = oracle.codebook_norms(W)
    f01 = np.array([0, 1])
    assert oracle.accept_bmu(W, norms, f01, 0, 1.0)[0]
    assert oracle.accept_bmu(W, norms, f01, 2, 1.0)[0]          # exact tie
    assert not oracle.accept_bmu(W, norms, f01, 1, 1.5)[0]      # outside the band
    assert not oracle.accept_bmu(W, norms, f01, 0, 1.0 + 1e-3)[0]
    assert oracle.accept_bmu(W, norms, f01, 0, 1.0 + 5e-6)[0]
    assert oracle.accept_bmu(W, norms, np.array([0]), 0, 1e-6)[0]   # cancelled: scale rule
    assert not oracle.accept_bmu(W, norms, np.array([0]), 0, 1e-3)[0]
    assert not oracle.accept_bmu(W, norms, f01, 3, 1.0)[0]


def test_accept_top2_rule():
    ex = _load("hand_examples.json")["examples"][1]     # B: ties and zeros
    W = _example_W(ex)
    norms = oracle.codebook_norms(W)
    f01, f0 = np.array([0, 1]), np.array([0])
    acc = lambda *a, **k: oracle.accept_top2(W, norms, *a, **k)[0]   # noqa: E731
    assert acc(f01, 0, 1.0, 2, 1.0)                  # d = (1, 3/2, 1): tie -> 0 then 2
    assert acc(f01, 2, 1.0, 0, 1.0)                  # the tie partner first is accepted
    assert not acc(f01, 0, 1.0, 1, 1.5)              # 1 is not the best other than 0
    assert not acc(f01, 0, 1.0, 0, 1.0)              # second must differ from first
    assert not acc(f01, 0, 1.0, 2, 1.0 + 1e-3)       # second distance off
    assert acc(f01, 0, 1.0, 2, 1.0 + 5e-6)
    assert not acc(f01, 1, 1.5, 0, 1.0)              # first rejected
    assert not acc(f01, 0, 1.0, 3, 1.0)              # out of range
    assert acc(f0, 0, 0.0, 1, 1.5)                   # d = (0, 3/2, 2)
    assert not acc(f0, 0, 0.0, 2, 2.0)
    W1 = W[:, :1].copy()
    n1 = oracle.codebook_norms(W1)
    assert oracle.accept_top2(W1, n1, f0, 0, 0.0, -1, np.inf)[0]     # N == 1: no second unit
    assert not oracle.accept_top2(W1, n1, f0, 0, 0.0, 0, 0.0)[0]
    assert not oracle.accept_top2(W1, n1, f0, 0, 0.0, -1, 5.0)[0]
    # near-tie band of the second place: d = (0.25, 1, 1 + eps) for one feature
    for eps, ok in ((1e-6, True), (1e-4, False)):
        Wn = np.array([[0.5, 0.0, 1.0 - np.sqrt(1.0 + eps)]])
        nn = oracle.codebook_norms(Wn)
        d = oracle.doc_distances(Wn, nn, f0)
        assert abs(d[2] - (1.0 + eps)) < 1e-12
        assert oracle.accept_top2(Wn, nn, f0, 0, 0.25, 1, 1.0)[0]
        assert oracle.accept_top2(Wn, nn, f0, 0, 0.25, 2, float(d[2]))[0] == ok


def test_rejects_unsorted_documents():
    W = np.ones((4, 2))
    with pytest.raises(ValueError):
        oracle.bmu_search(W, np.array([0, 2]), np.array([2, 1]))
    with pytest.raises(ValueError):
        oracle.bmu_search(W, np.array([0, 2]), np.array([1, 1]))
