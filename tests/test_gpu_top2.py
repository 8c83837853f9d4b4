"""GPU parity of the top-2 search (best and second-best unit in one pass)
through the C ABI, against the fp64 oracle.

Exact where the arithmetic is exact (hand-worked examples, dyadic codebooks
with duplicated neurons, so ties at the first and at the second place);
elsewhere the oracle's top-2 acceptance rule; and always: the best unit and
its distance are bit-identical to the plain search's, and the second unit is
bit-identical across every kernel, knob and tile order.
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from conftest import GOLDEN

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2609_05138_amd as som
else:  # collected on CPU-only machines, never run there
    som = None

DEV = "cuda:0"
REL = 1e-5

KNOBS = [dict(kernel=1, tile_docs=T) for T in (1, 4, 8, 16, 32)] + [
    dict(kernel=1, lane_neurons=8), dict(kernel=1, group_tiles=4, mask_mode=1),
    dict(kernel=2), dict(kernel=2, group_tiles=4, slice_neurons=64),
    dict(kernel=3), dict(kernel=3, tile_docs=128), dict(kernel=3, tile_docs=256),
    dict(kernel=3, mask_mode=2), dict(kernel=3, tile_docs=256, mask_mode=2), dict(kernel=3, schedule=2)]


def _csr(docs):
    indptr = np.zeros(len(docs) + 1, np.int64)
    indptr[1:] = np.cumsum([len(d) for d in docs])
    indices = np.array([f for d in docs for f in d], dtype=np.int64)
    return indptr, indices


def _i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def _dev_W(W, ldw=None):
    F, N = W.shape
    ld = ((N + 3) // 4 * 4) if ldw is None else ldw
    Wp = np.zeros((F, ld), np.float32)
    Wp[:, :N] = W
    return torch.from_numpy(Wp).to(DEV)


def _top2(W, indptr, indices, perm=None, ldw=None, **knobs):
    Wd = _dev_W(W, ldw)
    N = W.shape[1]
    norms = som.som_codebook_norms(Wd, N=N)
    p = None if perm is None else _i32(perm)
    out = som.som_bmu_search_top2(Wd, norms, _i32(indptr), _i32(indices), N=N, perm=p, **knobs)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in out]


def _random_docs(rng, B, F, mean):
    return [sorted(rng.choice(F, min(F, int(rng.poisson(mean))), replace=False).tolist()) for _ in range(B)]


def test_top2_hand_examples_bit_exact():
    for ex in json.load(open(os.path.join(GOLDEN, "hand_examples.json")))["examples"]:
        F, N = ex["F"], ex["N"]
        W = np.zeros((F, N), np.float32)
        for j, w in enumerate(ex["neurons"]):
            for f, v in enumerate(w):
                W[f, j] = float(Fraction(v))
        docs = [d["features"] for d in ex["docs"]]
        indptr, indices = _csr(docs)
        # the golden distances give the second place directly: smallest (d, j) with j != bmu
        want2 = []
        for d in ex["docs"]:
            rest = sorted((Fraction(v), j) for j, v in enumerate(d["d"]) if j != d["bmu"])
            want2.append((rest[0][1], float(rest[0][0])))
        for knobs in KNOBS:
            bmu, dist, bmu2, dist2 = _top2(W, indptr, indices, **knobs)
            assert bmu.tolist() == [d["bmu"] for d in ex["docs"]], knobs
            assert dist.tolist() == [float(Fraction(d["d"][d["bmu"]])) for d in ex["docs"]], knobs
            assert list(zip(bmu2.tolist(), dist2.tolist())) == want2, knobs


@pytest.mark.parametrize("N", [2, 3, 63, 256, 257, 1023, 2065])
def test_top2_dyadic_ties_bit_exact(N):
    """W in {0, 1/4, 1/2, 3/4} (every fp32 sum exact) with duplicated neurons,
    so the first and second places tie exactly: both must follow the
    lowest-index rule."""
    rng = np.random.default_rng(100 + N)
    F, B = 48, 257
    K = rng.integers(0, 4, (F, N))
    if N > 8:
        K[:, N - 1] = K[:, 3]
        K[:, N // 2] = K[:, 3]
        K[:, 7] = K[:, 1]
    W = K.astype(np.float32) / 4
    docs = _random_docs(rng, B, F, mean=10)
    indptr, indices = _csr(docs)
    W64 = W.astype(np.float64)
    ob, od, o2, od2 = oracle.bmu_search(W64, indptr, indices)
    exact = oracle.bmu_search_exact(K, 2, indptr, indices)
    for i, e in enumerate(exact):             # the fp64 oracle is exact here
        assert ob[i] == e[0] and Fraction(od[i]) == Fraction(e[1], 16)
        if len(e[2]) > 1:
            assert o2[i] == e[2][1] and od2[i] == od[i]
    perm = rng.permutation(B)
    for knobs in KNOBS:
        for p in (None, perm):
            bmu, dist, bmu2, dist2 = _top2(W, indptr, indices, perm=p, **knobs)
            assert np.array_equal(bmu, ob) and np.array_equal(dist.astype(np.float64), od), knobs
            assert np.array_equal(bmu2, o2) and np.array_equal(dist2.astype(np.float64), od2), knobs


def test_top2_single_neuron_has_no_second():
    rng = np.random.default_rng(3)
    W = rng.random((30, 1)).astype(np.float32)
    indptr, indices = _csr(_random_docs(rng, 70, 30, mean=5) + [[]])
    for knobs in (dict(kernel=1), dict(kernel=2), dict(kernel=3)):
        bmu, dist, bmu2, dist2 = _top2(W, indptr, indices, **knobs)
        assert np.all(bmu == 0) and np.all(bmu2 == -1) and np.all(np.isinf(dist2)) and np.all(dist2 > 0)


def test_top2_agrees_with_plain_search_and_across_knobs():
    from synth import codebook, documents
    W = codebook(2, N=4100, F=20000)
    indptr, indices = documents(2, 0, n_docs=3000)
    rng = np.random.default_rng(9)
    perms = [None, rng.permutation(3000), oracle.cluster_order(indptr, indices, 20000)]
    Wd = _dev_W(W, som.som_codebook_ldw(4100))
    norms = som.som_codebook_norms(Wd, N=4100)
    ip, ix = _i32(indptr), _i32(indices)
    # ascending sweeps: every kernel, knob and tile order gives the same bits
    b0, d0 = [t.cpu().numpy() for t in som.som_bmu_search(Wd, norms, ip, ix, N=4100, sweep=1)]
    ref = None
    for i, knobs in enumerate(KNOBS):
        for p in perms if i % 3 == 0 else perms[:2]:
            pd = None if p is None else _i32(p)
            out = [t.cpu().numpy() for t in som.som_bmu_search_top2(Wd, norms, ip, ix, N=4100, perm=pd,
                                                                    **{**knobs, "sweep": 1})]
            assert np.array_equal(out[0], b0) and np.array_equal(out[1], d0), knobs
            if ref is None:
                ref = out
            assert np.array_equal(out[2], ref[2]) and np.array_equal(out[3], ref[3]), knobs
    # the rotated sweeps (the automatic order of kernels 3 and 1): the first place equals
    # the plain search's with the same plan, the pair is accepted by the oracle
    rot = {}
    for knobs in (dict(), dict(kernel=3, tile_docs=128), dict(kernel=3, tile_docs=256), dict(kernel=1),
                  dict(kernel=1, tile_docs=4, group_tiles=4)):
        for p in perms:
            pd = None if p is None else _i32(p)
            out = [t.cpu().numpy() for t in som.som_bmu_search_top2(Wd, norms, ip, ix, N=4100, perm=pd, **knobs)]
            pb, pdist = [t.cpu().numpy() for t in som.som_bmu_search(Wd, norms, ip, ix, N=4100, perm=pd, **knobs)]
            assert np.array_equal(out[0], pb) and np.array_equal(out[1], pdist), knobs
            rot[len(rot)] = out
    # against the oracle's second place, on a sample
    W64 = W.astype(np.float64)
    norms64 = oracle.codebook_norms(W64)
    bad = []
    for d in np.unique(np.concatenate([[0, 2999], rng.choice(3000, 400, replace=False)])):
        feats = indices[indptr[d]:indptr[d + 1]].astype(np.int64)
        for o in [ref] + list(rot.values()):
            ok, why = oracle.accept_top2(W64, norms64, feats, int(o[0][d]), float(o[1][d]), int(o[2][d]),
                                         float(o[3][d]), REL)
            if not ok:
                bad.append((int(d), why))
    assert not bad, bad[:5]


def test_top2_config1_every_document():
    from synth import codebook, documents
    W = codebook(1)
    indptr, indices = documents(1, 0)
    W64 = W.astype(np.float64)
    norms64 = oracle.codebook_norms(W64)
    for knobs in (dict(), dict(kernel=2), dict(kernel=3)):
        bmu, dist, bmu2, dist2 = _top2(W, indptr, indices, **knobs)
        bad = []
        for d in range(len(indptr) - 1):
            feats = indices[indptr[d]:indptr[d + 1]].astype(np.int64)
            ok, why = oracle.accept_top2(W64, norms64, feats, int(bmu[d]), float(dist[d]), int(bmu2[d]),
                                         float(dist2[d]), REL)
            if not ok:
                bad.append((d, why))
        assert not bad, bad[:5]


def test_top2_planned_reuses_a_plan():
    from synth import codebook, documents
    W = codebook(2, N=3000, F=20000)
    indptr, indices = documents(2, 1, n_docs=2000)
    Wd = _dev_W(W)
    norms = som.som_codebook_norms(Wd, N=3000)
    ip, ix = _i32(indptr), _i32(indices)
    direct = [t.cpu().numpy() for t in som.som_bmu_search_top2(Wd, norms, ip, ix, N=3000)]
    plan = som.som_plan(ip, ix, 20000)
    for _ in range(2):
        out = [t.cpu().numpy() for t in som.som_bmu_search_top2_planned(Wd, norms, ip, plan, N=3000)]
        for a, b in zip(out, direct):
            assert np.array_equal(a, b)
    plain = [t.cpu().numpy() for t in som.som_bmu_search_planned(Wd, norms, ip, plan, N=3000)]
    assert np.array_equal(plain[0], direct[0]) and np.array_equal(plain[1], direct[1])
