"""GPU parity of the fp16-codebook search (two bytes per weight, fp32 sums)
through the C ABI, against the fp64 oracle run on the same rounded weights.

The oracle consumes the fp16 values themselves (widened exactly to fp64), so
its pins carry over unchanged.  Exact cases: norms of dyadic weights, the
hand-worked examples and dyadic codebooks with ties (all representable in
fp16).  Beyond those: the fp16 search equals the fp32 search of the widened
codebook bit for bit (same values, same ascending-feature sums), and the
generated workloads pass the acceptance rules.
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
KNOBS16 = [dict(), dict(tile_docs=1), dict(tile_docs=4), dict(tile_docs=16), dict(group_tiles=4),
           dict(mask_mode=1), dict(kernel=1, lane_neurons=8, group_tiles=2),
           dict(kernel=3), dict(kernel=3, tile_docs=128), dict(kernel=3, mask_mode=2),
           dict(kernel=3, tile_docs=128, mask_mode=2)]


def _csr(docs):
    indptr = np.zeros(len(docs) + 1, np.int64)
    indptr[1:] = np.cumsum([len(d) for d in docs])
    indices = np.array([f for d in docs for f in d], dtype=np.int64)
    return indptr, indices


def _i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def _dev(W, dtype, ldw=None):
    F, N = W.shape
    ld = ((N + 7) // 8 * 8) if ldw is None else ldw
    Wp = np.zeros((F, ld), dtype)
    Wp[:, :N] = W
    return torch.from_numpy(Wp).to(DEV)


def _run(W16, indptr, indices, top2=False, dtype=np.float16, perm=None, ldw=None, **knobs):
    """Search the fp16 codebook W16 (or its exact fp32 widening with dtype=np.float32)."""
    Wd = _dev(W16, dtype, ldw)
    N = W16.shape[1]
    norms = som.som_codebook_norms(Wd, N=N)
    p = None if perm is None else _i32(perm)
    fn = som.som_bmu_search_top2 if top2 else som.som_bmu_search
    out = fn(Wd, norms, _i32(indptr), _i32(indices), N=N, perm=p, **knobs)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in out] + [norms.cpu().numpy()]


def _docs(rng, B, F, mean):
    return [sorted(rng.choice(F, min(F, int(rng.poisson(mean))), replace=False).tolist()) for _ in range(B)]


@pytest.mark.parametrize("F,N,pad", [(1, 8, 0), (37, 1000, 24), (300, 4101, 0), (2000, 513, 8)])
def test_f16_norms_match_oracle(F, N, pad):
    rng = np.random.default_rng(F + N)
    W16 = rng.random((F, N)).astype(np.float16)
    ldw = (N + 7) // 8 * 8 + pad
    Wd = _dev(W16, np.float16, ldw)
    got = som.som_codebook_norms(Wd, N=N).cpu().numpy().astype(np.float64)
    want = oracle.codebook_norms(W16.astype(np.float64))
    # the device sums exact fp64 squares in another order, then rounds to fp32 once
    assert np.all(np.abs(got - want) <= np.spacing(want.astype(np.float32)).astype(np.float64))


def test_f16_norms_dyadic_bit_exact():
    rng = np.random.default_rng(1)
    W16 = (rng.integers(0, 4, (500, 777)) / 4).astype(np.float16)
    got = som.som_codebook_norms(_dev(W16, np.float16), N=777).cpu().numpy()
    assert np.array_equal(got.astype(np.float64), oracle.codebook_norms(W16.astype(np.float64)))


def test_f16_hand_examples_bit_exact():
    for ex in json.load(open(os.path.join(GOLDEN, "hand_examples.json")))["examples"]:
        F, N = ex["F"], ex["N"]
        W = np.zeros((F, N), np.float16)
        for j, w in enumerate(ex["neurons"]):
            for f, v in enumerate(w):
                W[f, j] = float(Fraction(v))
        assert all(float(W[f, j]) == float(Fraction(v)) for j, w in enumerate(ex["neurons"])
                   for f, v in enumerate(w))
        indptr, indices = _csr([d["features"] for d in ex["docs"]])
        for knobs in KNOBS16:
            bmu, dist, norms = _run(W, indptr, indices, **knobs)
            assert norms.tolist() == [float(Fraction(v)) for v in ex["norms"]]
            assert bmu.tolist() == [d["bmu"] for d in ex["docs"]], knobs
            assert dist.tolist() == [float(Fraction(d["d"][d["bmu"]])) for d in ex["docs"]], knobs


@pytest.mark.parametrize("N", [1, 7, 511, 512, 513, 1500, 4100])
def test_f16_dyadic_codebook_bit_exact_with_ties(N):
    rng = np.random.default_rng(N + 7)
    F, B = 64, 300
    K = rng.integers(0, 4, (F, N))
    if N > 8:
        K[:, N - 1] = K[:, 2]
        K[:, N // 2] = K[:, 5]
    W16 = (K / 4).astype(np.float16)
    indptr, indices = _csr(_docs(rng, B, F, mean=12) + [[]])
    exact = oracle.bmu_search_exact(K, 2, indptr, indices)
    ob, od, o2, od2 = oracle.bmu_search(W16.astype(np.float64), indptr, indices)
    for knobs in KNOBS16:
        bmu, dist, bmu2, dist2, _ = _run(W16, indptr, indices, top2=True, **knobs)
        assert bmu.tolist() == [e[0] for e in exact], knobs
        assert [Fraction(float(x)) for x in dist] == [Fraction(e[1], 16) for e in exact], knobs
        assert np.array_equal(bmu2, o2) and np.array_equal(dist2.astype(np.float64), od2), knobs


def test_f16_equals_fp32_search_of_the_widened_codebook():
    from synth import codebook, documents
    W16 = codebook(2, N=4100, F=20000).astype(np.float16)
    indptr, indices = documents(2, 0, n_docs=3000)
    rng = np.random.default_rng(4)
    perm = rng.permutation(3000)
    # ascending sweeps: every fp16 kernel and knob gives the fp32 search's bits
    ref = _run(W16, indptr, indices, top2=True, dtype=np.float32, ldw=som.som_codebook_ldw(4100), sweep=1)
    for knobs in KNOBS16:
        for p in (None, perm):
            out = _run(W16, indptr, indices, top2=True, perm=p, ldw=som.som_codebook_ldw(4100),
                       **{**knobs, "sweep": 1})
            for a, b in zip(out, ref):
                assert np.array_equal(a, b), knobs
    # the rotated sweeps take the same order for both storage types
    for knobs in (dict(kernel=3), dict(kernel=3, tile_docs=128), dict(kernel=1, tile_docs=8, lane_neurons=8),
                  dict(kernel=1, tile_docs=4, lane_neurons=8, group_tiles=2)):
        for p in (None, perm):
            r32 = _run(W16, indptr, indices, top2=True, perm=p, dtype=np.float32, ldw=som.som_codebook_ldw(4100),
                       **knobs)
            r16 = _run(W16, indptr, indices, top2=True, perm=p, ldw=som.som_codebook_ldw(4100), **knobs)
            for a, b in zip(r16, r32):
                assert np.array_equal(a, b), knobs


def test_f16_config1_every_document():
    from synth import codebook, documents
    W16 = codebook(1).astype(np.float16)
    indptr, indices = documents(1, 0)
    W64 = W16.astype(np.float64)
    norms64 = oracle.codebook_norms(W64)
    bmu, dist, bmu2, dist2, _ = _run(W16, indptr, indices, top2=True)
    bad = []
    for d in range(len(indptr) - 1):
        feats = indices[indptr[d]:indptr[d + 1]].astype(np.int64)
        ok, why = oracle.accept_top2(W64, norms64, feats, int(bmu[d]), float(dist[d]), int(bmu2[d]),
                                     float(dist2[d]), REL)
        if not ok:
            bad.append((d, why))
    assert not bad, bad[:5]


def test_f16_config2_first_batch():
    from synth import codebook, documents
    W16 = codebook(2).astype(np.float16)
    indptr, indices = documents(2, 0)
    B = len(indptr) - 1
    bmu, dist, _ = _run(W16, indptr, indices, ldw=som.som_codebook_ldw(W16.shape[1]))
    W64 = W16.astype(np.float64)
    norms64 = oracle.codebook_norms(W64)
    rng = np.random.default_rng(2)
    bad = []
    for d in np.unique(np.concatenate([[0, B - 1], rng.choice(B, 1000, replace=False)])):
        feats = indices[indptr[d]:indptr[d + 1]].astype(np.int64)
        ok, why = oracle.accept_bmu(W64, norms64, feats, int(bmu[d]), float(dist[d]), REL)
        if not ok:
            bad.append((int(d), why))
    assert not bad, bad[:5]


def test_f16_planned_search_shares_the_fp32_plan():
    from synth import codebook, documents
    W16 = codebook(2, N=2048, F=20000).astype(np.float16)
    indptr, indices = documents(2, 3, n_docs=1500)
    ip, ix = _i32(indptr), _i32(indices)
    W32d = _dev(W16, np.float32)
    W16d = _dev(W16, np.float16)
    n32 = som.som_codebook_norms(W32d, N=2048)
    n16 = som.som_codebook_norms(W16d, N=2048)
    assert torch.equal(n32, n16)
    ref = None
    for knobs in (dict(), dict(kernel=3), dict(kernel=3, tile_docs=128), dict(sweep=1),
                  dict(kernel=3, tile_docs=128, sweep=1)):
        # kernel 3: the same super-tile plan for both storage types (and with
        # the ascending sweep the same bits for every super-tile size)
        plan = som.som_plan(ip, ix, 20000, **knobs)
        a = [t.cpu().numpy() for t in som.som_bmu_search_top2_planned(W32d, n32, ip, plan, N=2048)]
        b = [t.cpu().numpy() for t in som.som_bmu_search_top2_planned(W16d, n16, ip, plan, N=2048)]
        c = [t.cpu().numpy() for t in som.som_bmu_search_planned(W16d, n16, ip, plan, N=2048)]
        for x, y in zip(a, b):
            assert np.array_equal(x, y), knobs
        assert np.array_equal(c[0], a[0]) and np.array_equal(c[1], a[1]), knobs
        if knobs.get("sweep") == 1:
            ref = a if ref is None else ref
            for x, y in zip(a, ref):
                assert np.array_equal(x, y), knobs
