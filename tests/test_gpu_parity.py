"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle.

Bit-exact where the arithmetic is exact (integer plan and clustering work,
dyadic codebooks whose every fp32 sum is exact, the hand-worked examples);
elsewhere the acceptance rule of the search: the device index equals the
oracle's BMU unless it lies in the oracle's 1e-5 relative near-tie band, and
the device distance is within 1e-5 relative of the oracle's distance for
that index.
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


def _csr(docs):
    indptr = np.zeros(len(docs) + 1, np.int64)
    indptr[1:] = np.cumsum([len(d) for d in docs])
    indices = np.array([f for d in docs for f in d], dtype=np.int64)
    return indptr, indices


def _dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def _dev_W(W, ldw=None):
    F, N = W.shape
    ld = ((N + 3) // 4 * 4) if ldw is None else ldw
    Wp = np.zeros((F, ld), np.float32)
    Wp[:, :N] = W
    return torch.from_numpy(Wp).to(DEV), ld


def _search(W, indptr, indices, N=None, ldw=None, perm=None, **kw):
    Wd, ld = _dev_W(W, ldw)
    n = W.shape[1] if N is None else N
    norms = som.som_codebook_norms(Wd, N=n)
    p = None if perm is None else _dev_i32(perm)
    bmu, dist = som.som_bmu_search(Wd, norms, _dev_i32(indptr), _dev_i32(indices), N=n, perm=p, **kw)
    torch.cuda.synchronize()
    return bmu.cpu().numpy().astype(np.int64), dist.cpu().numpy().astype(np.float64), norms.cpu().numpy()


def _random_docs(rng, B, F, mean, empty_every=0, big_every=0, big=0):
    docs = []
    for i in range(B):
        k = min(F, int(rng.poisson(mean)))
        if empty_every and i % empty_every == 0:
            k = 0
        if big_every and i % big_every == 1:
            k = min(F, big)
        docs.append(sorted(rng.choice(F, k, replace=False).tolist()))
    return docs


TILES = [1, 2, 4, 8, 16, 32]
SUPER = [64, 128, 256]          # kernel 3: documents per super-tile


# ----------------------------------------------------------------------------
# norms
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("F,N,pad", [(1, 1, 3), (7, 5, 0), (300, 1025, 4), (2048, 1024, 0), (129, 4099, 61)])
def test_norms_match_oracle(F, N, pad):
    rng = np.random.default_rng(F * 7 + N)
    W = rng.random((F, N), dtype=np.float32)
    ldw = (N + 3) // 4 * 4 + (pad // 4) * 4
    Wd, _ = _dev_W(W, ldw)
    got = som.som_codebook_norms(Wd, N=N).cpu().numpy()
    want = oracle.codebook_norms(W.astype(np.float64))
    # fp64 accumulation rounded once: equal to the correctly rounded value
    # except within fp64 rounding of a half-way point (at most 1 ulp)
    want32 = want.astype(np.float32)
    ulps = np.abs(got.view(np.int32).astype(np.int64) - want32.view(np.int32).astype(np.int64))
    assert ulps.max() <= 1
    assert np.count_nonzero(ulps) <= max(1, N // 1000)


def test_norms_dyadic_bit_exact():
    rng = np.random.default_rng(1)
    W = rng.integers(0, 4, (500, 777)).astype(np.float32) / 4
    Wd, _ = _dev_W(W)
    got = som.som_codebook_norms(Wd, N=777).cpu().numpy()
    assert np.array_equal(got.astype(np.float64), oracle.codebook_norms(W.astype(np.float64)))


# ----------------------------------------------------------------------------
# exact cases: hand-worked examples and dyadic codebooks
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("knobs", [dict(kernel=1, tile_docs=T) for T in TILES]
                         + [dict(kernel=2, group_tiles=G, slice_neurons=NB) for G in (4, 16) for NB in (32, 64)]
                         + [dict(kernel=3, tile_docs=D) for D in SUPER]
                         + [dict(kernel=3, tile_docs=D, mask_mode=2) for D in SUPER])
def test_hand_examples_bit_exact(knobs):
    ex_all = json.load(open(os.path.join(GOLDEN, "hand_examples.json")))["examples"]
    for ex in ex_all:
        F, N = ex["F"], ex["N"]
        W = np.zeros((F, N), np.float32)
        for j, w in enumerate(ex["neurons"]):
            for f, v in enumerate(w):
                W[f, j] = float(Fraction(v))
        docs = [d["features"] for d in ex["docs"]]
        indptr, indices = _csr(docs)
        bmu, dist, norms = _search(W, indptr, indices, **knobs)
        assert norms.tolist() == [float(Fraction(v)) for v in ex["norms"]]
        assert bmu.tolist() == [d["bmu"] for d in ex["docs"]]
        assert dist.tolist() == [float(Fraction(d["d"][d["bmu"]])) for d in ex["docs"]]


@pytest.mark.parametrize("N", [1, 3, 5, 63, 511, 513, 1023, 1025, 2065, 5000])
def test_dyadic_codebook_bit_exact_with_ties(N):
    """W in {0, 1/4, 1/2, 3/4}: every fp32 sum is exact, so indices (lowest on
    ties) and distances must equal the exact integer evaluation."""
    rng = np.random.default_rng(N)
    F, B = 64, 301
    K = rng.integers(0, 4, (F, N))
    if N > 8:
        K[:, N - 1] = K[:, 2]          # exact duplicate neurons -> ties
        K[:, N // 2] = K[:, 5]
    W = K.astype(np.float32) / 4
    docs = _random_docs(rng, B, F, mean=12, empty_every=17, big_every=50, big=60)
    indptr, indices = _csr(docs)
    exact = oracle.bmu_search_exact(K, 2, indptr, indices)
    for knobs in (dict(kernel=1, tile_docs=1), dict(kernel=1, tile_docs=8), dict(kernel=1, tile_docs=32),
                  dict(kernel=2), dict(kernel=2, group_tiles=4, slice_neurons=64),
                  dict(kernel=3), dict(kernel=3, tile_docs=128), dict(kernel=3, tile_docs=256),
                  dict(kernel=3, mask_mode=2), dict(kernel=3, tile_docs=256, mask_mode=2),
                  dict(kernel=3, schedule=2), dict(kernel=3, tile_docs=128, mask_mode=1, schedule=2),
                  dict(kernel=3, sweep=1), dict(kernel=3, tile_docs=128, sweep=2)):
        bmu, dist, _ = _search(W, indptr, indices, **knobs)
        assert bmu.tolist() == [e[2][0] for e in exact]
        assert [Fraction(float(x)) for x in dist] == [Fraction(e[1], 16) for e in exact]


# ----------------------------------------------------------------------------
# tile plan and clustering: integer work, bit-exact
# ----------------------------------------------------------------------------

def _mask_ints(um, T):
    """Plan masks as Python ints (one uint32 word per entry up to 32
    documents per tile, T / 32 words per entry beyond)."""
    w = um.view(np.uint32).reshape(len(um), -1) if T > 32 else um.view(np.uint32).reshape(-1, 1)
    return [sum(int(x) << (32 * k) for k, x in enumerate(row)) for row in w]


@pytest.mark.parametrize("T", TILES + SUPER)
def test_tile_plan_bit_exact(T):
    from synth import documents
    indptr, indices = documents(1, 0, n_docs=1001)      # ragged last tile
    rng = np.random.default_rng(T)
    for perm in (None, rng.permutation(1001)):
        pl = som.som_tile_plan(_dev_i32(indptr), _dev_i32(indices), 2048, T,
                               perm=None if perm is None else _dev_i32(perm))
        off, cnt, uf, um = (x.cpu().numpy() for x in pl)
        tiles = oracle.tile_union(indptr, indices, T, perm)
        assert len(cnt) == len(tiles)
        order = np.arange(1001) if perm is None else perm
        nnz_doc = np.diff(indptr)[order]
        assert off.tolist() == [0] + np.cumsum([nnz_doc[t * T:(t + 1) * T].sum() for t in range(len(tiles))]).tolist()
        for t, (feats, masks) in enumerate(tiles):
            assert cnt[t] == len(feats)
            assert uf[off[t]:off[t] + cnt[t]].tolist() == feats.tolist()
            assert _mask_ints(um[off[t]:off[t] + cnt[t]], T) == [int(m) for m in masks]


@pytest.mark.parametrize("T", [4, 256])
def test_tile_plan_large_feature_ids_use_several_windows(T):
    rng = np.random.default_rng(3)
    F = 70_000                                         # > one 32768-feature window (4096 at T = 256)
    docs = _random_docs(rng, 530, F, mean=30, empty_every=9)
    indptr, indices = _csr(docs)
    pl = som.som_tile_plan(_dev_i32(indptr), _dev_i32(indices), F, T)
    off, cnt, uf, um = (x.cpu().numpy() for x in pl)
    for t, (feats, masks) in enumerate(oracle.tile_union(indptr, indices, T)):
        assert uf[off[t]:off[t] + cnt[t]].tolist() == feats.tolist()
        assert _mask_ints(um[off[t]:off[t] + cnt[t]], T) == [int(m) for m in masks]


@pytest.mark.parametrize("D", [1, 7, 256, 1024])
def test_group_plan_bit_exact(D):
    """Group union = tile union with a tile of D documents; entry_pos = the
    position of each nonzero's feature in its group's union."""
    from synth import documents
    indptr, indices = documents(1, 0, n_docs=2500)
    B = 2500
    rng = np.random.default_rng(D)
    for perm in (None, rng.permutation(B)):
        off, cnt, gf, pos = (x.cpu().numpy() for x in som.som_group_plan(
            _dev_i32(indptr), _dev_i32(indices), 2048, D, perm=None if perm is None else _dev_i32(perm)))
        order = np.arange(B) if perm is None else perm
        groups = oracle.tile_union(indptr, indices, D, perm)
        assert len(cnt) == len(groups)
        for g, (feats, _) in enumerate(groups):
            assert cnt[g] == len(feats)
            assert gf[off[g]:off[g] + cnt[g]].tolist() == feats.tolist()
            rank = {int(f): i for i, f in enumerate(feats)}
            for d in order[g * D:(g + 1) * D]:
                a, b = indptr[d], indptr[d + 1]
                assert pos[a:b].tolist() == [rank[int(f)] for f in indices[a:b]]


def test_cluster_order_golden():
    ex_all = json.load(open(os.path.join(GOLDEN, "cluster_examples.json")))["examples"]
    for ex in ex_all:
        indptr, indices = _csr(ex["docs"])
        perm = som.som_cluster_order(_dev_i32(indptr), _dev_i32(indices), ex["F"]).cpu().numpy()
        assert perm.tolist() == ex["perm"]


# sizes reach every launch form of the sort: steps inside 2,048-element
# blocks only, and one, two or three wide steps per launch (n2 = 2^18 runs
# seven merge levels above the block size)
@pytest.mark.parametrize("cfg,n", [(5, 20000), (2, 8000), (1, 10000), (2, 150000)])
def test_cluster_order_bit_exact(cfg, n):
    from synth import CONFIGS, documents
    indptr, indices = documents(cfg, 0, n_docs=n)
    F = CONFIGS[cfg].F
    got = som.som_cluster_order(_dev_i32(indptr), _dev_i32(indices), F).cpu().numpy()
    assert got.tolist() == oracle.cluster_order(indptr, indices, F).tolist()


# ----------------------------------------------------------------------------
# generated workloads under the acceptance rule
# ----------------------------------------------------------------------------

def _check_docs(W64, norms64, indptr, indices, bmu, dist, docs, N=None):
    bad = []
    for d in docs:
        feats = np.asarray(indices[indptr[d]:indptr[d + 1]], np.int64)
        ok, why = oracle.accept_bmu(W64, norms64, feats, int(bmu[d]), float(dist[d]), REL, N)
        if not ok:
            bad.append((int(d), why))
    assert not bad, bad[:5]


def test_config1_every_document():
    from synth import codebook, documents
    W = codebook(1)
    indptr, indices = documents(1, 0)
    for knobs in (dict(kernel=1, tile_docs=1), dict(kernel=1, tile_docs=8), dict(kernel=2),
                  dict(kernel=2, group_tiles=4, slice_neurons=64), dict(kernel=3), dict(kernel=3, tile_docs=256),
                  dict(kernel=3, sweep=1)):
        bmu, dist, _ = _search(W, indptr, indices, **knobs)
        W64 = W.astype(np.float64)
        _check_docs(W64, oracle.codebook_norms(W64), indptr, indices, bmu, dist, range(len(indptr) - 1))


def test_config2_first_batch():
    from synth import codebook, documents
    W = codebook(2)
    indptr, indices = documents(2, 0)                   # 65,536 documents
    B = len(indptr) - 1
    ldw = som.som_codebook_ldw(W.shape[1])
    # the benchmark's launch for this map: automatic (kernel 3, 64-document
    # super-tiles, rotated sweep) on the clustered order
    perm = oracle.cluster_order(indptr, indices, W.shape[0])
    bmu, dist, _ = _search(W, indptr, indices, ldw=ldw, perm=perm)
    # ascending sweeps: kernel 3 on the clustered order and kernel 1 on the
    # input order give the same bits on the whole batch
    b1, d1, _ = _search(W, indptr, indices, ldw=ldw, kernel=1, sweep=1)
    b3, d3, _ = _search(W, indptr, indices, ldw=ldw, perm=perm, kernel=3, sweep=1)
    assert np.array_equal(b3, b1) and np.array_equal(d3, d1)
    # the rotated sweep sums in another order: some distances differ in
    # rounding (so the rotation is in effect), all by a few ulp at most
    assert not np.array_equal(dist, d1)
    assert np.all(np.abs(dist.astype(np.float64) - d1) <= 1e-6 * np.abs(d1.astype(np.float64)))
    W64 = W.astype(np.float64)
    norms64 = oracle.codebook_norms(W64)
    rng = np.random.default_rng(0)
    sample = np.unique(np.concatenate([[0, B - 1], rng.choice(B, 1500, replace=False)]))
    _check_docs(W64, norms64, indptr, indices, bmu, dist, sample)
    # where the two sweeps pick different neurons, both must be in the oracle's near-tie band
    flips = np.nonzero(b1 != bmu)[0]
    assert len(flips) <= 20, len(flips)
    _check_docs(W64, norms64, indptr, indices, bmu, dist, flips)
    _check_docs(W64, norms64, indptr, indices, b1, d1, flips)
    # every document: the reported distance is the distance of the reported neuron
    nnz = np.diff(indptr)
    g = np.repeat(bmu, nnz)
    dot = np.add.reduceat(W64[indices, g], indptr[:-1]) if len(indices) else np.zeros(B)
    d_at_g = nnz + norms64[bmu] - 2 * dot
    assert np.all(np.abs(dist - d_at_g) <= REL * np.abs(d_at_g))


def test_results_identical_across_tile_chunk_and_order():
    """With the ascending sweep each document's dot product is summed in
    ascending feature order whatever the tiling, so the outputs are
    bit-identical."""
    from synth import codebook, documents
    W = codebook(2, N=4100, F=20000)
    indptr, indices = documents(2, 0, n_docs=3000)
    ref = None
    rng = np.random.default_rng(5)
    perms = [None, rng.permutation(3000), oracle.cluster_order(indptr, indices, 20000)]
    variants = [dict(kernel=2, group_tiles=G, slice_neurons=NB) for G in (4, 8, 16) for NB in (32, 64)]
    for T in TILES:
        for K, G, mode in ((0, 0, 0), (4, 1, 1), (8 if T < 32 else 4, 8, 2), (4, 2, 2)):
            variants.append(dict(kernel=1, tile_docs=T, lane_neurons=K, group_tiles=G, mask_mode=mode))
    variants += [dict(kernel=3, tile_docs=D, mask_mode=m, sweep=1) for D in SUPER for m in (1, 2)]
    # schedule chunks of the neuron axis (17 slices of 256 neurons here: full
    # and partial last chunks, and one chunk wider than the map)
    variants += [dict(kernel=1, neuron_chunk=nc) for nc in (512, 768, 4096, 1 << 20)]
    variants += [dict(kernel=1, tile_docs=16, group_tiles=4, neuron_chunk=768),
                 dict(kernel=1, lane_neurons=8, neuron_chunk=1024)]
    variants += [dict(kernel=3, neuron_chunk=nc) for nc in (512, 768, 4096)]
    variants += [dict(kernel=3, tile_docs=128, neuron_chunk=512), dict(kernel=3, mask_mode=1, neuron_chunk=1024),
                 dict(kernel=3, neuron_chunk=256, sweep=1), dict(kernel=3, schedule=2)]
    for i, v in enumerate(variants):
        for perm in perms if (i % 5 == 0 or v["kernel"] == 3) else perms[:2]:
            out = _search(W, indptr, indices, perm=perm, **{**v, "sweep": 1})
            if ref is None:
                ref = out
            assert np.array_equal(out[0], ref[0]) and np.array_equal(out[1], ref[1]), v
    # the row stride is a layout choice only
    for ldw in (som.som_codebook_ldw(4100), 4104, 4100 + 1024):
        for v in (dict(sweep=1), dict(kernel=1, lane_neurons=8, sweep=1), dict(kernel=2), dict(kernel=3, sweep=1)):
            out = _search(W, indptr, indices, ldw=ldw, **v)
            assert np.array_equal(out[0], ref[0]) and np.array_equal(out[1], ref[1]), (ldw, v)


def test_repeated_runs_are_bit_identical():
    from synth import codebook, documents
    W = codebook(1)
    indptr, indices = documents(1, 0)
    a = _search(W, indptr, indices)
    for _ in range(3):
        b = _search(W, indptr, indices)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_rotated_sweep_order_is_fixed_and_within_tolerance():
    """Rotated sweeps (the automatic order of kernels 3 and 1): the order depends on the
    plan and the launch's tile grid only, so the results are the same across
    repeated calls, row strides, planned and unplanned searches, top-2 and
    one-slice schedule chunks; they differ from the ascending sweep's only in
    rounding (some distances do differ: the rotation is in effect), and both
    are accepted by the oracle on every document."""
    from synth import codebook, documents
    W = codebook(2, N=4100, F=20000)
    indptr, indices = documents(2, 0, n_docs=3000)
    perm = oracle.cluster_order(indptr, indices, 20000)
    W64 = W.astype(np.float64)
    norms64 = oracle.codebook_norms(W64)
    for D in SUPER:
        ref = _search(W, indptr, indices, perm=perm, kernel=3, tile_docs=D)
        for v in (dict(sweep=2), dict(neuron_chunk=256), dict(sweep=2, neuron_chunk=256)):
            out = _search(W, indptr, indices, perm=perm, kernel=3, tile_docs=D, **v)
            assert np.array_equal(out[0], ref[0]) and np.array_equal(out[1], ref[1]), (D, v)
        for ldw in (4104, 4100 + 1024):
            out = _search(W, indptr, indices, perm=perm, ldw=ldw, kernel=3, tile_docs=D)
            assert np.array_equal(out[0], ref[0]) and np.array_equal(out[1], ref[1]), (D, ldw)
        Wd, _ = _dev_W(W)
        norms = som.som_codebook_norms(Wd, N=4100)
        ip, ix, pd = _dev_i32(indptr), _dev_i32(indices), _dev_i32(perm)
        plan = som.som_plan(ip, ix, 20000, perm=pd, kernel=3, tile_docs=D)
        pl = som.som_bmu_search_planned(Wd, norms, ip, plan, N=4100)
        t2 = som.som_bmu_search_top2(Wd, norms, ip, ix, N=4100, perm=pd, kernel=3, tile_docs=D)
        torch.cuda.synchronize()
        for b, d in (pl, t2[:2]):
            assert np.array_equal(b.cpu().numpy(), ref[0]) and np.array_equal(d.cpu().numpy(), ref[1]), D
        asc = _search(W, indptr, indices, perm=perm, kernel=3, tile_docs=D, sweep=1)
        assert not np.array_equal(asc[1], ref[1]), D
        rel = np.abs(asc[1].astype(np.float64) - ref[1]) / np.abs(asc[1].astype(np.float64))
        assert rel.max() <= 1e-6, (D, rel.max())
        _check_docs(W64, norms64, indptr, indices, ref[0], ref[1], range(3000))
        del Wd, norms, plan
    # kernel 1's rotated sweep (its automatic order): the same properties
    for k1 in (dict(kernel=1), dict(kernel=1, tile_docs=16, group_tiles=4), dict(kernel=1, tile_docs=2, mask_mode=1)):
        ref = _search(W, indptr, indices, perm=perm, **k1)
        for v in (dict(sweep=2), dict(neuron_chunk=256)):
            out = _search(W, indptr, indices, perm=perm, **k1, **v)
            assert np.array_equal(out[0], ref[0]) and np.array_equal(out[1], ref[1]), (k1, v)
        out = _search(W, indptr, indices, perm=perm, ldw=4100 + 1024, **k1)
        assert np.array_equal(out[0], ref[0]) and np.array_equal(out[1], ref[1]), k1
        Wd, _ = _dev_W(W)
        norms = som.som_codebook_norms(Wd, N=4100)
        ip, ix, pd = _dev_i32(indptr), _dev_i32(indices), _dev_i32(perm)
        plan = som.som_plan(ip, ix, 20000, perm=pd, **k1)
        pl = som.som_bmu_search_planned(Wd, norms, ip, plan, N=4100)
        t2 = som.som_bmu_search_top2(Wd, norms, ip, ix, N=4100, perm=pd, **k1)
        torch.cuda.synchronize()
        for b, d in (pl, t2[:2]):
            assert np.array_equal(b.cpu().numpy(), ref[0]) and np.array_equal(d.cpu().numpy(), ref[1]), k1
        asc = _search(W, indptr, indices, perm=perm, sweep=1, **k1)
        assert not np.array_equal(asc[1], ref[1]), k1
        rel = np.abs(asc[1].astype(np.float64) - ref[1]) / np.abs(asc[1].astype(np.float64))
        assert rel.max() <= 1e-6, (k1, rel.max())
        _check_docs(W64, norms64, indptr, indices, ref[0], ref[1], range(0, 3000, 3))
        del Wd, norms, plan


def test_rotated_sweep_exact_on_a_dyadic_codebook():
    """Rotated sweeps with long unions and many super-tiles per XCD (so the
    super-tiles start at nonzero stages and wrap round, ragged last stages
    included): on a dyadic codebook every fp32 sum is exact, so whatever the
    order each index (lowest on ties) and distance must equal the exact
    integer evaluation; a skipped or repeated row would not."""
    rng = np.random.default_rng(31)
    F, N, B = 2000, 61, 10240
    K = rng.integers(0, 4, (F, N))
    K[:, 60] = K[:, 7]                                  # exact duplicate neurons -> ties
    W = K.astype(np.float32) / 4
    nnz = rng.poisson(40, B).clip(1, 200)
    nnz[::97] = 0                                       # some empty documents
    indptr = np.concatenate([[0], np.cumsum(nnz)])
    indices = np.concatenate([np.sort(rng.choice(F, k, replace=False)) for k in nnz])
    exact = oracle.bmu_search_exact(K, 2, indptr, indices)
    want_b = [e[0] for e in exact]
    want_d = [Fraction(e[1], 16) for e in exact]
    perm = oracle.cluster_order(indptr, indices, F)
    for knobs in (dict(), dict(sweep=2), dict(tile_docs=128), dict(sweep=2, neuron_chunk=256),
                  dict(sweep=1), dict(kernel=1), dict(kernel=1, tile_docs=16, group_tiles=4, sweep=2),
                  dict(kernel=1, tile_docs=4, mask_mode=1), dict(kernel=1, sweep=1)):
        for p in (None, perm):
            bmu, dist, _ = _search(W, indptr, indices, perm=p, **knobs)
            assert bmu.tolist() == want_b, knobs
            assert [Fraction(float(x)) for x in dist] == want_d, knobs


# ----------------------------------------------------------------------------
# edge cases
# ----------------------------------------------------------------------------

def test_empty_batch_and_empty_documents():
    rng = np.random.default_rng(9)
    W = rng.random((10, 33), dtype=np.float32)
    bmu, dist, _ = _search(W, np.zeros(1, np.int64), np.zeros(0, np.int64))
    assert bmu.size == 0 and dist.size == 0
    indptr, indices = _csr([[], [], []])
    bmu, dist, norms = _search(W, indptr, indices)
    first = int(np.argmin(oracle.codebook_norms(W.astype(np.float64))))
    assert bmu.tolist() == [first] * 3


def test_single_neuron_and_long_documents():
    rng = np.random.default_rng(10)
    W = rng.random((5000, 1), dtype=np.float32)
    docs = _random_docs(rng, 40, 5000, mean=5, big_every=3, big=4000)
    indptr, indices = _csr(docs)
    bmu, dist, _ = _search(W, indptr, indices, ldw=4)
    assert np.all(bmu == 0)
    W64 = W.astype(np.float64)
    _check_docs(W64, oracle.codebook_norms(W64), indptr, indices, bmu, dist, range(40))


def test_largest_neuron_count_of_one_launch():
    # one launch takes at most 65,535 neuron slices (the grid's second
    # dimension): 256-neuron slices give N = 65,535 * 256.  Neurons planted
    # equal to a document (distance exactly 0) in the last slice and in the
    # first must be found; an exact tie across slices goes to the lower index.
    rng = np.random.default_rng(17)
    F, NMAX = 8, 65535 * 256
    ldw = NMAX + 64
    W = np.zeros((F, ldw), np.float32)
    W[:, :NMAX + 1] = rng.random((F, NMAX + 1), dtype=np.float32) * 0.5 + 0.25
    docs = _random_docs(rng, 40, F, mean=3, empty_every=13)
    docs[1], docs[2], docs[3] = [0, 3, 5], [1, 2, 7], [4, 6]
    plant = {1: [NMAX - 1], 2: [NMAX - 300], 3: [70000, 5]}   # doc -> neurons equal to it
    for d, js in plant.items():
        x = np.zeros(F, np.float32)
        x[docs[d]] = 1.0
        for j in js:
            W[:, j] = x
    indptr, indices = _csr(docs)
    W64 = W.astype(np.float64)
    norms64 = oracle.codebook_norms(W64, NMAX)
    Wd = torch.from_numpy(W).to(DEV)
    norms = som.som_codebook_norms(Wd, N=NMAX)
    ip, ix = _dev_i32(indptr), _dev_i32(indices)
    first = None
    for knobs in (dict(), dict(kernel=1, tile_docs=16), dict(kernel=1, lane_neurons=8), dict(kernel=3)):
        bmu, dist = som.som_bmu_search(Wd, norms, ip, ix, N=NMAX, sweep=1, **knobs)
        torch.cuda.synchronize()
        b, dd = bmu.cpu().numpy().astype(np.int64), dist.cpu().numpy().astype(np.float64)
        assert (b[1], b[2], b[3]) == (NMAX - 1, NMAX - 300, 5), (knobs, b[1:4])
        assert np.all(dd[1:4] == 0.0)
        if first is None:   # the oracle once; with the ascending sweep every launch form sums in the same order
            _check_docs(W64, norms64, indptr, indices, b, dd, range(len(docs)), N=NMAX)
            first = (b, dd)
        else:
            assert np.array_equal(b, first[0]) and np.array_equal(dd, first[1]), knobs
    # one neuron more needs a 65,536th slice at 256 neurons per slice (and
    # kernel 2's 32-neuron slices run out long before)
    norms1 = som.som_codebook_norms(Wd, N=NMAX + 1)
    for N, knobs in ((NMAX + 1, dict()), (NMAX + 1, dict(kernel=3)), (NMAX, dict(kernel=2))):
        with pytest.raises(som.SomError) as e:
            som.som_bmu_search(Wd, norms1[:N], ip, ix, N=N, **knobs)
        assert e.value.status == 1 and "slices" in str(e.value)
    # 512-neuron slices still fit: N = NMAX + 1 with 8 neurons per lane
    bmu, dist = som.som_bmu_search(Wd, norms1, ip, ix, N=NMAX + 1, kernel=1, lane_neurons=8)
    torch.cuda.synchronize()
    b = bmu.cpu().numpy().astype(np.int64)
    assert (b[1], b[2], b[3]) == (NMAX - 1, NMAX - 300, 5)
    _check_docs(W64, oracle.codebook_norms(W64, NMAX + 1), indptr, indices, b,
                dist.cpu().numpy().astype(np.float64), range(len(docs)), N=NMAX + 1)


def test_largest_tile_count_of_one_launch():
    # one launch takes fewer than 2^24 tiles: with one-document tiles the
    # largest batch is 2^24 - 1 documents (most of them empty here, so the
    # test stays small), and one more is rejected until the tiles grow
    rng = np.random.default_rng(19)
    F, N, B = 50, 300, (1 << 24) - 1
    W = rng.random((F, N), dtype=np.float32)
    lens = np.zeros(B + 1, np.int64)
    full = np.sort(rng.choice(B + 1, 400, replace=False))
    lens[full] = rng.integers(1, 12, full.size)
    docs = {int(d): np.sort(rng.choice(F, int(lens[d]), replace=False)) for d in full}
    indptr = np.zeros(B + 2, np.int64)
    indptr[1:] = np.cumsum(lens)
    indices = np.concatenate([docs[int(d)] for d in full])
    W64 = W.astype(np.float64)
    norms64 = oracle.codebook_norms(W64)
    Wd, ld = _dev_W(W)
    norms = som.som_codebook_norms(Wd, N=N)
    ipB = _dev_i32(indptr[:B + 1])
    nnzB = int(indptr[B])
    ixB = _dev_i32(indices[:nnzB])
    bmu, dist = som.som_bmu_search(Wd, norms, ipB, ixB, N=N, tile_docs=1, sweep=1)
    torch.cuda.synchronize()
    b, dd = bmu.cpu().numpy().astype(np.int64), dist.cpu().numpy().astype(np.float64)
    empty = lens[:B] == 0
    e0 = int(np.flatnonzero(empty)[0])
    _check_docs(W64, norms64, indptr, indices, b, dd, [e0] + [int(d) for d in full if d < B], N=N)
    assert np.all(b[empty] == b[e0]) and np.all(dd[empty] == dd[e0])
    # 2^24 documents: too many one-document tiles, fine as two-document tiles
    ip1, ix1 = _dev_i32(indptr), _dev_i32(indices)
    with pytest.raises(som.SomError) as e:
        som.som_bmu_search(Wd, norms, ip1, ix1, N=N, tile_docs=1)
    assert e.value.status == 1 and "too many tiles" in str(e.value)
    bmu2, dist2 = som.som_bmu_search(Wd, norms, ip1, ix1, N=N, tile_docs=2, sweep=1)
    torch.cuda.synchronize()
    b2, d2 = bmu2.cpu().numpy().astype(np.int64), dist2.cpu().numpy().astype(np.float64)
    assert np.array_equal(b2[:B], b) and np.array_equal(d2[:B], dd)
    _check_docs(W64, norms64, indptr, indices, b2, d2, [B], N=N)


def test_neuron_ranges_compose_to_the_full_search():
    # The neuron-sharded form on one GPU: each column range of W is searched
    # through the C ABI at a pointer offset into the same feature-major rows
    # (same ldw, the norms at the same offset); keeping each document's smaller
    # distance, the earlier range's on a tie, gives the whole-map search bit for
    # bit, exact ties across ranges included.
    import ctypes
    from paper_2609_05138_amd import som as abi
    rng = np.random.default_rng(23)
    F, N = 300, 1000
    W = rng.random((F, N), dtype=np.float32)
    docs = _random_docs(rng, 700, F, mean=12, empty_every=97)
    for d, cols in ((5, (100, 700)), (6, (3, 950)), (7, (255, 256))):   # planted exact ties
        x = np.zeros(F, np.float32)
        x[docs[d]] = 1.0
        for j in cols:
            W[:, j] = x
    W[:, 604] = W[:, 603]                                               # a tie at a range edge
    indptr, indices = _csr(docs)
    B = len(docs)
    # a range at offset r0 reads no row beyond round_up(n, 4) elements from
    # W + r0, so the buffer needs no slack after its last row
    ldw = 1024
    buf = torch.zeros(F * ldw, dtype=torch.float32, device=DEV)
    Wd = buf[:F * ldw].view(F, ldw)
    Wd[:, :N] = torch.from_numpy(W).to(DEV)
    norms = som.som_codebook_norms(Wd, N=N)
    ip, ix = _dev_i32(indptr), _dev_i32(indices)
    lib = som.load()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for knobs in (dict(), dict(kernel=1, tile_docs=16), dict(kernel=3)):
        full_b, full_d = som.som_bmu_search(Wd, norms, ip, ix, N=N, **knobs)
        best_b = np.full(B, -1, np.int64)
        best_d = np.full(B, np.inf, np.float32)
        for r0, r1 in ((0, 256), (256, 604), (604, N)):                 # offsets keep 16-byte rows
            n = r1 - r0
            o = abi.som_bmu_opts(int(knobs.get("kernel", 0)), int(knobs.get("tile_docs", 0)), 0, 0, 0, 0, 0, 0)
            need = int(lib.som_bmu_workspace_bytes(F, n, B, len(indices), ctypes.byref(o)))
            ws = torch.empty(max(need, 1), dtype=torch.uint8, device=DEV)
            bmu = torch.empty(B, dtype=torch.int32, device=DEV)
            dist = torch.empty(B, dtype=torch.float32, device=DEV)
            st = lib.som_bmu_search(Wd.data_ptr() + 4 * r0, F, n, ldw, norms.data_ptr() + 4 * r0, ip.data_ptr(),
                                    ix.data_ptr(), B, len(indices), None, bmu.data_ptr(), dist.data_ptr(),
                                    ctypes.byref(o), ws.data_ptr(), ws.numel(), stream)
            assert st == abi.SOM_OK, lib.som_last_error()
            torch.cuda.synchronize()
            b = bmu.cpu().numpy().astype(np.int64) + r0
            dd = dist.cpu().numpy()
            take = dd < best_d                                           # strict: the earlier range keeps ties
            best_b[take], best_d[take] = b[take], dd[take]
        torch.cuda.synchronize()
        assert np.array_equal(best_b, full_b.cpu().numpy().astype(np.int64)), knobs
        assert np.array_equal(best_d, full_d.cpu().numpy()), knobs
        assert (best_b[5], best_b[6], best_b[7]) == (100, 3, 255)


def test_binding_rejects_short_norms():
    # the C ABI cannot size device buffers: the binding checks norms against N
    rng = np.random.default_rng(29)
    W = rng.random((40, 96), dtype=np.float32)
    Wd, _ = _dev_W(W)
    norms = som.som_codebook_norms(Wd, N=90)
    ip, ix = _dev_i32(np.array([0, 2, 3])), _dev_i32(np.array([1, 7, 5]))
    with pytest.raises(ValueError):
        som.som_bmu_search(Wd, norms, ip, ix, N=96)         # the row stride is not N
    with pytest.raises(ValueError):
        som.som_bmu_search_top2(Wd, norms, ip, ix, N=91)
    plan = som.som_plan(ip, ix, 40)
    with pytest.raises(ValueError):
        som.som_bmu_search_planned(Wd, norms, ip, plan, N=96)
    bmu, dist = som.som_bmu_search(Wd, norms, ip, ix, N=90)
    # without N the binding takes the norms' length, never the padded stride
    b0, d0 = som.som_bmu_search(Wd, norms, ip, ix)
    torch.cuda.synchronize()
    assert torch.equal(b0, bmu) and torch.equal(d0, dist)
    W64 = W.astype(np.float64)
    _check_docs(W64, oracle.codebook_norms(W64, 90), np.array([0, 2, 3]), np.array([1, 7, 5]),
                bmu.cpu().numpy(), dist.cpu().numpy(), range(2), N=90)


def test_validate_rejects_malformed_batches():
    rng = np.random.default_rng(11)
    W = rng.random((50, 64), dtype=np.float32)
    Wd, _ = _dev_W(W)
    norms = som.som_codebook_norms(Wd)
    good_ptr, good_idx = _csr([[1, 4, 9], [2], [], [0, 49]])
    som.som_bmu_search(Wd, norms, _dev_i32(good_ptr), _dev_i32(good_idx), validate=True)
    cases = [
        (good_ptr, np.array([1, 9, 4, 2, 0, 49])),            # unsorted
        (good_ptr, np.array([1, 4, 4, 2, 0, 49])),            # duplicate
        (good_ptr, np.array([1, 4, 9, 2, 0, 50])),            # out of range
        (good_ptr, np.array([1, 4, 9, 2, -1, 49])),           # negative
        (np.array([0, 3, 2, 4, 6]), good_idx),                # indptr decreases
    ]
    for ip, ix in cases:
        with pytest.raises(som.SomError) as e:
            som.som_bmu_search(Wd, norms, _dev_i32(ip), _dev_i32(ix), validate=True)
        assert e.value.status == 2
    with pytest.raises(som.SomError) as e:
        som.som_bmu_search(Wd, norms, _dev_i32(good_ptr), _dev_i32(good_idx),
                           perm=_dev_i32(np.array([0, 1, 1, 3])), validate=True)
    assert e.value.status == 2


def test_planned_search_reuses_a_plan_across_codebooks():
    from synth import codebook, documents
    indptr, indices = documents(1, 0, n_docs=2500)
    ip, ix = _dev_i32(indptr), _dev_i32(indices)
    perm = _dev_i32(oracle.cluster_order(indptr, indices, 2048))
    plan = som.som_plan(ip, ix, 2048, perm=perm, sweep=1)       # kernel 3, ascending sweep
    plan1 = som.som_plan(ip, ix, 2048, perm=perm, kernel=1, tile_docs=4, sweep=1)
    planr = som.som_plan(ip, ix, 2048, perm=perm)                # kernel 3, rotated sweep
    for seed in (0, 1):
        W = codebook(1, seed=seed)
        Wd, _ = _dev_W(W)
        norms = som.som_codebook_norms(Wd)
        a = som.som_bmu_search_planned(Wd, norms, ip, plan)
        b = som.som_bmu_search(Wd, norms, ip, ix, perm=perm, kernel=1, tile_docs=4, sweep=1)
        c = som.som_bmu_search_planned(Wd, norms, ip, plan1)
        r = som.som_bmu_search_planned(Wd, norms, ip, planr)
        r0 = som.som_bmu_search(Wd, norms, ip, ix, perm=perm)
        torch.cuda.synchronize()
        assert torch.equal(r[0], r0[0]) and torch.equal(r[1], r0[1])
        assert torch.equal(a[0], c[0]) and torch.equal(a[1], c[1])
        torch.cuda.synchronize()
        assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
        W64 = W.astype(np.float64)
        _check_docs(W64, oracle.codebook_norms(W64), indptr, indices, a[0].cpu().numpy(),
                    a[1].cpu().numpy(), range(0, 2500, 7))


def test_read_probe_runs_and_leaves_the_buffer_alone():
    """The bandwidth probe only reads: the buffer is unchanged after several
    passes, at sizes that are not multiples of its workgroup step."""
    buf = torch.arange(1 << 18, dtype=torch.int32, device=DEV)      # 1 MiB
    ref = buf.clone()
    sink = torch.zeros(1, dtype=torch.int32, device=DEV)
    for nbytes, passes in ((16, 1), (4096 + 16, 3), (1 << 20, 2)):
        som.som_probe_read(buf, nbytes, passes, sink)
    torch.cuda.synchronize()
    assert torch.equal(buf, ref)


def test_lds_probe_reports_its_bytes():
    """The LDS probe runs four 8-wave workgroups per CU, each wave reading
    `iters` 1 KB rows, and reports exactly those bytes."""
    sink = torch.zeros(1, dtype=torch.int32, device=DEV)
    cus = torch.cuda.get_device_properties(DEV).multi_processor_count
    for iters in (4, 1024):
        assert som.som_probe_lds(iters, sink) == cus * 4 * 8 * iters * 1024
    torch.cuda.synchronize()
