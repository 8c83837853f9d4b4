"""GPU parity of the batch-SOM update (accumulate, neighbourhood blur,
write-back) through the C ABI, against the fp64 oracle (oracle/update.py).

Accumulation is integer work: bit-exact.  With sigma = 0 the write-back is a
quotient of two exact integers: bit-exact against IEEE fp32 division.  With
sigma > 0 the device forms each numerator and denominator with two passes of
at most 2R + 1 fp32 products of positive terms (taps rounded once from fp64),
so each carries a relative error below (2 (2R + 1) + 1) u, u = 2^-24, and the
quotient below twice that plus u: the tolerance used here is
(4 (2R + 1) + 4) u relative.  Units whose neighbourhood caught nothing keep
their weights bit for bit.
"""

import math

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2609_05138_amd as som
else:  # collected on CPU-only machines, never run there
    som = None

DEV = "cuda:0"
U = 2.0 ** -24


def _csr(docs):
    indptr = np.zeros(len(docs) + 1, np.int64)
    indptr[1:] = np.cumsum([len(d) for d in docs])
    indices = np.array([f for d in docs for f in d], dtype=np.int64)
    return indptr, indices


def _i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def _batch(rng, B, F, N, mean=8, bmu_pool=None):
    docs = [np.unique(rng.integers(0, F, int(rng.poisson(mean)))).tolist() for _ in range(B)]
    pool = N if bmu_pool is None else bmu_pool
    return docs, rng.integers(0, pool, B)


def _accumulate(batches, F, N, ld=None):
    ld = N if ld is None else ld
    acc = torch.zeros((F, ld), dtype=torch.int32, device=DEV)
    cnt = torch.zeros(N, dtype=torch.int32, device=DEV)
    for docs, bmu in batches:
        indptr, indices = _csr(docs)
        som.som_update_accumulate(_i32(indptr), _i32(indices), _i32(bmu), F, N, acc, cnt)
    return acc, cnt


def test_accumulate_is_exact_over_batches_and_ignores_foreign_units():
    rng = np.random.default_rng(0)
    F, N = 70, 48
    batches = [_batch(rng, B, F, N) for B in (300, 1, 157)]
    bad_docs, bad_bmu = _batch(rng, 20, F, N)
    bad_bmu[::2] = N + 3                                   # not units of this map
    bad_bmu[1::4] = -1
    acc, cnt = _accumulate(batches + [(bad_docs, bad_bmu)], F, N, ld=N + 5)
    want_a, want_c = None, None
    for docs, bmu in batches:
        want_a, want_c = oracle.update_accumulate(*_csr(docs), bmu, F, N, acc=want_a, count=want_c)
    keep = (bad_bmu >= 0) & (bad_bmu < N)
    want_a, want_c = oracle.update_accumulate(*_csr([d for d, k in zip(bad_docs, keep) if k]), bad_bmu[keep], F, N,
                                              acc=want_a, count=want_c)
    a = acc.cpu().numpy().astype(np.int64)
    assert np.array_equal(a[:, :N], want_a) and np.all(a[:, N:] == 0)
    assert np.array_equal(cnt.cpu().numpy().astype(np.int64), want_c)


def _finish(W, acc, cnt, rows, cols, sigma, f16=False):
    dt = torch.float16 if f16 else torch.float32
    Wd = torch.from_numpy(W.astype(np.float16 if f16 else np.float32)).to(DEV)
    assert Wd.dtype == dt
    som.som_update_finish(Wd, rows, cols, sigma, acc, cnt)
    torch.cuda.synchronize()
    return Wd.cpu().numpy()


@pytest.mark.parametrize("rows,cols", [(4, 5), (16, 16), (1, 37), (33, 8)])
def test_sigma_zero_is_the_exact_mean(rows, cols):
    rng = np.random.default_rng(rows * 100 + cols)
    F, N = 50, rows * cols
    docs, bmu = _batch(rng, 400, F, N, bmu_pool=max(1, N - 3))
    acc, cnt = _accumulate([(docs, bmu)], F, N)
    W = rng.random((F, N)).astype(np.float32)
    got = _finish(W, acc, cnt, rows, cols, 0.0)
    oa, oc = oracle.update_accumulate(*_csr(docs), bmu, F, N)
    a, c = oa.astype(np.float32), oc.astype(np.float32)   # exact: counts are far below 2^24
    want = W.copy()
    moved = c > 0
    want[:, moved] = a[:, moved] / c[moved]               # IEEE fp32 division of exact integers
    assert np.array_equal(got, want)
    ref = oracle.update_finish(W.astype(np.float64), oa, oc, rows, cols, 0.0)
    assert np.array_equal(got, ref.astype(np.float32))


@pytest.mark.parametrize("rows,cols,sigma", [(4, 5, 0.5), (16, 16, 1.0), (1, 37, 2.5), (33, 8, 2.5),
                                             (12, 12, 7.3), (9, 20, 0.2), (20, 130, 2.0), (70, 67, 5.3),
                                             (5, 200, 1.7)])
def test_blur_matches_oracle(rows, cols, sigma):
    rng = np.random.default_rng(int(sigma * 10) + rows)
    F, N = 40, rows * cols
    docs, bmu = _batch(rng, 500, F, N, bmu_pool=max(1, N // 2))   # far units may catch nothing
    acc, cnt = _accumulate([(docs, bmu)], F, N)
    W = rng.random((F, N)).astype(np.float32)
    got = _finish(W, acc, cnt, rows, cols, sigma).astype(np.float64)
    oa, oc = oracle.update_accumulate(*_csr(docs), bmu, F, N)
    ref = oracle.update_finish(W.astype(np.float64), oa, oc, rows, cols, sigma)
    R = oracle.neighbourhood_radius(sigma)
    tol = (4 * (2 * R + 1) + 4) * U
    den = oc.astype(np.float64) @ oracle.neighbourhood(rows, cols, sigma)
    moved = den > 0
    assert np.all(np.abs(got[:, moved] - ref[:, moved]) <= tol * np.abs(ref[:, moved]) + 1e-30)
    assert np.array_equal(got[:, ~moved], W[:, ~moved].astype(np.float64))


def test_fp16_write_back_rounds_the_fp32_quotient():
    rng = np.random.default_rng(11)
    rows, cols, sigma, F = 10, 12, 1.3, 30
    N = rows * cols
    docs, bmu = _batch(rng, 300, F, N)
    acc, cnt = _accumulate([(docs, bmu)], F, N)
    W = rng.random((F, N)).astype(np.float16)
    got16 = _finish(W, acc, cnt, rows, cols, sigma, f16=True)
    got32 = _finish(W.astype(np.float32), acc, cnt, rows, cols, sigma)
    assert np.array_equal(got16, got32.astype(np.float16))    # same quotient, rounded once to fp16


def test_many_feature_chunks_and_a_large_radius():
    """More feature planes than one workspace chunk: sigma = 0 everywhere and
    sigma > 0 on a sample of features (features are independent)."""
    rows, cols = 256, 16
    N = rows * cols
    planes = (1 << 26) // N                                   # planes per chunk
    F = planes * 2 + 37
    rng = np.random.default_rng(21)
    docs, bmu = _batch(rng, 20000, F, N, mean=60)
    acc, cnt = _accumulate([(docs, bmu)], F, N)
    W = rng.random((F, N)).astype(np.float32)
    # the oracle's own accumulators: the device's must equal them exactly
    oa, oc = oracle.update_accumulate(*_csr(docs), bmu, F, N)
    assert np.array_equal(acc.cpu().numpy().astype(np.int64), oa)
    assert np.array_equal(cnt.cpu().numpy().astype(np.int64), oc)
    got0 = _finish(W, acc, cnt, rows, cols, 0.0)
    c = oc.astype(np.float32)
    moved = c > 0
    want0 = W.copy()
    want0[:, moved] = oa[:, moved].astype(np.float32) / c[moved]    # exact integers, one IEEE division
    assert np.array_equal(got0, want0)
    sigma = 9.0
    got = _finish(W, acc, cnt, rows, cols, sigma).astype(np.float64)
    sample = np.unique(np.concatenate([[0, planes - 1, planes, 2 * planes, F - 1], rng.choice(F, 25, replace=False)]))
    ref = oracle.update_finish(W[sample].astype(np.float64), oa[sample], oc, rows, cols, sigma)
    R = oracle.neighbourhood_radius(sigma)
    tol = (4 * (2 * R + 1) + 4) * U
    assert np.all(np.abs(got[sample] - ref) <= tol * np.abs(ref) + 1e-30)
    assert math.isfinite(float(got.sum()))


def test_full_size_update_on_the_512_map():
    """The benchmark's update configuration, on sampled outputs: a 512 x 512
    map, F = 20,000, one 1,048,576-document batch of the 512^2 workload and
    sigma = 2 (R = 6).  The assignments are seeded inputs (not search
    results).  The oracle accumulates the sampled features only (the scatter
    is independent per feature) and evaluates the window sums at sampled
    units, borders and corners included."""
    from synth import documents
    rows = cols = 512
    N, F, sigma = rows * cols, 20000, 2.0
    indptr, indices = documents(4, 0)
    B = len(indptr) - 1
    rng = np.random.default_rng(31)
    bmu = rng.integers(0, N, B)
    ldw = som.som_codebook_ldw(N)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(7)
    W = torch.rand((F, ldw), generator=gen, device=DEV)
    feats = np.unique(np.concatenate([[0, 1, 9, 99, 999, F - 1], rng.choice(F, 10, replace=False)]))
    fidx = torch.from_numpy(feats).to(DEV)
    old = W[fidx].cpu().numpy()                         # this test's own input, before the update
    acc = torch.zeros((F, N), dtype=torch.int32, device=DEV)
    cnt = torch.zeros(N, dtype=torch.int32, device=DEV)
    som.som_update_accumulate(_i32(indptr), _i32(indices), _i32(bmu), F, N, acc, cnt)
    som.som_update_finish(W, rows, cols, sigma, acc, cnt)
    torch.cuda.synchronize()
    got_acc = acc[fidx].cpu().numpy().astype(np.int64)
    got_cnt = cnt.cpu().numpy().astype(np.int64)
    new = W[fidx].cpu().numpy().astype(np.float64)
    del acc, W
    torch.cuda.empty_cache()
    keep = np.isin(indices, feats)
    docid = np.repeat(np.arange(B), np.diff(indptr))
    ip_f = np.zeros(B + 1, np.int64)
    ip_f[1:] = np.cumsum(np.bincount(docid[keep], minlength=B))
    ix_f = np.searchsorted(feats, indices[keep])
    oa, oc = oracle.update_accumulate(ip_f, ix_f, bmu, len(feats), N)
    assert np.array_equal(got_acc, oa) and np.array_equal(got_cnt, oc)
    edge = [0, 1, cols - 1, N - cols, N - 1, 5 * cols, 8 * cols - 2, N - 4, 256 * cols + 256]
    units = np.unique(np.concatenate([edge, rng.choice(N, 120, replace=False)]))
    ref = oracle.update_finish_at(old[:, units].astype(np.float64), oa, oc, rows, cols, sigma, units)
    R = oracle.neighbourhood_radius(sigma)
    tol = (4 * (2 * R + 1) + 4) * U
    assert np.all(np.abs(new[:, units] - ref) <= tol * np.abs(ref) + 1e-30)
