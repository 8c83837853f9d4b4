"""The seeded input generators: determinism, structure and distributions."""

import numpy as np
import pytest

from synth import CONFIGS, batch_sizes, codebook, codebook_rows, documents, topic_subsets, zipf_cdf


def _check_csr(indptr, indices, F):
    assert indptr.dtype == np.int32 and indices.dtype == np.int32
    assert indptr[0] == 0 and indptr[-1] == len(indices)
    assert np.all(np.diff(indptr) >= 0)
    assert indices.min() >= 0 and indices.max() < F
    starts = np.zeros(len(indices), bool)
    starts[indptr[:-1][np.diff(indptr) > 0]] = True
    inc = np.diff(indices.astype(np.int64))
    assert np.all(inc[~starts[1:]] > 0), "indices must be strictly ascending within a row"


def test_batch_sizes_cover_every_document():
    for c in CONFIGS.values():
        s = batch_sizes(c)
        assert sum(s) == c.docs and all(0 < x <= c.batch for x in s)
    assert batch_sizes(2)[-1] == 16_960 and len(batch_sizes(2)) == 16
    assert batch_sizes(4) == [1_048_576, 951_424]
    assert len(batch_sizes(5)) == 27 and batch_sizes(5)[-1] == 900_000


def test_documents_are_deterministic_and_distinct_per_batch():
    a = documents(2, 0, n_docs=3000)
    b = documents(2, 0, n_docs=3000)
    c = documents(2, 1, n_docs=3000)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert not np.array_equal(a[1][:200], c[1][:200])
    d = documents(2, 0, seed=1, n_docs=3000)
    assert not np.array_equal(a[1][:200], d[1][:200])


@pytest.mark.parametrize("cfg,n", [(1, None), (2, 20000), (3, 20000), (5, 20000)])
def test_documents_are_valid_csr(cfg, n):
    ip, ix = documents(cfg, 0, n_docs=n)
    _check_csr(ip, ix, CONFIGS[cfg].F)
    assert np.diff(ip).min() >= 1


def test_poisson_nnz_and_zipf_document_frequencies():
    ip, ix = documents(2, 0)          # one full 65,536-document batch
    nnz = np.diff(ip)
    assert abs(nnz.mean() - 80.0) < 0.3 and abs(nnz.var() - 80.0) < 4.0
    df = np.bincount(ix, minlength=20_000) / len(nnz)
    # successive sampling from Zipf(1.1): the head is in nearly every
    # document, rank 10 in ~3/4, rank 100 in ~1/9, rank 1000 in ~1/100
    assert df[0] > 0.99
    assert 0.70 < df[9] < 0.84
    assert 0.08 < df[99] < 0.14
    assert 0.005 < df[999] < 0.02
    assert np.all(np.diff(df[:50]) <= 0.02)     # frequency-ordered ids


def test_lognormal_nnz():
    ip, _ = documents(3, 0, n_docs=40000)
    nnz = np.diff(ip)
    assert abs(np.median(nnz) - 70) <= 2
    assert nnz.min() >= 1 and nnz.max() <= 2000
    ls = np.log(nnz[(nnz > 1) & (nnz < 2000)])
    assert abs(ls.std() - 0.6) < 0.03


def test_topic_workload_has_no_global_head():
    c = CONFIGS[5]
    sub = topic_subsets(5)
    assert sub.shape == (256, 2000)
    assert all(len(set(r.tolist())) == 2000 for r in sub[:8])
    ip, ix = documents(5, 0, n_docs=40000)
    df = np.bincount(ix, minlength=c.F) / (len(ip) - 1)
    assert df.max() < 0.05
    assert np.count_nonzero(df) > 19_000
    nnz = np.diff(ip)
    assert abs(np.median(nnz) - 80) <= 3 and nnz.max() <= 4000
    # every document draws only from the union of at most three topic subsets
    topic_of = np.zeros((256, c.F), bool)
    for t in range(256):
        topic_of[t, sub[t]] = True
    for d in range(0, 400, 7):
        feats = ix[ip[d]:ip[d + 1]]
        covering = topic_of[:, feats].all(axis=1)
        if not covering.any():
            # needs two or three topics: check some set of <= 3 topics covers it
            cnt = topic_of[:, feats].sum(axis=1)
            top = np.argsort(-cnt)[:12]
            ok = False
            for a in top:
                for b in top:
                    for e in top:
                        if (topic_of[a, feats] | topic_of[b, feats] | topic_of[e, feats]).all():
                            ok = True
                            break
                    if ok:
                        break
                if ok:
                    break
            assert ok, d


def test_codebook_values_are_dyadic_and_regenerable():
    W = codebook(1, N=64, F=40, ldw=68)
    assert W.shape == (40, 68) and W.dtype == np.float32
    assert np.all(W[:, 64:] == 0)
    body = W[:, :64].astype(np.float64)
    assert body.min() >= 0 and body.max() < 1
    k = body * (1 << 24)
    assert np.array_equal(k, np.rint(k))
    rows = codebook_rows(1, [0, 17, 39], N=64)
    assert np.array_equal(rows, W[[0, 17, 39], :64])
    assert abs(body.mean() - 0.5) < 0.02


def test_zipf_cdf():
    cdf = zipf_cdf(5, 1.0)
    h = 1 + 1 / 2 + 1 / 3 + 1 / 4 + 1 / 5
    assert np.allclose(cdf, np.cumsum([1, 1 / 2, 1 / 3, 1 / 4, 1 / 5]) / h)
    assert cdf[-1] == 1.0
