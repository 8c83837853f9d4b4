"""Pins of the batch-SOM update oracle (oracle/update.py) against closed
forms and invariants; see that module for the reading of the neighbourhood."""

import math

import numpy as np
import pytest

import oracle


def _csr(docs):
    indptr = np.zeros(len(docs) + 1, np.int64)
    indptr[1:] = np.cumsum([len(d) for d in docs])
    indices = np.array([f for d in docs for f in d], dtype=np.int64)
    return indptr, indices


def _dense(docs, F):
    X = np.zeros((len(docs), F))
    for i, d in enumerate(docs):
        X[i, d] = 1.0
    return X


def _random(rng, B, F, N, mean=6):
    docs = [sorted(rng.choice(F, min(F, int(rng.poisson(mean))), replace=False).tolist()) for _ in range(B)]
    return docs, rng.integers(0, N, B)


def test_sigma_zero_gives_each_unit_the_mean_of_its_documents():
    rng = np.random.default_rng(0)
    F, rows, cols = 30, 3, 4
    N = rows * cols
    docs, bmu = _random(rng, 50, F, N - 2)          # the last two units catch nothing
    W = rng.random((F, N))
    acc, cnt = oracle.update_accumulate(*_csr(docs), bmu, F, N)
    new = oracle.update_finish(W, acc, cnt, rows, cols, 0.0)
    X = _dense(docs, F)
    for j in range(N):
        mine = X[bmu == j]
        want = mine.mean(axis=0) if len(mine) else W[:, j]
        assert np.allclose(new[:, j], want, rtol=0, atol=1e-15), j


def test_one_document_moves_its_whole_neighbourhood_onto_itself():
    F, rows, cols, sigma = 12, 5, 6, 1.2
    N = rows * cols
    doc, b = [1, 4, 7], 14                           # unit 14 = row 2, column 2
    W = np.full((F, N), 0.25)
    acc, cnt = oracle.update_accumulate(*_csr([doc]), np.array([b]), F, N)
    new = oracle.update_finish(W, acc, cnt, rows, cols, sigma)
    x = _dense([doc], F)[0]
    R = oracle.neighbourhood_radius(sigma)
    assert R == 4
    for j in range(N):
        inside = abs(j // cols - b // cols) <= R and abs(j % cols - b % cols) <= R
        assert np.allclose(new[:, j], x if inside else W[:, j], rtol=0, atol=1e-15), j


@pytest.mark.parametrize("rows,cols,sigma", [(1, 7, 0.5), (4, 4, 1.0), (6, 3, 2.2), (5, 9, 0.34)])
def test_neighbourhood_is_a_symmetric_product_of_truncated_1d_gaussians(rows, cols, sigma):
    H = oracle.neighbourhood(rows, cols, sigma)
    R = math.ceil(3 * sigma)

    def g(k):
        return math.exp(-k * k / (2 * sigma * sigma)) if abs(k) <= R else 0.0

    N = rows * cols
    for i in range(N):
        for j in range(N):
            want = g(i // cols - j // cols) * g(i % cols - j % cols)
            assert abs(H[i, j] - want) <= 1e-15 * max(1.0, want), (i, j)
    assert np.array_equal(H, H.T)


def test_hand_worked_three_unit_line():
    # 1 x 3 map, sigma = 1 (R = 3): document {0} lands on unit 0, document {1} on
    # unit 2.  Unit 1 sees both at weight e^-1/2: (1/2, 1/2).  Unit 0 sees its own
    # document at weight 1 and the other at e^-2: (1, e^-2) / (1 + e^-2).
    W = np.zeros((2, 3))
    acc, cnt = oracle.update_accumulate(*_csr([[0], [1]]), np.array([0, 2]), 2, 3)
    new = oracle.update_finish(W, acc, cnt, 1, 3, 1.0)
    e2 = math.exp(-2.0)
    assert np.allclose(new[:, 1], [0.5, 0.5], rtol=0, atol=1e-15)
    assert np.allclose(new[:, 0], [1 / (1 + e2), e2 / (1 + e2)], rtol=0, atol=1e-15)
    assert np.allclose(new[:, 2], [e2 / (1 + e2), 1 / (1 + e2)], rtol=0, atol=1e-15)


def test_accumulation_is_linear_and_order_free():
    rng = np.random.default_rng(3)
    F, N = 40, 20
    d1, b1 = _random(rng, 60, F, N)
    d2, b2 = _random(rng, 45, F, N)
    a1, c1 = oracle.update_accumulate(*_csr(d1), b1, F, N)
    a12, c12 = oracle.update_accumulate(*_csr(d2), b2, F, N, acc=a1.copy(), count=c1.copy())
    a, c = oracle.update_accumulate(*_csr(d1 + d2), np.concatenate([b1, b2]), F, N)
    assert np.array_equal(a12, a) and np.array_equal(c12, c)
    p = rng.permutation(len(d1))
    ap, cp = oracle.update_accumulate(*_csr([d1[i] for i in p]), b1[p], F, N)
    assert np.array_equal(ap, a1) and np.array_equal(cp, c1)
    assert cp.sum() == len(d1) and ap.sum() == sum(len(d) for d in d1)


def test_update_equals_the_weighted_mean_written_out():
    # the batch map: w_j = sum_d h(b_d, j) x_d / sum_d h(b_d, j)
    rng = np.random.default_rng(5)
    F, rows, cols, sigma = 15, 3, 5, 0.8
    N = rows * cols
    docs, bmu = _random(rng, 70, F, N)
    W = rng.random((F, N))
    acc, cnt = oracle.update_accumulate(*_csr(docs), bmu, F, N)
    new = oracle.update_finish(W, acc, cnt, rows, cols, sigma)
    H = oracle.neighbourhood(rows, cols, sigma)
    X = _dense(docs, F)
    for j in range(N):
        wts = np.array([H[b, j] for b in bmu])
        if wts.sum() > 0:
            assert np.allclose(new[:, j], (wts[:, None] * X).sum(axis=0) / wts.sum(), rtol=1e-13, atol=1e-15)
        else:
            assert np.array_equal(new[:, j], W[:, j])


@pytest.mark.parametrize("rows,cols,sigma", [(6, 7, 0.0), (6, 7, 0.8), (9, 5, 1.7), (1, 40, 2.5), (12, 12, 3.1)])
def test_pointwise_finish_equals_the_dense_one(rows, cols, sigma):
    # every unit, borders included (truncated windows)
    rng = np.random.default_rng(int(sigma * 10) + rows)
    F, N = 20, rows * cols
    docs, bmu = _random(rng, 120, F, max(1, N - 5))
    W = rng.random((F, N))
    acc, cnt = oracle.update_accumulate(*_csr(docs), bmu, F, N)
    dense = oracle.update_finish(W, acc, cnt, rows, cols, sigma)
    units = np.arange(N)
    at = oracle.update_finish_at(W[:, units], acc, cnt, rows, cols, sigma, units)
    assert np.allclose(at, dense, rtol=1e-12, atol=0.0)


def test_pointwise_finish_closed_forms_on_a_512_map():
    # one document moves exactly the units of its window onto itself; with
    # sigma = 0 a unit becomes the mean of its documents
    rows = cols = 512
    N = rows * cols
    F = 6
    x = [1, 4]
    b = 3 * cols + 500                                   # near a corner: a clipped window
    acc, cnt = oracle.update_accumulate(*_csr([x]), np.array([b]), F, N)
    W = np.full((F, 5), 0.25)
    units = np.array([b, b - 2 * cols + 3, b + 6 * cols, b + 7 * cols, 0])   # in, in, in (R = 6), out, out
    got = oracle.update_finish_at(W, acc, cnt, rows, cols, 2.0, units)
    want = np.zeros(F)
    want[x] = 1.0
    for k in range(3):
        assert np.array_equal(got[:, k], want)
    assert np.array_equal(got[:, 3:], W[:, 3:])
    docs = [[0, 2], [2, 5], [1]]
    bm = np.array([77, 77, 9000])
    acc, cnt = oracle.update_accumulate(*_csr(docs), bm, F, N)
    got = oracle.update_finish_at(np.zeros((F, 3)), acc, cnt, rows, cols, 0.0, [77, 9000, 78])
    assert np.array_equal(got[:, 0], np.array([0.5, 0, 1.0, 0, 0, 0.5]))
    assert np.array_equal(got[:, 1], np.array([0, 1.0, 0, 0, 0, 0]))
    assert np.array_equal(got[:, 2], np.zeros(F))
