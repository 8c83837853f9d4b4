"""The allocation-free search (som_bmu_search_noalloc) through the C ABI.

Collected last (its name) so that, run after every other test, it also shows
that nothing earlier leaves state it depends on.

Host-only checks (no GPU): sizes beyond the static scratch array and the
synchronising validation are rejected before any HIP call.  GPU checks: two
calls in a row, the second on a smaller batch of another shape, each
bit-identical to som_bmu_search on the same inputs (the two run the same
kernels; the second call must not see anything the first left in the shared
array), plus an oracle check of sampled documents.
"""

import ctypes
import os

import numpy as np
import pytest

import oracle

som = pytest.importorskip("paper_2609_05138_amd.som")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(som.LIB_PATH):
        pytest.fail("libsom.so is not built (run python -m paper_2609_05138_amd.build)")
    return som.load()


def _call(lib, W, F, N, ldw, norms, indptr, indices, B, nnz, perm, bmu, dist, opts, stream=None):
    st = lib.som_bmu_search_noalloc(W, F, N, ldw, norms, indptr, indices, B, nnz, perm, bmu, dist, opts, stream)
    return st, lib.som_last_error().decode()


def test_noalloc_rejects_oversized_batches_on_the_host(lib):
    fake = ctypes.c_void_p(0x1000)          # never dereferenced: rejected before any HIP call
    # a 1M-document, 84M-nonzero plan needs far more than the 64 MiB array
    st, msg = _call(lib, fake, 20000, 262144, 262208, fake, fake, fake, 1 << 20, 84_000_000, None, fake, fake, None)
    assert st == som.SOM_ERR_INVALID_ARG and "more than" in msg, msg
    need = lib.som_bmu_workspace_bytes(20000, 262144, 1 << 20, 84_000_000, None)
    assert need > som.NOALLOC_SCRATCH_BYTES
    o = som.som_bmu_opts()
    o.validate = 1
    st, msg = _call(lib, fake, 64, 64, 64, fake, fake, fake, 8, 80, None, fake, fake, ctypes.byref(o))
    assert st == som.SOM_ERR_INVALID_ARG and "validate" in msg, msg
    st, _ = _call(lib, None, 64, 64, 64, fake, fake, fake, 8, 80, None, fake, fake, None)
    assert st == som.SOM_ERR_INVALID_ARG
    # an empty batch is a no-op that touches nothing
    st, _ = _call(lib, fake, 64, 64, 64, fake, fake, None, 0, 0, None, None, None, None)
    assert st == som.SOM_OK


def _gpu_case(lib, cfg, batch, n_docs, N, F, cluster, knobs):
    import torch
    from synth import codebook, documents
    dev = torch.device("cuda:0")
    W = codebook(cfg, N=N, F=F)
    indptr, indices = documents(cfg, batch, n_docs=n_docs)
    B, nnz = len(indptr) - 1, len(indices)
    print(f"[noalloc] cfg{cfg} batch {batch}: B={B} nnz={nnz} N={N} F={F} knobs={knobs}", flush=True)
    ldw = som.som_codebook_ldw(N)
    Wp = np.zeros((F, ldw), np.float32)
    Wp[:, :N] = W
    Wd = torch.from_numpy(Wp).to(dev)
    ip = torch.from_numpy(indptr).to(dev)
    ix = torch.from_numpy(indices).to(dev)
    norms = som.som_codebook_norms(Wd, N=N)
    perm = som.som_cluster_order(ip, ix, F) if cluster else None
    ref_b, ref_d = som.som_bmu_search(Wd, norms, ip, ix, N=N, perm=perm, **knobs)
    bmu = torch.full((B,), -7, dtype=torch.int32, device=dev)
    dist = torch.full((B,), -7.0, dtype=torch.float32, device=dev)
    o = som._opts(**knobs)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    need = lib.som_bmu_workspace_bytes(F, N, B, nnz, ctypes.byref(o))
    assert need <= som.NOALLOC_SCRATCH_BYTES
    vp = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
    st, msg = _call(lib, vp(Wd), F, N, ldw, vp(norms), vp(ip), vp(ix), B, nnz, vp(perm), vp(bmu), vp(dist),
                    ctypes.byref(o), stream)
    assert st == som.SOM_OK, msg
    torch.cuda.synchronize()
    assert torch.equal(bmu, ref_b) and torch.equal(dist, ref_d), "noalloc differs from som_bmu_search"
    b, d = bmu.cpu().numpy(), dist.cpu().numpy()
    n64 = oracle.codebook_norms(W)
    rng = np.random.default_rng(cfg * 100 + batch)
    sample = np.unique(np.concatenate([[0, B - 1], rng.choice(B, min(B, 200), replace=False)]))
    for i in sample:
        feats = indices[indptr[i]:indptr[i + 1]].astype(np.int64)
        ok, why = oracle.accept_bmu(W, n64, feats, int(b[i]), float(d[i]))
        assert ok, (int(i), why)
    print(f"[noalloc] bit-identical to som_bmu_search on {B} documents; {len(sample)} sampled documents "
          f"accepted by the oracle", flush=True)


@pytest.mark.gpu
def test_noalloc_matches_the_workspace_search_on_two_calls(lib):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    # first call: 10,000 documents of the 32^2 workload, clustered, automatic knobs
    _gpu_case(lib, 1, 0, None, 1024, 2048, True, {})
    # second call, smaller and of another shape: 1,500 Poisson(80) documents
    # against 3,000 neurons over 20,000 features, input order, 8-document tiles
    _gpu_case(lib, 2, 5, 1500, 3000, 20000, False, {"tile_docs": 8})
    # third call, kernel 3 (64-document super-tiles, a larger plan per entry)
    _gpu_case(lib, 2, 6, 4000, 2048, 20000, True, {"kernel": 3})
