"""C ABI checks that need no GPU: the library loads, exports every entry point
the header declares, and rejects bad arguments on the host before any HIP
call (so these run on a machine without a GPU)."""

import ctypes
import os
import re

import pytest

from conftest import ROOT

som = pytest.importorskip("paper_2609_05138_amd.som")

HEADER = os.path.join(ROOT, "include", "som.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(som_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(som.LIB_PATH):
        pytest.fail("libsom.so is not built (run python -m paper_2609_05138_amd.build)")
    return som.load()


def test_header_declares_the_boundary():
    names = _declared()
    for must in ("som_codebook_norms", "som_bmu_search", "som_bmu_workspace_bytes",
                 "som_tile_plan", "som_cluster_order", "som_last_error"):
        assert must in names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(som.EXPORTS)


def test_abi_version(lib):
    assert som.som_abi_version() == 15


def test_automatic_launch_follows_the_storage_type(lib):
    # som_plan resolves the automatic launch from opts->storage: kernel 3 with
    # 64-document super-tiles for fp32, kernel 1 with 8-document tiles for
    # fp16; a knob only kernel 1 has (here 16-document tiles) selects kernel 1
    B, nnz = 1 << 20, 84_000_000
    O = som.som_bmu_opts

    def plan_bytes(o, storage=0):
        o.storage = storage
        return lib.som_plan_bytes(B, nnz, ctypes.byref(o))

    p32, p16 = plan_bytes(O()), plan_bytes(O(), 1)
    assert p32 == plan_bytes(O(3, 64)) and p32 != plan_bytes(O(1, 16))
    assert p16 == plan_bytes(O(1, 8), 1) == plan_bytes(O(1, 8))
    assert plan_bytes(O(0, 16)) == plan_bytes(O(1, 16))
    assert plan_bytes(O(0, 0, 0, 4)) == plan_bytes(O(1, 16))       # group_tiles: kernel 1, 16-document tiles
    # a search that plans internally may be either storage type: its
    # workspace covers the larger automatic plan
    assert lib.som_bmu_workspace_bytes(20000, 262144, B, nnz, None) >= max(p32, p16) + 8 * B
    # the planned workspace holds keys only
    f16 = O()
    f16.storage = 1
    assert (lib.som_bmu_search_planned_workspace_bytes(262144, B, ctypes.byref(f16))
            == lib.som_bmu_search_planned_workspace_bytes(262144, B, ctypes.byref(O())))


def test_probe_rejects_bad_arguments(lib):
    fake = ctypes.c_void_p(0x1000)          # never dereferenced: rejected first
    for args in ((None, 64, 1, fake), (fake, 64, 1, None), (fake, 8, 1, fake), (fake, 40, 1, fake),
                 (ctypes.c_void_p(0x1004), 64, 1, fake), (fake, 64, 0, fake)):
        st, _ = _status(lib, "som_probe_read", *args, None)
        assert st == som.SOM_ERR_INVALID_ARG, args
    n = ctypes.c_int64(-1)
    for args in ((4, None, ctypes.byref(n)), (4, fake, None), (4, ctypes.c_void_p(0x1002), ctypes.byref(n)),
                 (0, fake, ctypes.byref(n)), (3, fake, ctypes.byref(n)), (6, fake, ctypes.byref(n)),
                 (-4, fake, ctypes.byref(n)), ((1 << 24) + 4, fake, ctypes.byref(n))):
        st, _ = _status(lib, "som_probe_lds", *args, None)
        assert st == som.SOM_ERR_INVALID_ARG, args
    assert n.value == -1                    # nothing written on a rejected call


def test_codebook_ldw_is_host_only(lib):
    # the recommended stride is 256-byte aligned, never below N, and never a
    # multiple of 2 KB (so row slices rotate over the L2 channels)
    for N, want in ((262144, 262208), (65536, 65600), (16384, 16448), (1024, 1088), (512, 576),
                    (3, 64), (64, 64), (100, 128), (1000, 1088), (1100, 1152), (1 << 30, (1 << 30) + 64)):
        got = som.som_codebook_ldw(N)
        assert got == want, (N, got)
        assert got >= N and got % 64 == 0 and (4 * got) % 2048 != 0
    assert som.som_codebook_ldw(0) == 0 and som.som_codebook_ldw(-5) == 0


def test_workspace_sizes_are_host_only(lib):
    for kernel in (0, 1, 2, 3):
        o = som.som_bmu_opts(kernel)
        a = lib.som_bmu_workspace_bytes(20000, 262144, 1 << 20, 84_000_000, ctypes.byref(o))
        assert a > 0 and a % 256 == 0
        # the plan (two int32 per nonzero) dominates; one packed key per document
        assert a >= 8 * 84_000_000 + 8 * (1 << 20)
        assert lib.som_plan_bytes(1 << 20, 84_000_000, ctypes.byref(o)) >= 8 * 84_000_000
        assert lib.som_bmu_search_planned_workspace_bytes(262144, 1 << 20, ctypes.byref(o)) >= 8 * (1 << 20)
        v = som.som_bmu_opts(kernel)
        v.validate = 1
        b = lib.som_bmu_workspace_bytes(20000, 262144, 1 << 20, 84_000_000, ctypes.byref(v))
        assert b > a                   # validation needs a scratch array
    # kernel 3 (64-document super-tiles by default): two mask words per entry,
    # plus a padding of 256 entries after the features and the masks
    o = som.som_bmu_opts(3)
    assert lib.som_plan_bytes(1 << 20, 84_000_000, ctypes.byref(o)) >= (4 + 8) * (84_000_000 + 256)
    o = som.som_bmu_opts(3, 256)
    assert lib.som_plan_bytes(1 << 20, 84_000_000, ctypes.byref(o)) >= (4 + 32) * (84_000_000 + 256)
    assert lib.som_bmu_workspace_bytes(0, 10, 10, 10, None) == 0
    assert lib.som_bmu_workspace_bytes(10, 10, -1, 10, None) == 0
    bad = som.som_bmu_opts(4)
    assert lib.som_bmu_workspace_bytes(10, 10, 10, 10, ctypes.byref(bad)) == 0


def _status(lib, fn, *args):
    st = getattr(lib, fn)(*args)
    return st, lib.som_last_error().decode()


def test_norms_rejects_bad_arguments(lib):
    null = None
    fake = ctypes.c_void_p(0x1000)            # never dereferenced: rejected first
    mis = ctypes.c_void_p(0x1004)
    assert _status(lib, "som_codebook_norms", null, 4, 4, 4, fake, null)[0] == som.SOM_ERR_INVALID_ARG
    assert _status(lib, "som_codebook_norms", fake, 0, 4, 4, fake, null)[0] == som.SOM_ERR_INVALID_ARG
    assert _status(lib, "som_codebook_norms", fake, 4, 0, 4, fake, null)[0] == som.SOM_ERR_INVALID_ARG
    st, msg = _status(lib, "som_codebook_norms", fake, 4, 8, 4, fake, null)
    assert st == som.SOM_ERR_INVALID_ARG and "ldw" in msg
    assert _status(lib, "som_codebook_norms", fake, 4, 5, 6, fake, null)[0] == som.SOM_ERR_INVALID_ARG
    st, msg = _status(lib, "som_codebook_norms", mis, 4, 4, 4, fake, null)
    assert st == som.SOM_ERR_INVALID_ARG and "aligned" in msg
    assert _status(lib, "som_codebook_norms", fake, 4, 4, 4, null, null)[0] == som.SOM_ERR_INVALID_ARG


def test_search_rejects_bad_arguments(lib):
    null = None
    fake = ctypes.c_void_p(0x1000)
    ws_bad = ctypes.c_void_p(0x1010)
    o = som.som_bmu_opts()
    args = dict(W=fake, F=8, N=8, ldw=8, norms=fake, indptr=fake, indices=fake, B=4, nnz=10,
                perm=null, bmu=fake, dist=fake, opts=ctypes.byref(o), ws=fake, ws_bytes=1 << 30,
                stream=null)

    def call(**kw):
        a = dict(args, **kw)
        return _status(lib, "som_bmu_search", *a.values())

    assert call(W=null)[0] == som.SOM_ERR_INVALID_ARG
    assert call(norms=null)[0] == som.SOM_ERR_INVALID_ARG
    assert call(indptr=null)[0] == som.SOM_ERR_INVALID_ARG
    assert call(indices=null)[0] == som.SOM_ERR_INVALID_ARG
    assert call(bmu=null)[0] == som.SOM_ERR_INVALID_ARG
    assert call(B=-1)[0] == som.SOM_ERR_INVALID_ARG
    assert call(nnz=-1)[0] == som.SOM_ERR_INVALID_ARG
    assert call(ldw=6)[0] == som.SOM_ERR_INVALID_ARG
    assert call(F=1 << 30, ldw=1 << 40)[0] == som.SOM_ERR_INVALID_ARG   # F * ldw beyond 64-bit byte offsets
    st, msg = call(ws_bytes=16)
    assert st == som.SOM_ERR_WORKSPACE and "need" in msg
    assert call(ws=null)[0] == som.SOM_ERR_WORKSPACE
    assert call(ws=ws_bad)[0] == som.SOM_ERR_INVALID_ARG
    res = som.som_bmu_opts()
    res.storage = 2
    O = som.som_bmu_opts
    for bad in (O(4), O(-1), O(3, 32), O(3, 16), O(3, 0, 8), O(3, 0, 0, 2), O(3, 0, 0, 0, 3), O(3, 0, 0, 0, 0, 32),
                O(1, 5), O(1, 0, 3), res, O(1, 0, 0, 16), O(1, 0, 0, 0, 3), O(1, 32, 8),
                O(0, 0, 0, 0, 0, 0, 2), O(1, 0, 0, -1), O(2, 8), O(2, 0, 4), O(2, 0, 0, 1),
                O(2, 0, 0, 0, 1), O(2, 0, 0, 0, 0, 48), O(1, 0, 0, 0, 0, 32),
                O(0, 0, 0, 0, 0, 0, 0, 0, 3), O(1, 0, 0, 0, 0, 0, 0, 0, 2), O(3, 0, 0, 0, 0, 0, 0, 0, -1),
                # neuron_chunk: a multiple of the slice width, kernels 1 and 3, one launch
                O(1, 0, 0, 0, 0, 0, 0, 0, 0, 100), O(3, 0, 0, 0, 0, 0, 0, 0, 0, -256),
                O(2, 0, 0, 0, 0, 0, 0, 0, 0, 256), O(3, 0, 0, 0, 0, 0, 0, 0, 2, 256),
                O(1, 0, 8, 0, 0, 0, 0, 0, 0, 256),
                # sweep: 0, 1 or 2; the rotated sweep needs kernel 1 or kernel 3's
                # document-major form as one launch of one-slice chunks
                O(0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 3), O(3, 0, 0, 0, 0, 0, 0, 0, 0, 0, -1),
                O(2, 0, 0, 0, 0, 0, 0, 0, 0, 0, 2),
                O(3, 0, 0, 0, 1, 0, 0, 0, 0, 0, 2), O(3, 0, 0, 0, 0, 0, 0, 0, 2, 0, 2)):
        st, msg = call(opts=ctypes.byref(bad))
        assert st == som.SOM_ERR_INVALID_ARG, msg
    # rotated sweeps with chunks of two slices (the map has four)
    for k in (1, 3):
        st, msg = call(opts=ctypes.byref(O(k, 0, 4, 0, 0, 0, 0, 0, 0, 512, 2)), N=1024, ldw=1024)
        assert st == som.SOM_ERR_INVALID_ARG and "sweep" in msg, (k, msg)
    # a chunk wider than the map covers it whole
    assert call(opts=ctypes.byref(O(1, 0, 0, 0, 0, 0, 0, 0, 0, 1 << 20)), ws=fake, B=0, nnz=0, indices=null,
                bmu=null, dist=null)[0] == som.SOM_OK
    # the rotated sweep with one-slice chunks, the ascending sweep anywhere
    for good in (O(0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 2), O(3, 128, 0, 0, 2, 0, 0, 0, 1, 256, 2),
                 O(1, 0, 0, 0, 0, 0, 0, 0, 0, 0, 2), O(1, 4, 0, 2, 1, 0, 0, 0, 0, 256, 2),
                 O(2, 0, 0, 0, 0, 0, 0, 0, 0, 0, 1), O(3, 0, 0, 0, 1, 0, 0, 0, 2, 0, 1)):
        assert call(opts=ctypes.byref(good), ws=fake, B=0, nnz=0, indices=null, bmu=null,
                    dist=null)[0] == som.SOM_OK
    # an empty batch is a valid no-op that touches nothing
    assert call(B=0, nnz=0, indices=null, bmu=null, dist=null, ws=null, ws_bytes=0)[0] == som.SOM_OK
    assert lib.som_last_error().decode() == ""


def test_top2_rejects_bad_arguments(lib):
    null = None
    fake = ctypes.c_void_p(0x1000)
    o = som.som_bmu_opts()
    args = dict(W=fake, F=8, N=8, ldw=8, norms=fake, indptr=fake, indices=fake, B=4, nnz=10,
                perm=null, bmu=fake, dist=fake, bmu2=fake, dist2=fake, opts=ctypes.byref(o), ws=fake,
                ws_bytes=1 << 30, stream=null)

    def call(**kw):
        a = dict(args, **kw)
        return _status(lib, "som_bmu_search_top2", *a.values())

    for k in ("bmu", "dist", "bmu2", "dist2", "W", "norms"):
        st, msg = call(**{k: null})
        assert st == som.SOM_ERR_INVALID_ARG, (k, msg)
    st, msg = call(ws_bytes=16)
    assert st == som.SOM_ERR_WORKSPACE and "need" in msg
    assert call(B=0, nnz=0, indices=null, bmu=null, dist=null, bmu2=null, dist2=null, ws=null,
                ws_bytes=0)[0] == som.SOM_OK
    big = 1 << 30
    # W, F, N, ldw, norms, indptr, B, nnz, perm, plan, plan_bytes, bmu, dist, bmu2, dist2, opts, ws, ws_bytes, stream
    st, msg = _status(lib, "som_bmu_search_top2_planned", fake, 8, 8, 8, fake, fake, 4, 10, null, fake, big,
                      fake, fake, null, fake, ctypes.byref(o), fake, big, null)
    assert st == som.SOM_ERR_INVALID_ARG and "bmu2" in msg
    st, _ = _status(lib, "som_bmu_search_top2_planned", fake, 8, 8, 8, fake, fake, 4, 10, null, fake, big,
                    fake, fake, fake, fake, ctypes.byref(o), fake, 8, null)
    assert st == som.SOM_ERR_WORKSPACE
    # the planned workspace holds both key arrays: 16 B per document
    assert lib.som_bmu_search_planned_workspace_bytes(1024, 1000, ctypes.byref(o)) >= 16 * 1000


def test_f16_rejects_bad_arguments(lib):
    null = None
    fake = ctypes.c_void_p(0x1000)
    O = som.som_bmu_opts

    def call(ldw=16, opts=None, **kw):
        o = opts if opts is not None else O()
        return _status(lib, "som_bmu_search_f16", fake, 8, 12, ldw, fake, fake, fake, 4, 10, null, fake, fake,
                       ctypes.byref(o), fake, 1 << 30, null)

    st, msg = call(ldw=12)                    # fine for fp32, not for fp16 (8 halves per load)
    assert st == som.SOM_ERR_INVALID_ARG and "multiple of 8" in msg
    for bad in (O(2), O(1, 0, 4), O(1, 32), O(1, 32, 4), O(3, 256), O(3, 0, 4)):
        st, msg = call(opts=bad)
        assert st == som.SOM_ERR_INVALID_ARG, msg
    st, msg = _status(lib, "som_codebook_norms_f16", fake, 8, 12, 12, fake, null)
    assert st == som.SOM_ERR_INVALID_ARG and "multiple of 8" in msg
    st, _ = _status(lib, "som_codebook_norms_f16", null, 8, 8, 8, fake, null)
    assert st == som.SOM_ERR_INVALID_ARG


def test_update_rejects_bad_arguments(lib):
    null = None
    fake = ctypes.c_void_p(0x1000)
    # indptr, indices, B, nnz, bmu, F, N, acc, ld_acc, count, stream
    assert _status(lib, "som_update_accumulate", fake, fake, 4, 10, fake, 8, 16, fake, 15, fake, null)[0] \
        == som.SOM_ERR_INVALID_ARG                                          # ld_acc < N
    assert _status(lib, "som_update_accumulate", fake, fake, 4, 10, null, 8, 16, fake, 16, fake, null)[0] \
        == som.SOM_ERR_INVALID_ARG
    assert _status(lib, "som_update_accumulate", null, null, 0, 0, null, 8, 16, null, 16, null, null)[0] == som.SOM_OK
    ws = lib.som_update_workspace_bytes(20000, 262144)
    assert ws >= 4 * ((1 << 26) + 2 * 262144) and ws % 256 == 0
    assert lib.som_update_workspace_bytes(0, 10) == 0

    def fin(rows=4, cols=4, sigma=1.0, ldw=16, ld_acc=16, ws=fake, ws_bytes=1 << 40, W=fake):
        return _status(lib, "som_update_finish", W, 8, ldw, rows, cols, sigma, fake, ld_acc, fake, ws, ws_bytes, null)

    for kw in (dict(rows=0), dict(cols=0), dict(rows=1025), dict(cols=16385), dict(sigma=-1.0),
               dict(sigma=float("nan")), dict(sigma=float("inf")), dict(sigma=2000.0), dict(ldw=15),
               dict(ld_acc=15), dict(W=null)):
        st, msg = fin(**kw)
        assert st == som.SOM_ERR_INVALID_ARG, (kw, msg)
    assert fin(ws=null)[0] == som.SOM_ERR_WORKSPACE
    assert fin(ws_bytes=64)[0] == som.SOM_ERR_WORKSPACE


def test_unfused_rejects_bad_arguments(lib):
    null = None
    fake = ctypes.c_void_p(0x1000)
    O = som.som_bmu_opts

    def call(opts=None, block=64, ws_bytes=1 << 40):
        o = opts if opts is not None else O()
        return _status(lib, "som_bmu_search_unfused", fake, 8, 8, 8, fake, fake, fake, 4, 10, null, fake, fake,
                       ctypes.byref(o), block, fake, ws_bytes, null)

    for bad in (dict(opts=O(2)), dict(opts=O(3)), dict(block=0), dict(block=12), dict(block=-8),
                dict(opts=O(1, 0, 0, 0, 0, 0, 0, 0, 0, 0, 2))):   # the comparator sweeps in ascending order
        st, msg = call(**bad)
        assert st == som.SOM_ERR_INVALID_ARG, (bad, msg)
    assert call(ws_bytes=64)[0] == som.SOM_ERR_WORKSPACE
    o = O()
    need = lib.som_bmu_search_unfused_workspace_bytes(20000, 262144, 1 << 20, 84_000_000, ctypes.byref(o), 8192)
    assert need >= 4 * 8192 * 262144
    assert lib.som_bmu_search_unfused_workspace_bytes(20000, 262144, 1 << 20, 84_000_000, ctypes.byref(o), 12) == 0


def test_plan_and_cluster_reject_bad_arguments(lib):
    null = None
    fake = ctypes.c_void_p(0x1000)
    st, msg = _status(lib, "som_tile_plan", fake, fake, 4, 8, 10, null, 3, fake, fake, fake, fake, null)
    assert st == som.SOM_ERR_INVALID_ARG and "tile_docs" in msg
    st, _ = _status(lib, "som_tile_plan", fake, fake, 4, 0, 10, null, 4, fake, fake, fake, fake, null)
    assert st == som.SOM_ERR_INVALID_ARG
    st, _ = _status(lib, "som_tile_plan", fake, fake, 4, 8, 10, null, 4, null, fake, fake, fake, null)
    assert st == som.SOM_ERR_INVALID_ARG
    st, msg = _status(lib, "som_group_plan", fake, fake, 4, 8, 10, null, 0, fake, fake, fake, fake, null)
    assert st == som.SOM_ERR_INVALID_ARG and "group_docs" in msg
    o = som.som_bmu_opts()
    assert lib.som_bmu_search_planned_workspace_bytes(1024, 100, ctypes.byref(o)) >= 8 * 100
    big = 1 << 30
    # W, F, N, ldw, norms, indptr, B, nnz, perm, plan, plan_bytes, bmu, dist, opts, ws, ws_bytes, stream
    st, _ = _status(lib, "som_bmu_search_planned", fake, 8, 8, 8, fake, fake, 4, 10, null, fake, big,
                    fake, fake, ctypes.byref(o), fake, 4, null)
    assert st == som.SOM_ERR_WORKSPACE
    st, _ = _status(lib, "som_bmu_search_planned", fake, 8, 8, 8, fake, fake, 4, 10, null, null, big,
                    fake, fake, ctypes.byref(o), fake, big, null)
    assert st == som.SOM_ERR_INVALID_ARG
    st, msg = _status(lib, "som_bmu_search_planned", fake, 8, 8, 8, fake, fake, 4, 10, null, fake, 16,
                      fake, fake, ctypes.byref(o), fake, big, null)
    assert st == som.SOM_ERR_INVALID_ARG and "plan" in msg
    v = som.som_bmu_opts()
    v.validate = 1
    st, _ = _status(lib, "som_bmu_search_planned", fake, 8, 8, 8, fake, fake, 4, 10, null, fake, big,
                    fake, fake, ctypes.byref(v), fake, big, null)
    assert st == som.SOM_ERR_INVALID_ARG
    st, _ = _status(lib, "som_plan", fake, fake, 4, 8, 10, null, ctypes.byref(o), fake, 16, null)
    assert st == som.SOM_ERR_WORKSPACE
    st, _ = _status(lib, "som_cluster_order", fake, fake, 4, 8, 10, null, fake, 1 << 20, null)
    assert st == som.SOM_ERR_INVALID_ARG
    st, _ = _status(lib, "som_cluster_order", fake, fake, 4, 8, 10, fake, null, 1 << 20, null)
    assert st == som.SOM_ERR_WORKSPACE
    assert _status(lib, "som_cluster_order", null, null, 0, 8, 0, null, null, 0, null)[0] == som.SOM_OK


def test_binding_refuses_cpu_tensors(lib):
    import torch
    W = torch.zeros(4, 4)
    with pytest.raises(ValueError):
        som.som_codebook_norms(W)
