"""Thin ctypes binding of libsom (include/som.h) for torch device tensors.

Argument marshalling only: every step of the search runs in the HIP
library.  There is no CPU path: if the library is not built, or a tensor is
not on a ROCm device, calls raise.  Function names match the C entry points.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch  # imported before the library so both share one HIP runtime

_PKG = os.path.dirname(os.path.abspath(__file__))
# SOM_LIBRARY names another build of the same library (the host-sanitized
# one, for CPU-side checks); it must exist like the default one
LIB_PATH = os.environ.get("SOM_LIBRARY") or os.path.join(_PKG, "libsom.so")

SOM_OK = 0
SOM_ERR_INVALID_ARG = 1
SOM_ERR_INVALID_CSR = 2
SOM_ERR_WORKSPACE = 3
SOM_ERR_HIP = 4

EXPORTS = (
    "som_abi_version",
    "som_last_error",
    "som_codebook_norms",
    "som_codebook_ldw",
    "som_bmu_workspace_bytes",
    "som_bmu_search",
    "som_bmu_search_top2",
    "som_bmu_search_noalloc",
    "som_plan_bytes",
    "som_plan",
    "som_bmu_search_planned_workspace_bytes",
    "som_bmu_search_planned",
    "som_bmu_search_top2_planned",
    "som_tile_plan",
    "som_group_plan",
    "som_cluster_workspace_bytes",
    "som_cluster_order",
    "som_codebook_norms_f16",
    "som_bmu_search_f16",
    "som_bmu_search_top2_f16",
    "som_bmu_search_planned_f16",
    "som_bmu_search_top2_planned_f16",
    "som_bmu_search_unfused_workspace_bytes",
    "som_bmu_search_unfused",
    "som_update_accumulate",
    "som_update_workspace_bytes",
    "som_update_finish",
    "som_update_finish_f16",
    "som_probe_read",
    "som_probe_lds",
)


class SomError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libsom status {status}: {msg}")
        self.status = status


class som_bmu_opts(ctypes.Structure):
    _fields_ = [
        ("kernel", ctypes.c_int32),
        ("tile_docs", ctypes.c_int32),
        ("lane_neurons", ctypes.c_int32),
        ("group_tiles", ctypes.c_int32),
        ("mask_mode", ctypes.c_int32),
        ("slice_neurons", ctypes.c_int32),
        ("validate", ctypes.c_int32),
        ("storage", ctypes.c_int32),
        ("schedule", ctypes.c_int32),
        ("neuron_chunk", ctypes.c_int32),
        ("sweep", ctypes.c_int32),
    ]


_lib = None

_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_vp = ctypes.c_void_p
_sz = ctypes.c_size_t


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libsom.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is missing: build it with `python -m paper_2609_05138_amd.build` "
            "(there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    lib.som_abi_version.restype = _i32
    lib.som_abi_version.argtypes = []
    lib.som_last_error.restype = ctypes.c_char_p
    lib.som_last_error.argtypes = []
    lib.som_codebook_norms.restype = _i32
    lib.som_codebook_norms.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp]
    lib.som_codebook_ldw.restype = _i64
    lib.som_codebook_ldw.argtypes = [_i64]
    lib.som_bmu_workspace_bytes.restype = _sz
    lib.som_bmu_workspace_bytes.argtypes = [_i64, _i64, _i64, _i64, ctypes.POINTER(som_bmu_opts)]
    lib.som_bmu_search.restype = _i32
    lib.som_bmu_search.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _vp,
                                   ctypes.POINTER(som_bmu_opts), _vp, _sz, _vp]
    lib.som_bmu_search_noalloc.restype = _i32
    lib.som_bmu_search_noalloc.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _vp,
                                           ctypes.POINTER(som_bmu_opts), _vp]
    lib.som_plan_bytes.restype = _sz
    lib.som_plan_bytes.argtypes = [_i64, _i64, ctypes.POINTER(som_bmu_opts)]
    lib.som_plan.restype = _i32
    lib.som_plan.argtypes = [_vp, _vp, _i64, _i64, _i64, _vp, ctypes.POINTER(som_bmu_opts), _vp, _sz, _vp]
    lib.som_bmu_search_planned_workspace_bytes.restype = _sz
    lib.som_bmu_search_planned_workspace_bytes.argtypes = [_i64, _i64, ctypes.POINTER(som_bmu_opts)]
    lib.som_bmu_search_top2.restype = _i32
    lib.som_bmu_search_top2.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _vp, _vp, _vp,
                                        ctypes.POINTER(som_bmu_opts), _vp, _sz, _vp]
    lib.som_bmu_search_top2_planned.restype = _i32
    lib.som_bmu_search_top2_planned.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp, _i64, _i64, _vp, _vp, _sz,
                                                _vp, _vp, _vp, _vp, ctypes.POINTER(som_bmu_opts), _vp, _sz, _vp]
    lib.som_bmu_search_planned.restype = _i32
    lib.som_bmu_search_planned.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp, _i64, _i64, _vp, _vp, _sz,
                                           _vp, _vp, ctypes.POINTER(som_bmu_opts), _vp, _sz, _vp]
    lib.som_tile_plan.restype = _i32
    lib.som_tile_plan.argtypes = [_vp, _vp, _i64, _i64, _i64, _vp, _i32, _vp, _vp, _vp, _vp, _vp]
    lib.som_group_plan.restype = _i32
    lib.som_group_plan.argtypes = [_vp, _vp, _i64, _i64, _i64, _vp, _i32, _vp, _vp, _vp, _vp, _vp]
    lib.som_cluster_workspace_bytes.restype = _sz
    lib.som_cluster_workspace_bytes.argtypes = [_i64, _i64, _i64]
    # the fp16 functions take the same arguments (W as binary16 bit patterns)
    for base in ("som_codebook_norms", "som_bmu_search", "som_bmu_search_top2", "som_bmu_search_planned",
                 "som_bmu_search_top2_planned"):
        fn = getattr(lib, base + "_f16")
        fn.restype = _i32
        fn.argtypes = getattr(lib, base).argtypes
    lib.som_bmu_search_unfused_workspace_bytes.restype = _sz
    lib.som_bmu_search_unfused_workspace_bytes.argtypes = [_i64, _i64, _i64, _i64, ctypes.POINTER(som_bmu_opts), _i64]
    lib.som_bmu_search_unfused.restype = _i32
    lib.som_bmu_search_unfused.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _vp,
                                           ctypes.POINTER(som_bmu_opts), _i64, _vp, _sz, _vp]
    lib.som_update_accumulate.restype = _i32
    lib.som_update_accumulate.argtypes = [_vp, _vp, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _vp, _vp]
    lib.som_update_workspace_bytes.restype = _sz
    lib.som_update_workspace_bytes.argtypes = [_i64, _i64]
    for fn in (lib.som_update_finish, lib.som_update_finish_f16):
        fn.restype = _i32
        fn.argtypes = [_vp, _i64, _i64, _i32, _i32, ctypes.c_double, _vp, _i64, _vp, _vp, _sz, _vp]
    lib.som_probe_read.restype = _i32
    lib.som_probe_read.argtypes = [_vp, _i64, _i32, _vp, _vp]
    lib.som_probe_lds.restype = _i32
    lib.som_probe_lds.argtypes = [_i32, _vp, ctypes.POINTER(ctypes.c_int64), _vp]
    lib.som_cluster_order.restype = _i32
    lib.som_cluster_order.argtypes = [_vp, _vp, _i64, _i64, _i64, _vp, _vp, _sz, _vp]
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != SOM_OK:
        raise SomError(status, load().som_last_error().decode(errors="replace"))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, dtype, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a ROCm device (got {t.device})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _codebook(W: torch.Tensor) -> str:
    """Check the codebook tensor; return the C function suffix for its dtype."""
    if isinstance(W, torch.Tensor) and W.dtype == torch.float16:
        _dev(W, torch.float16, "W")
        return "_f16"
    _dev(W, torch.float32, "W")
    return ""


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _opts(kernel=0, tile_docs=0, lane_neurons=0, group_tiles=0, mask_mode=0, slice_neurons=0,
          validate=False, storage=0, schedule=0, neuron_chunk=0, sweep=0) -> som_bmu_opts:
    return som_bmu_opts(int(kernel), int(tile_docs), int(lane_neurons), int(group_tiles), int(mask_mode),
                        int(slice_neurons), int(bool(validate)), int(storage), int(schedule), int(neuron_chunk),
                        int(sweep))


def _n_neurons(N, norms, W) -> int:
    """N of a search: explicit, else the length of the norms vector.

    The codebook's second dimension is its row stride, which may exceed N
    (padding to the recommended stride); its padding columns are not
    neurons, so they are never the default."""
    if N is not None:
        return int(N)
    return int(norms.numel())


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns 256-byte (or better) aligned blocks
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def som_abi_version() -> int:
    return int(load().som_abi_version())


def som_last_error() -> str:
    return load().som_last_error().decode(errors="replace")


def som_codebook_ldw(N: int) -> int:
    """Recommended row stride (floats) of a feature-major codebook of N neurons."""
    return int(load().som_codebook_ldw(int(N)))


def som_codebook_norms(W: torch.Tensor, N: Optional[int] = None, norms: Optional[torch.Tensor] = None,
                       stream=None) -> torch.Tensor:
    """||w_j||^2 for j < N of the feature-major codebook W [F, ldw] (fp32 or fp16).

    N defaults to the length of ``norms`` when it is given, else to ldw (a
    codebook padded beyond N needs N)."""
    lib = load()
    sfx = _codebook(W)
    F, ldw = W.shape
    n = int(N) if N is not None else (int(norms.numel()) if norms is not None else ldw)
    if norms is None:
        norms = torch.empty(n, dtype=torch.float32, device=W.device)
    _dev(norms, torch.float32, "norms")
    if norms.numel() < n:
        raise ValueError("norms is too small")
    _check(getattr(lib, "som_codebook_norms" + sfx)(_ptr(W), F, n, ldw, _ptr(norms), _stream(stream)))
    return norms


def som_bmu_workspace_bytes(F: int, N: int, B: int, nnz: int, validate=False, **knobs) -> int:
    o = _opts(validate=validate, **knobs)
    return int(load().som_bmu_workspace_bytes(F, N, B, nnz, ctypes.byref(o)))


def _outputs(B, device, pairs):
    out = []
    for t, dtype, name in pairs:
        if t is None:
            t = torch.empty(B, dtype=dtype, device=device)
        _dev(t, dtype, name)
        if t.numel() < B:
            raise ValueError(f"{name} is too small")
        out.append(t)
    return out


def _search(top2, W, norms, indptr, indices, N, perm, validate, outs, ws, stream, knobs):
    lib = load()
    sfx = _codebook(W)
    _dev(norms, torch.float32, "norms")
    _dev(indptr, torch.int32, "indptr")
    _dev(indices, torch.int32, "indices")
    F, ldw = W.shape
    n = _n_neurons(N, norms, W)
    if norms.numel() < n:
        raise ValueError("norms must hold at least N values")
    B = indptr.numel() - 1
    nnz = indices.numel()
    if perm is not None:
        _dev(perm, torch.int32, "perm")
        if perm.numel() != B:
            raise ValueError("perm must have B entries")
    names = (("bmu", torch.int32), ("dist", torch.float32), ("bmu2", torch.int32), ("dist2", torch.float32))
    outs = _outputs(B, W.device, [(t, dt, nm) for t, (nm, dt) in zip(outs, names)])
    o = _opts(validate=validate, **knobs)
    need = int(lib.som_bmu_workspace_bytes(F, n, B, nnz, ctypes.byref(o)))
    if ws is None:
        ws = _workspace(need, W.device)
    _dev(ws, torch.uint8, "ws")
    common = (_ptr(W), F, n, ldw, _ptr(norms), _ptr(indptr), _ptr(indices), B, nnz, _ptr(perm))
    tail = (ctypes.byref(o), _ptr(ws), ws.numel(), _stream(stream))
    if top2:
        _check(getattr(lib, "som_bmu_search_top2" + sfx)(*common, *(_ptr(t) for t in outs), *tail))
    else:
        _check(getattr(lib, "som_bmu_search" + sfx)(*common, *(_ptr(t) for t in outs), *tail))
    return tuple(outs)


def som_bmu_search(W: torch.Tensor, norms: torch.Tensor, indptr: torch.Tensor, indices: torch.Tensor,
                   N: Optional[int] = None, perm: Optional[torch.Tensor] = None, validate: bool = False,
                   bmu: Optional[torch.Tensor] = None, dist: Optional[torch.Tensor] = None,
                   ws: Optional[torch.Tensor] = None, stream=None, **knobs) -> Tuple[torch.Tensor, torch.Tensor]:
    """BMU index (int32) and squared distance (fp32) of every CSR document.

    ``N`` defaults to the length of ``norms``.  ``knobs``: kernel, tile_docs,
    lane_neurons, group_tiles, mask_mode, slice_neurons, schedule,
    neuron_chunk, sweep (fields of som_bmu_opts; only sweep changes a
    result, in rounding: 1 = ascending feature order, 2 = rotated, the
    kernel-3 default)."""
    return _search(False, W, norms, indptr, indices, N, perm, validate, (bmu, dist), ws, stream, knobs)


def som_bmu_search_top2(W: torch.Tensor, norms: torch.Tensor, indptr: torch.Tensor, indices: torch.Tensor,
                        N: Optional[int] = None, perm: Optional[torch.Tensor] = None, validate: bool = False,
                        bmu: Optional[torch.Tensor] = None, dist: Optional[torch.Tensor] = None,
                        bmu2: Optional[torch.Tensor] = None, dist2: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None, stream=None, **knobs):
    """(bmu, dist, bmu2, dist2): best and second-best unit of every document
    (bmu2 = -1 and dist2 = +inf when N == 1)."""
    return _search(True, W, norms, indptr, indices, N, perm, validate, (bmu, dist, bmu2, dist2), ws, stream,
                   knobs)


NOALLOC_SCRATCH_BYTES = 64 << 20


def som_bmu_search_noalloc(W: torch.Tensor, norms: torch.Tensor, indptr: torch.Tensor, indices: torch.Tensor,
                           N: Optional[int] = None, perm: Optional[torch.Tensor] = None,
                           bmu: Optional[torch.Tensor] = None, dist: Optional[torch.Tensor] = None, stream=None,
                           **knobs) -> Tuple[torch.Tensor, torch.Tensor]:
    """som_bmu_search whose workspace is the library's static device array
    (no allocation by the library; fp32 codebook; bmu and dist are allocated
    here only when not given)."""
    lib = load()
    _dev(W, torch.float32, "W")
    _dev(norms, torch.float32, "norms")
    _dev(indptr, torch.int32, "indptr")
    _dev(indices, torch.int32, "indices")
    F, ldw = W.shape
    n = _n_neurons(N, norms, W)
    if norms.numel() < n:
        raise ValueError("norms must hold at least N values")
    B = indptr.numel() - 1
    if perm is not None:
        _dev(perm, torch.int32, "perm")
        if perm.numel() != B:
            raise ValueError("perm must have B entries")
    bmu, dist = _outputs(B, W.device, [(bmu, torch.int32, "bmu"), (dist, torch.float32, "dist")])
    o = _opts(**knobs)
    _check(lib.som_bmu_search_noalloc(_ptr(W), F, n, ldw, _ptr(norms), _ptr(indptr), _ptr(indices), B,
                                      indices.numel(), _ptr(perm), _ptr(bmu), _ptr(dist), ctypes.byref(o),
                                      _stream(stream)))
    return bmu, dist


class Plan:
    """An opaque search plan (device buffer) and how it was built."""

    def __init__(self, buf, knobs, B, nnz, perm):
        self.buf = buf
        self.knobs = dict(knobs)
        self.B = B
        self.nnz = nnz
        self.perm = perm


def som_plan(indptr: torch.Tensor, indices: torch.Tensor, F: int, perm: Optional[torch.Tensor] = None,
             plan: Optional[torch.Tensor] = None, stream=None, **knobs) -> Plan:
    """Plan of a batch for som_bmu_search_planned (codebook-independent).

    ``knobs`` as for som_bmu_search, plus ``storage`` (0 = fp32, 1 = fp16):
    the storage type whose automatic tile size the plan takes; the planned
    search resolves the same geometry from the plan's knobs, whatever the
    codebook it is given."""
    lib = load()
    _dev(indptr, torch.int32, "indptr")
    _dev(indices, torch.int32, "indices")
    B = indptr.numel() - 1
    nnz = indices.numel()
    if perm is not None:
        _dev(perm, torch.int32, "perm")
    o = _opts(**knobs)
    need = int(lib.som_plan_bytes(B, nnz, ctypes.byref(o)))
    if plan is None:
        plan = _workspace(need, indptr.device)
    _dev(plan, torch.uint8, "plan")
    _check(lib.som_plan(_ptr(indptr), _ptr(indices), B, F, nnz, _ptr(perm), ctypes.byref(o), _ptr(plan),
                        plan.numel(), _stream(stream)))
    return Plan(plan, knobs, B, nnz, perm)


def som_bmu_search_planned_workspace_bytes(N: int, B: int, **knobs) -> int:
    o = _opts(**knobs)
    return int(load().som_bmu_search_planned_workspace_bytes(N, B, ctypes.byref(o)))


def _planned(top2, W, norms, indptr, plan, N, outs, ws, stream):
    lib = load()
    sfx = _codebook(W)
    _dev(norms, torch.float32, "norms")
    _dev(indptr, torch.int32, "indptr")
    F, ldw = W.shape
    n = _n_neurons(N, norms, W)
    if norms.numel() < n:
        raise ValueError("norms must hold at least N values")
    B = indptr.numel() - 1
    if B != plan.B:
        raise ValueError("plan was built for another batch")
    names = (("bmu", torch.int32), ("dist", torch.float32), ("bmu2", torch.int32), ("dist2", torch.float32))
    outs = _outputs(B, W.device, [(t, dt, nm) for t, (nm, dt) in zip(outs, names)])
    o = _opts(**plan.knobs)
    if ws is None:
        ws = _workspace(lib.som_bmu_search_planned_workspace_bytes(n, B, ctypes.byref(o)), W.device)
    _dev(ws, torch.uint8, "ws")
    common = (_ptr(W), F, n, ldw, _ptr(norms), _ptr(indptr), B, plan.nnz, _ptr(plan.perm), _ptr(plan.buf),
              plan.buf.numel())
    tail = (ctypes.byref(o), _ptr(ws), ws.numel(), _stream(stream))
    if top2:
        _check(getattr(lib, "som_bmu_search_top2_planned" + sfx)(*common, *(_ptr(t) for t in outs), *tail))
    else:
        _check(getattr(lib, "som_bmu_search_planned" + sfx)(*common, *(_ptr(t) for t in outs), *tail))
    return tuple(outs)


def som_bmu_search_planned(W: torch.Tensor, norms: torch.Tensor, indptr: torch.Tensor, plan: Plan,
                           N: Optional[int] = None, bmu: Optional[torch.Tensor] = None,
                           dist: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                           stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """The search stage on a prebuilt plan (same indptr, perm and knobs)."""
    return _planned(False, W, norms, indptr, plan, N, (bmu, dist), ws, stream)


def som_bmu_search_top2_planned(W: torch.Tensor, norms: torch.Tensor, indptr: torch.Tensor, plan: Plan,
                                N: Optional[int] = None, bmu: Optional[torch.Tensor] = None,
                                dist: Optional[torch.Tensor] = None, bmu2: Optional[torch.Tensor] = None,
                                dist2: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                                stream=None):
    """Top-2 search stage on a prebuilt plan: (bmu, dist, bmu2, dist2)."""
    return _planned(True, W, norms, indptr, plan, N, (bmu, dist, bmu2, dist2), ws, stream)


def som_tile_plan(indptr: torch.Tensor, indices: torch.Tensor, F: int, tile_docs: int = 8,
                  perm: Optional[torch.Tensor] = None, stream=None):
    """Tile plan as explicit arrays: (tile_offset, tile_count, union_feat, union_mask).

    union_mask is int32 [nnz] for tile_docs <= 32, else [nnz, tile_docs // 32]
    (bit s of the entry's mask in word s // 32)."""
    lib = load()
    _dev(indptr, torch.int32, "indptr")
    _dev(indices, torch.int32, "indices")
    B = indptr.numel() - 1
    nnz = indices.numel()
    T = int(tile_docs)
    ntiles = (B + T - 1) // T if T > 0 else 0
    dev = indptr.device
    if perm is not None:
        _dev(perm, torch.int32, "perm")
    tile_offset = torch.empty(ntiles + 1, dtype=torch.int32, device=dev)
    tile_count = torch.empty(max(ntiles, 1), dtype=torch.int32, device=dev)
    union_feat = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    mw = (T + 31) // 32 if T > 0 else 1
    union_mask = torch.empty((max(nnz, 1), mw) if mw > 1 else max(nnz, 1), dtype=torch.int32, device=dev)
    _check(lib.som_tile_plan(_ptr(indptr), _ptr(indices), B, F, nnz, _ptr(perm), T, _ptr(tile_offset),
                             _ptr(tile_count), _ptr(union_feat), _ptr(union_mask), _stream(stream)))
    return tile_offset, tile_count[:ntiles], union_feat, union_mask


def som_group_plan(indptr: torch.Tensor, indices: torch.Tensor, F: int, group_docs: int = 1024,
                   perm: Optional[torch.Tensor] = None, stream=None):
    """Kernel-2 group plan as explicit arrays: (group_offset, group_count, group_feat, entry_pos)."""
    lib = load()
    _dev(indptr, torch.int32, "indptr")
    _dev(indices, torch.int32, "indices")
    B = indptr.numel() - 1
    nnz = indices.numel()
    D = int(group_docs)
    ng = (B + D - 1) // D if D > 0 else 0
    dev = indptr.device
    if perm is not None:
        _dev(perm, torch.int32, "perm")
    offset = torch.empty(ng + 1, dtype=torch.int32, device=dev)
    count = torch.empty(max(ng, 1), dtype=torch.int32, device=dev)
    feat = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    pos = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    _check(lib.som_group_plan(_ptr(indptr), _ptr(indices), B, F, nnz, _ptr(perm), D, _ptr(offset),
                              _ptr(count), _ptr(feat), _ptr(pos), _stream(stream)))
    return offset, count[:ng], feat, pos


def som_cluster_workspace_bytes(B: int, F: int, nnz: int) -> int:
    return int(load().som_cluster_workspace_bytes(B, F, nnz))


def som_cluster_order(indptr: torch.Tensor, indices: torch.Tensor, F: int,
                      perm: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    """Tile order grouping documents by their two highest-df features."""
    lib = load()
    _dev(indptr, torch.int32, "indptr")
    _dev(indices, torch.int32, "indices")
    B = indptr.numel() - 1
    nnz = indices.numel()
    if perm is None:
        perm = torch.empty(max(B, 1), dtype=torch.int32, device=indptr.device)
    _dev(perm, torch.int32, "perm")
    if ws is None:
        ws = _workspace(lib.som_cluster_workspace_bytes(B, F, nnz), indptr.device)
    _dev(ws, torch.uint8, "ws")
    _check(lib.som_cluster_order(_ptr(indptr), _ptr(indices), B, F, nnz, _ptr(perm), _ptr(ws), ws.numel(),
                                 _stream(stream)))
    return perm[:B]


def som_update_accumulate(indptr: torch.Tensor, indices: torch.Tensor, bmu: torch.Tensor, F: int, N: int,
                          acc: torch.Tensor, count: torch.Tensor, stream=None) -> None:
    """acc [F, ld_acc] and count [N] (int32 tensors holding uint32 counts) += one searched batch."""
    lib = load()
    for t, name in ((indptr, "indptr"), (indices, "indices"), (bmu, "bmu"), (acc, "acc"), (count, "count")):
        _dev(t, torch.int32, name)
    B = indptr.numel() - 1
    if acc.dim() != 2 or acc.shape[0] != F or acc.shape[1] < N or count.numel() < N or bmu.numel() < B:
        raise ValueError("acc must be [F, >= N], count [>= N], bmu [>= B]")
    _check(lib.som_update_accumulate(_ptr(indptr), _ptr(indices), B, indices.numel(), _ptr(bmu), F, N, _ptr(acc),
                                     acc.shape[1], _ptr(count), _stream(stream)))


def som_update_workspace_bytes(F: int, N: int) -> int:
    return int(load().som_update_workspace_bytes(F, N))


def som_update_finish(W: torch.Tensor, rows: int, cols: int, sigma: float, acc: torch.Tensor, count: torch.Tensor,
                      ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """Blur the accumulators over the neighbourhood and write the new weights into W (fp32 or fp16)."""
    lib = load()
    sfx = _codebook(W)
    _dev(acc, torch.int32, "acc")
    _dev(count, torch.int32, "count")
    F, ldw = W.shape
    if acc.dim() != 2 or acc.shape[0] != F:
        raise ValueError("acc must be [F, ld_acc]")
    if ws is None:
        ws = _workspace(lib.som_update_workspace_bytes(F, rows * cols), W.device)
    _dev(ws, torch.uint8, "ws")
    _check(getattr(lib, "som_update_finish" + sfx)(_ptr(W), F, ldw, rows, cols, float(sigma), _ptr(acc),
                                                   acc.shape[1], _ptr(count), _ptr(ws), ws.numel(),
                                                   _stream(stream)))


def som_bmu_search_unfused_workspace_bytes(F: int, N: int, B: int, nnz: int, block_docs: int, **knobs) -> int:
    o = _opts(**knobs)
    return int(load().som_bmu_search_unfused_workspace_bytes(F, N, B, nnz, ctypes.byref(o), int(block_docs)))


def som_bmu_search_unfused(W: torch.Tensor, norms: torch.Tensor, indptr: torch.Tensor, indices: torch.Tensor,
                           N: Optional[int] = None, perm: Optional[torch.Tensor] = None, block_docs: int = 8192,
                           bmu: Optional[torch.Tensor] = None, dist: Optional[torch.Tensor] = None,
                           ws: Optional[torch.Tensor] = None, stream=None, **knobs) -> Tuple[torch.Tensor, torch.Tensor]:
    """The search with a materialised score block (the unfused comparator):
    same (bmu, dist) as som_bmu_search, bit for bit."""
    lib = load()
    _dev(W, torch.float32, "W")
    _dev(norms, torch.float32, "norms")
    _dev(indptr, torch.int32, "indptr")
    _dev(indices, torch.int32, "indices")
    F, ldw = W.shape
    n = _n_neurons(N, norms, W)
    if norms.numel() < n:
        raise ValueError("norms must hold at least N values")
    B = indptr.numel() - 1
    nnz = indices.numel()
    if perm is not None:
        _dev(perm, torch.int32, "perm")
    bmu, dist = _outputs(B, W.device, [(bmu, torch.int32, "bmu"), (dist, torch.float32, "dist")])
    o = _opts(**knobs)
    if ws is None:
        ws = _workspace(lib.som_bmu_search_unfused_workspace_bytes(F, n, B, nnz, ctypes.byref(o), int(block_docs)),
                        W.device)
    _dev(ws, torch.uint8, "ws")
    _check(lib.som_bmu_search_unfused(_ptr(W), F, n, ldw, _ptr(norms), _ptr(indptr), _ptr(indices), B, nnz,
                                      _ptr(perm), _ptr(bmu), _ptr(dist), ctypes.byref(o), int(block_docs), _ptr(ws),
                                      ws.numel(), _stream(stream)))
    return bmu, dist


def som_probe_read(buf: torch.Tensor, nbytes: int, passes: int = 1, sink: Optional[torch.Tensor] = None,
                   stream=None) -> None:
    """Read-bandwidth probe over the first nbytes of a device tensor (see som.h)."""
    lib = load()
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous ROCm device tensor")
    if nbytes > buf.numel() * buf.element_size():
        raise ValueError("nbytes exceeds the tensor")
    if sink is None:
        sink = torch.empty(1, dtype=torch.int32, device=buf.device)
    _check(lib.som_probe_read(_ptr(buf), int(nbytes), int(passes), _ptr(sink), _stream(stream)))


def som_probe_lds(iters: int, sink: torch.Tensor, stream=None) -> int:
    """LDS read probe (see som.h); returns the bytes the launch reads from LDS."""
    lib = load()
    _dev(sink, torch.int32, "sink")
    nbytes = ctypes.c_int64(0)
    _check(lib.som_probe_lds(int(iters), _ptr(sink), ctypes.byref(nbytes), _stream(stream)))
    return int(nbytes.value)

