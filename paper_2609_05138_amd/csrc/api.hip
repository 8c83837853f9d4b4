// C ABI of libsom (declared in include/som.h): host-side argument checks,
// workspace carving and kernel sequencing.  No entry point allocates device
// memory; every array comes from the caller.
#include <string>

#include "../../include/som.h"
#include "common.h"

namespace {

thread_local std::string g_error;

som_status fail(som_status s, const std::string& msg) {
  g_error = msg;
  return s;
}

som_status ok() {
  g_error.clear();
  return SOM_OK;
}

som_status hip_fail(hipError_t e, const char* where) {
  return fail(SOM_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

constexpr int64_t kI32Max = 2147483647;
constexpr int64_t kMaxTiles = int64_t(1) << 24;

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

som_status check_codebook(const float* W, int64_t F, int64_t N, int64_t ldw) {
  if (!W) return fail(SOM_ERR_INVALID_ARG, "W is NULL");
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  if (N < 1 || N > kI32Max) return fail(SOM_ERR_INVALID_ARG, "N must be in [1, 2^31)");
  if (ldw < N) return fail(SOM_ERR_INVALID_ARG, "ldw must be >= N");
  if (ldw % 4 != 0) return fail(SOM_ERR_INVALID_ARG, "ldw must be a multiple of 4");
  if (!aligned(W, 16)) return fail(SOM_ERR_INVALID_ARG, "W must be 16-byte aligned");
  return SOM_OK;
}

struct Plan {
  int T = 8;
  int K = 8;
  int group = 1;
  int mask_mode = 1;        // SearchArgs encoding: 0 = fma, 1 = branch
  int64_t ntiles = 0;
  int64_t nchunks = 0;
};

// Defaults chosen by measurement on MI355X (512^2 map, F = 20,000).
constexpr int kDefaultT = 8;
constexpr int kDefaultK = 8;
constexpr int kDefaultGroup = 1;

som_status make_plan(int64_t N, int64_t B, const som_bmu_opts* opts, Plan* p) {
  som_bmu_opts o{};
  if (opts) o = *opts;
  if (o.reserved[0] || o.reserved[1] || o.reserved[2])
    return fail(SOM_ERR_INVALID_ARG, "opts->reserved must be 0");
  if (o.validate != 0 && o.validate != 1) return fail(SOM_ERR_INVALID_ARG, "opts->validate must be 0 or 1");
  const int T = o.tile_docs ? o.tile_docs : kDefaultT;
  if (T != 1 && T != 2 && T != 4 && T != 8 && T != 16 && T != 32)
    return fail(SOM_ERR_INVALID_ARG, "opts->tile_docs must be 0, 1, 2, 4, 8, 16 or 32");
  const int K = o.lane_neurons ? o.lane_neurons : (T >= 32 ? 4 : kDefaultK);
  if (K != 4 && K != 8) return fail(SOM_ERR_INVALID_ARG, "opts->lane_neurons must be 0, 4 or 8");
  if (T == 32 && K != 4) return fail(SOM_ERR_INVALID_ARG, "opts->lane_neurons must be 4 when tile_docs is 32");
  const int G = o.group_tiles ? o.group_tiles : kDefaultGroup;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(SOM_ERR_INVALID_ARG, "opts->group_tiles must be 0, 1, 2, 4 or 8");
  if (o.mask_mode < 0 || o.mask_mode > 2) return fail(SOM_ERR_INVALID_ARG, "opts->mask_mode must be 0, 1 or 2");
  p->T = T;
  p->K = K;
  p->group = G;
  p->mask_mode = o.mask_mode == 2 ? 1 : (o.mask_mode == 1 ? 0 : (T <= 4 ? 0 : 1));
  p->ntiles = (B + T - 1) / T;
  p->nchunks = (N + 64 * K - 1) / (64 * K);
  // one 256-thread plan workgroup per tile, and the search grid (tile
  // groups, slices): work-items per grid dimension must stay below 2^32
  if (p->ntiles >= kMaxTiles)
    return fail(SOM_ERR_INVALID_ARG, "batch too large for one launch: ceil(B/T) must be < 2^24");
  if (p->nchunks > 65535)
    return fail(SOM_ERR_INVALID_ARG, "too many neuron slices for one launch (N / (64*K) must be <= 65535)");
  return SOM_OK;
}

// Workspace layout of som_bmu_search (each region 256-byte aligned): the
// tile plan, then the per-document packed minima (the planned search's part).
struct SearchWs {
  size_t tile_offset, tile_count, union_feat, union_mask, partial, flag, seen, total;
};

size_t partial_bytes(const Plan& p) { return sizeof(uint64_t) * p.ntiles * p.T; }

SearchWs search_ws(const Plan& p, int64_t B, int64_t nnz, bool validate) {
  SearchWs w{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = som::align_up(o + (bytes ? bytes : 1), 256);
    return at;
  };
  w.tile_offset = take(sizeof(int32_t) * (p.ntiles + 1));
  w.tile_count = take(sizeof(int32_t) * p.ntiles);
  w.union_feat = take(sizeof(int32_t) * nnz);
  w.union_mask = take(sizeof(uint32_t) * nnz);
  w.flag = take(sizeof(int32_t) * 4);
  w.seen = validate ? take(sizeof(int32_t) * B) : 0;
  w.partial = take(partial_bytes(p));
  w.total = o;
  return w;
}

template <typename P>
P* at(void* base, size_t off) {
  return reinterpret_cast<P*>(static_cast<char*>(base) + off);
}

som_status check_batch(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz) {
  if (B < 0 || B >= kI32Max) return fail(SOM_ERR_INVALID_ARG, "B must be in [0, 2^31 - 1)");
  if (nnz < 0 || nnz > kI32Max) return fail(SOM_ERR_INVALID_ARG, "nnz must be in [0, 2^31)");
  if (B > 0 && !indptr) return fail(SOM_ERR_INVALID_ARG, "indptr is NULL");
  if (nnz > 0 && !indices) return fail(SOM_ERR_INVALID_ARG, "indices is NULL");
  return SOM_OK;
}

som_status run_validate(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                        int64_t nnz, const int32_t* perm, int32_t* seen, int32_t* flag,
                        hipStream_t stream) {
  hipError_t e = som::launch_validate(indptr, indices, B, F, nnz, perm, seen, flag, stream);
  if (e != hipSuccess) return hip_fail(e, "validate launch");
  int32_t host_flag = 0;
  e = hipMemcpyAsync(&host_flag, flag, sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return hip_fail(e, "validate read-back");
  e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "validate synchronize");
  if (host_flag) {
    std::string why;
    if (host_flag & 1) why += " indptr[0] != 0 or indptr[B] != nnz;";
    if (host_flag & 2) why += " indptr not non-decreasing within [0, nnz];";
    if (host_flag & 4) why += " feature ids out of [0, F) or not strictly ascending;";
    if (host_flag & 8) why += " perm value out of [0, B);";
    if (host_flag & 16) why += " perm repeats a document;";
    return fail(SOM_ERR_INVALID_CSR, "invalid batch:" + why);
  }
  return SOM_OK;
}

som_status run_planned(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                       const int32_t* indptr, int64_t B, const int32_t* perm, const int32_t* tile_offset,
                       const int32_t* tile_count, const int32_t* union_feat, const uint32_t* union_mask,
                       int32_t* bmu, float* dist, const Plan& p, uint64_t* partial, hipStream_t stream) {
  som::SearchArgs a{};
  a.W = W;
  a.F = F;
  a.N = N;
  a.ldw = ldw;
  a.norms = norms;
  a.indptr = indptr;
  a.perm = perm;
  a.B = B;
  a.T = p.T;
  a.K = p.K;
  a.group = p.group;
  a.mask_mode = p.mask_mode;
  a.ntiles = p.ntiles;
  a.nchunks = p.nchunks;
  a.tile_offset = tile_offset;
  a.tile_count = tile_count;
  a.union_feat = union_feat;
  a.union_mask = union_mask;
  a.keys = partial;
  a.bmu = bmu;
  a.dist = dist;
  hipError_t e = som::launch_search(a, stream);
  if (e != hipSuccess) return hip_fail(e, "search launch");
  e = som::launch_merge(a, stream);
  if (e != hipSuccess) return hip_fail(e, "merge launch");
  return ok();
}

}  // namespace

extern "C" {

int32_t som_abi_version(void) { return 3; }

const char* som_last_error(void) { return g_error.c_str(); }

som_status som_codebook_norms(const float* W, int64_t F, int64_t N, int64_t ldw, float* norms,
                              hipStream_t stream) {
  som_status s = check_codebook(W, F, N, ldw);
  if (s != SOM_OK) return s;
  if (!norms) return fail(SOM_ERR_INVALID_ARG, "norms is NULL");
  hipError_t e = som::launch_norms(W, F, N, ldw, norms, stream);
  if (e != hipSuccess) return hip_fail(e, "norms launch");
  return ok();
}

size_t som_bmu_workspace_bytes(int64_t F, int64_t N, int64_t B, int64_t nnz, const som_bmu_opts* opts) {
  if (F < 1 || N < 1 || B < 0 || nnz < 0) return 0;
  Plan p;
  if (make_plan(N, B, opts, &p) != SOM_OK) return 0;
  const bool validate = opts && opts->validate;
  return search_ws(p, B, nnz, validate).total;
}

som_status som_bmu_search(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                          const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                          const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  som_status s = check_codebook(W, F, N, ldw);
  if (s != SOM_OK) return s;
  if (!norms) return fail(SOM_ERR_INVALID_ARG, "norms is NULL");
  s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (B > 0 && (!bmu || !dist)) return fail(SOM_ERR_INVALID_ARG, "bmu or dist is NULL");
  Plan p;
  s = make_plan(N, B, opts, &p);
  if (s != SOM_OK) return s;
  const bool validate = opts && opts->validate;
  const SearchWs w = search_ws(p, B, nnz, validate);
  if (B == 0) return ok();
  if (!ws) return fail(SOM_ERR_WORKSPACE, "ws is NULL");
  if (!aligned(ws, 256)) return fail(SOM_ERR_INVALID_ARG, "ws must be 256-byte aligned");
  if (ws_bytes < w.total)
    return fail(SOM_ERR_WORKSPACE, "workspace too small: need " + std::to_string(w.total) + " bytes");

  if (validate) {
    s = run_validate(indptr, indices, B, F, nnz, perm, at<int32_t>(ws, w.seen), at<int32_t>(ws, w.flag), stream);
    if (s != SOM_OK) return s;
  }
  hipError_t e = som::launch_tile_plan(indptr, indices, B, F, perm, p.T, at<int32_t>(ws, w.tile_offset),
                                       at<int32_t>(ws, w.tile_count), at<int32_t>(ws, w.union_feat),
                                       at<uint32_t>(ws, w.union_mask), stream);
  if (e != hipSuccess) return hip_fail(e, "tile plan launch");
  return run_planned(W, F, N, ldw, norms, indptr, B, perm, at<int32_t>(ws, w.tile_offset),
                     at<int32_t>(ws, w.tile_count), at<int32_t>(ws, w.union_feat),
                     at<uint32_t>(ws, w.union_mask), bmu, dist, p, at<uint64_t>(ws, w.partial), stream);
}

size_t som_bmu_search_planned_workspace_bytes(int64_t N, int64_t B, const som_bmu_opts* opts) {
  if (N < 1 || B < 0) return 0;
  Plan p;
  if (make_plan(N, B, opts, &p) != SOM_OK) return 0;
  return som::align_up(partial_bytes(p) ? partial_bytes(p) : 1, 256);
}

som_status som_bmu_search_planned(const float* W, int64_t F, int64_t N, int64_t ldw,
                                  const float* norms, const int32_t* indptr, int64_t B,
                                  const int32_t* perm, const int32_t* tile_offset,
                                  const int32_t* tile_count, const int32_t* union_feat,
                                  const uint32_t* union_mask, int32_t* bmu, float* dist,
                                  const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                                  hipStream_t stream) {
  som_status s = check_codebook(W, F, N, ldw);
  if (s != SOM_OK) return s;
  if (!norms) return fail(SOM_ERR_INVALID_ARG, "norms is NULL");
  if (B < 0 || B >= kI32Max) return fail(SOM_ERR_INVALID_ARG, "B must be in [0, 2^31 - 1)");
  Plan p;
  s = make_plan(N, B, opts, &p);
  if (s != SOM_OK) return s;
  if (opts && opts->validate) return fail(SOM_ERR_INVALID_ARG, "validate is not available on a planned search");
  if (B == 0) return ok();
  if (!indptr || !bmu || !dist || !tile_offset || !tile_count || !union_feat || !union_mask)
    return fail(SOM_ERR_INVALID_ARG, "a required pointer is NULL");
  if (!ws) return fail(SOM_ERR_WORKSPACE, "ws is NULL");
  if (!aligned(ws, 256)) return fail(SOM_ERR_INVALID_ARG, "ws must be 256-byte aligned");
  if (ws_bytes < partial_bytes(p))
    return fail(SOM_ERR_WORKSPACE, "workspace too small: need " + std::to_string(partial_bytes(p)) + " bytes");
  return run_planned(W, F, N, ldw, norms, indptr, B, perm, tile_offset, tile_count, union_feat, union_mask,
                     bmu, dist, p, static_cast<uint64_t*>(ws), stream);
}

som_status som_tile_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                         int64_t nnz, const int32_t* perm, int32_t tile_docs, int32_t* tile_offset,
                         int32_t* tile_count, int32_t* union_feat, uint32_t* union_mask,
                         hipStream_t stream) {
  som_status s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  const int T = tile_docs;
  if (T != 1 && T != 2 && T != 4 && T != 8 && T != 16 && T != 32)
    return fail(SOM_ERR_INVALID_ARG, "tile_docs must be 1, 2, 4, 8, 16 or 32");
  if ((B + T - 1) / T >= kMaxTiles)
    return fail(SOM_ERR_INVALID_ARG, "batch too large for one launch: ceil(B/T) must be < 2^24");
  if (B == 0) return ok();
  if (!tile_offset || !tile_count || (nnz > 0 && (!union_feat || !union_mask)))
    return fail(SOM_ERR_INVALID_ARG, "an output array is NULL");
  hipError_t e = som::launch_tile_plan(indptr, indices, B, F, perm, T, tile_offset, tile_count,
                                       union_feat, union_mask, stream);
  if (e != hipSuccess) return hip_fail(e, "tile plan launch");
  return ok();
}

size_t som_cluster_workspace_bytes(int64_t B, int64_t F, int64_t nnz) {
  if (B < 0 || F < 1 || nnz < 0 || B >= kI32Max) return 0;
  size_t o = 0;
  auto take = [&](size_t bytes) { o = som::align_up(o + (bytes ? bytes : 1), 256); };
  take(sizeof(int32_t) * F);        // df
  take(sizeof(uint64_t) * B);       // keys
  take(sizeof(uint64_t) * B);       // sorted keys
  take(sizeof(int32_t) * B);        // iota
  take(som::cluster_sort_temp_bytes(B, F));
  return o;
}

som_status som_cluster_order(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                             int64_t nnz, int32_t* perm, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  som_status s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  if (B == 0) return ok();
  if (!perm) return fail(SOM_ERR_INVALID_ARG, "perm is NULL");
  if (!ws) return fail(SOM_ERR_WORKSPACE, "ws is NULL");
  if (!aligned(ws, 256)) return fail(SOM_ERR_INVALID_ARG, "ws must be 256-byte aligned");
  const size_t need = som_cluster_workspace_bytes(B, F, nnz);
  if (ws_bytes < need)
    return fail(SOM_ERR_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes");
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t a = o;
    o = som::align_up(o + (bytes ? bytes : 1), 256);
    return a;
  };
  const size_t o_df = take(sizeof(int32_t) * F);
  const size_t o_keys = take(sizeof(uint64_t) * B);
  const size_t o_sorted = take(sizeof(uint64_t) * B);
  const size_t o_iota = take(sizeof(int32_t) * B);
  const size_t tb = som::cluster_sort_temp_bytes(B, F);
  const size_t o_tmp = take(tb);
  hipError_t e = som::launch_cluster(indptr, indices, B, F, nnz, perm, at<int32_t>(ws, o_df),
                                     at<uint64_t>(ws, o_keys), at<uint64_t>(ws, o_sorted),
                                     at<int32_t>(ws, o_iota), at<void>(ws, o_tmp), tb, stream);
  if (e != hipSuccess) return hip_fail(e, "cluster launch");
  return ok();
}

}  // extern "C"
