// C ABI of libsom (declared in include/som.h): host-side argument checks,
// workspace carving and kernel sequencing.  No entry point allocates device
// memory; every array comes from the caller.
#include <cmath>
#include <cstdint>
#include <mutex>
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
constexpr int64_t kMaxTiles = int64_t(1) << 24;  // tiles or groups per launch

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

template <typename P>
P* at(void* base, size_t off) {
  return reinterpret_cast<P*>(static_cast<char*>(base) + off);
}

template <typename P>
const P* at(const void* base, size_t off) {
  return reinterpret_cast<const P*>(static_cast<const char*>(base) + off);
}

// One 128-bit load holds 4 fp32 or 8 fp16 weights; rows must start on one.
som_status check_codebook(const void* W, int weights, int64_t F, int64_t N, int64_t ldw) {
  if (!W) return fail(SOM_ERR_INVALID_ARG, "W is NULL");
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  if (N < 1 || N > kI32Max) return fail(SOM_ERR_INVALID_ARG, "N must be in [1, 2^31)");
  if (ldw < N) return fail(SOM_ERR_INVALID_ARG, "ldw must be >= N");
  // row offsets f * ldw are formed in 64-bit byte arithmetic on the device
  if (ldw > (INT64_MAX / 4) / F) return fail(SOM_ERR_INVALID_ARG, "F * ldw exceeds the addressable range");
  if (weights == som::kWeightsF16 && ldw % 8 != 0)
    return fail(SOM_ERR_INVALID_ARG, "ldw must be a multiple of 8 for an fp16 codebook");
  if (ldw % 4 != 0) return fail(SOM_ERR_INVALID_ARG, "ldw must be a multiple of 4");
  if (!aligned(W, 16)) return fail(SOM_ERR_INVALID_ARG, "W must be 16-byte aligned");
  return SOM_OK;
}

som_status check_batch(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz) {
  if (B < 0 || B >= kI32Max) return fail(SOM_ERR_INVALID_ARG, "B must be in [0, 2^31 - 1)");
  if (nnz < 0 || nnz > kI32Max) return fail(SOM_ERR_INVALID_ARG, "nnz must be in [0, 2^31)");
  if (B > 0 && !indptr) return fail(SOM_ERR_INVALID_ARG, "indptr is NULL");
  if (nnz > 0 && !indices) return fail(SOM_ERR_INVALID_ARG, "indices is NULL");
  return SOM_OK;
}

// Resolved knobs.  The automatic choices follow measurements on MI355X (512^2
// and 256^2 maps, F = 20,000, 1M-document batches).
struct Plan {
  int kernel = 1;
  // kernel 1
  int T = 8;
  int K = 4;
  int mask_mode = 1;  // SearchArgs encoding: 0 = fma, 1 = branch
  // kernel 1: tiles per workgroup; kernel 2: waves per workgroup
  int group = 16;
  // kernel 2
  int NB = 32;
  int64_t D = 1024;     // documents per tile (kernel 1) or per group (kernel 2)
  int64_t nunits = 0;   // tiles or groups
  int64_t nchunks = 0;  // neuron slices
  bool stage_masks = false;  // kernel 3, document-major: masks stored per stage and document
  int schedule = 1;          // 1 = one launch, 2 = round-synchronised launches (kernel 3)
  int chunk_slices = 1;      // kernels 1 and 3: neuron slices per schedule chunk
  bool rotate = false;       // kernel 3: rotated union sweeps (opts->sweep)
};

// Kernel-1 tiles per workgroup chosen automatically: four consecutive tiles
// of 16 documents share one CU (and its vector L1) on large fp32 maps, where
// it ran a 1M-document batch of the 512^2 map 2.9% faster; one elsewhere (the
// 256^2 map and fp16 codebooks were neutral or slower).
constexpr int64_t kGroupTilesMinN = 131072;

// `weights` is the storage type of the codebook searched (it fixes the load
// width K); `auto_weights` the one the automatic tile size is chosen for:
// the entry point's own type when it plans internally, opts->storage for
// som_plan and the planned searches, so that a plan and its search always
// resolve the same tile geometry.
som_status make_plan(int64_t N, int64_t B, const som_bmu_opts* opts, Plan* p, int weights, int auto_weights) {
  som_bmu_opts o{};
  if (opts) o = *opts;
  const bool f16 = weights == som::kWeightsF16;
  const bool auto16 = auto_weights == som::kWeightsF16;
  if (f16 && o.kernel == 2) return fail(SOM_ERR_INVALID_ARG, "an fp16 codebook is searched by kernels 1 and 3 only");
  if (o.storage != 0 && o.storage != 1) return fail(SOM_ERR_INVALID_ARG, "opts->storage must be 0 (fp32) or 1 (fp16)");
  if (o.validate != 0 && o.validate != 1) return fail(SOM_ERR_INVALID_ARG, "opts->validate must be 0 or 1");
  if (o.schedule < 0 || o.schedule > 2) return fail(SOM_ERR_INVALID_ARG, "opts->schedule must be 0, 1 or 2");
  if (o.kernel < 0 || o.kernel > 3) return fail(SOM_ERR_INVALID_ARG, "opts->kernel must be 0, 1, 2 or 3");
  // automatic kernel: the shared-union super-tiles (kernel 3) for an fp32
  // codebook, measured faster at every map size from 32^2 to 512^2 and on the
  // topic workload; kernel 1 for fp16 (8-document tiles, measured faster
  // there) and whenever a knob only kernel 1 has is given
  const bool k1_knob = (o.tile_docs > 0 && o.tile_docs <= 32) || o.lane_neurons || o.group_tiles;
  const int kernel = o.kernel ? o.kernel : ((auto16 || k1_knob) ? 1 : 3);
  p->kernel = kernel;
  if (kernel == 1) {
    // automatic tile size: 16 documents for fp32 (about 5% faster than 8 on
    // the 512^2 map), 8 for fp16 (whose 512-neuron slices leave fewer
    // registers for accumulators)
    const int T = o.tile_docs ? o.tile_docs : (auto16 ? 8 : 16);
    if (T != 1 && T != 2 && T != 4 && T != 8 && T != 16 && T != 32)
      return fail(SOM_ERR_INVALID_ARG, "opts->tile_docs must be 0, 1, 2, 4, 8, 16 or 32");
    if (f16 && T == 32) return fail(SOM_ERR_INVALID_ARG, "opts->tile_docs 32 is not available for an fp16 codebook");
    const int K = o.lane_neurons ? o.lane_neurons : (f16 ? 8 : 4);
    if (K != 4 && K != 8) return fail(SOM_ERR_INVALID_ARG, "opts->lane_neurons must be 0, 4 or 8");
    if (T == 32 && K != 4) return fail(SOM_ERR_INVALID_ARG, "opts->lane_neurons must be 4 when tile_docs is 32");
    if (f16 && K != 8) return fail(SOM_ERR_INVALID_ARG, "opts->lane_neurons must be 0 or 8 for an fp16 codebook");
    const int G = o.group_tiles ? o.group_tiles : ((!f16 && !auto16 && T == 16 && N >= kGroupTilesMinN) ? 4 : 1);
    if (G != 1 && G != 2 && G != 4 && G != 8)
      return fail(SOM_ERR_INVALID_ARG, "opts->group_tiles must be 0, 1, 2, 4 or 8 for kernel 1");
    if (o.mask_mode < 0 || o.mask_mode > 2) return fail(SOM_ERR_INVALID_ARG, "opts->mask_mode must be 0, 1 or 2");
    if (o.slice_neurons != 0) return fail(SOM_ERR_INVALID_ARG, "opts->slice_neurons applies to kernel 2 only");
    p->T = T;
    p->K = K;
    p->group = G;
    p->mask_mode = o.mask_mode == 2 ? 1 : (o.mask_mode == 1 ? 0 : (T <= 4 ? 0 : 1));
    p->D = T;
    p->nchunks = (N + 64 * K - 1) / (64 * K);
  } else if (kernel == 3) {
    // super-tile of D documents; waves of 8 documents (16 for D = 256 with an
    // fp32 codebook, as a workgroup holds at most 16 waves)
    if (o.group_tiles || o.slice_neurons)
      return fail(SOM_ERR_INVALID_ARG, "opts->group_tiles and slice_neurons must be 0 for kernel 3");
    if (o.mask_mode < 0 || o.mask_mode > 2) return fail(SOM_ERR_INVALID_ARG, "opts->mask_mode must be 0, 1 or 2");
    const int D = o.tile_docs ? o.tile_docs : 64;
    if (D != 64 && D != 128 && D != 256)
      return fail(SOM_ERR_INVALID_ARG, "opts->tile_docs must be 0, 64, 128 or 256 for kernel 3");
    if (f16 && D == 256) return fail(SOM_ERR_INVALID_ARG, "opts->tile_docs 256 is not available for an fp16 codebook");
    const int K = f16 ? 8 : 4;
    if (o.lane_neurons && o.lane_neurons != K)
      return fail(SOM_ERR_INVALID_ARG, "opts->lane_neurons must be 0 (or 4 for fp32, 8 for fp16) for kernel 3");
    p->T = D == 256 ? 16 : 8;
    p->K = K;
    p->group = D / p->T;
    // SearchArgs encoding for kernel 3: 1 = row-major dispatch, 2 = document-major
    // (automatic: measured faster on the 128^2, 512^2 and topic workloads); the
    // document-major form reads its plan's masks stage by stage, per document
    p->mask_mode = o.mask_mode ? o.mask_mode : 2;
    p->stage_masks = p->mask_mode == 2;
    p->schedule = o.schedule ? o.schedule : 1;
    p->D = D;
    p->nchunks = (N + 64 * K - 1) / (64 * K);
  } else {
    if (o.tile_docs || o.lane_neurons || o.mask_mode)
      return fail(SOM_ERR_INVALID_ARG, "opts->tile_docs, lane_neurons and mask_mode apply to kernels 1 and 3 only");
    const int G = o.group_tiles ? o.group_tiles : 16;
    if (G != 4 && G != 8 && G != 16)
      return fail(SOM_ERR_INVALID_ARG, "opts->group_tiles must be 0, 4, 8 or 16 for kernel 2");
    const int NB = o.slice_neurons ? o.slice_neurons : 32;
    if (NB != 32 && NB != 64) return fail(SOM_ERR_INVALID_ARG, "opts->slice_neurons must be 0, 32 or 64");
    p->group = G;
    p->NB = NB;
    p->D = 64 * G;
    p->nchunks = (N + NB - 1) / NB;
  }
  if (kernel != 3 && o.schedule == 2)
    return fail(SOM_ERR_INVALID_ARG, "opts->schedule 2 (round-synchronised launches) applies to kernel 3 only");
  if (o.neuron_chunk < 0) return fail(SOM_ERR_INVALID_ARG, "opts->neuron_chunk must be >= 0");
  if (o.neuron_chunk) {
    const int64_t width = 64 * static_cast<int64_t>(p->K);
    if (kernel == 2) return fail(SOM_ERR_INVALID_ARG, "opts->neuron_chunk applies to kernels 1 and 3 only");
    if (p->schedule == 2) return fail(SOM_ERR_INVALID_ARG, "opts->neuron_chunk needs schedule 1 (one launch)");
    if (o.neuron_chunk % width)
      return fail(SOM_ERR_INVALID_ARG, "opts->neuron_chunk must be a multiple of the slice width (64 * K neurons)");
    const int64_t q = o.neuron_chunk / width;
    p->chunk_slices = static_cast<int>(q < p->nchunks ? q : (p->nchunks > 0 ? p->nchunks : 1));
  }
  // sweep order: rotated wherever kernel 1 or kernel 3's document-major form
  // runs as one launch of one-slice chunks (measured 19% faster with kernel 3
  // and 17% with fp16 kernel 1 on the topic workload, within 1.3% either way
  // on the Zipf maps), ascending elsewhere
  if (o.sweep < 0 || o.sweep > 2) return fail(SOM_ERR_INVALID_ARG, "opts->sweep must be 0, 1 or 2");
  const bool can_rotate = p->chunk_slices == 1 && p->schedule == 1 &&
                          ((kernel == 3 && p->mask_mode == 2) || kernel == 1);
  if (o.sweep == 2 && !can_rotate)
    return fail(SOM_ERR_INVALID_ARG,
                "opts->sweep 2 (rotated) needs kernel 1, or kernel 3 with mask_mode 2, as one launch of "
                "one-slice chunks (schedule 1)");
  p->rotate = o.sweep == 2 || (o.sweep == 0 && can_rotate);
  p->nunits = (B + p->D - 1) / p->D;
  if (p->nunits >= kMaxTiles)
    return fail(SOM_ERR_INVALID_ARG, "batch too large for one launch: too many tiles or groups");
  if (p->nchunks > 65535)
    return fail(SOM_ERR_INVALID_ARG, "too many neuron slices for one launch (N / slice width must be <= 65535)");
  return SOM_OK;
}

// Storage type named by the options (for som_plan and the planned searches).
int opts_storage(const som_bmu_opts* opts) {
  return (opts && opts->storage == 1) ? som::kWeightsF16 : som::kWeightsF32;
}

size_t take(size_t& o, size_t bytes) {
  const size_t a = o;
  o = som::align_up(o + (bytes ? bytes : 1), 256);
  return a;
}

// Plan layout (each region 256-byte aligned): offsets [nunits+1], counts
// [nunits], union features [nnz], then kernel 1 masks or kernel 2 entry
// positions [nnz]; kernel 3: features [nnz + pad], masks [nnz + pad][D / 32],
// pad = 256 entries, plus 16 per tile with stage masks.
struct PlanLayout {
  size_t offset, count, feat, extra, total;
};

PlanLayout plan_layout(const Plan& p, int64_t nnz) {
  PlanLayout l{};
  size_t o = 0;
  l.offset = take(o, sizeof(int32_t) * (p.nunits + 1));
  l.count = take(o, sizeof(int32_t) * p.nunits);
  // kernel 3 reads whole stages, and feature ids a few stages ahead, past a
  // union's end; with stage masks each tile's region is rounded up to whole
  // 16-entry stages
  const int64_t pad = p.kernel == 3 ? 256 + (p.stage_masks ? 16 * p.nunits : 0) : 0;
  l.feat = take(o, sizeof(int32_t) * (nnz + pad));
  l.extra = take(o, sizeof(int32_t) * (p.kernel == 3 ? (nnz + pad) * (p.D / 32) : nnz));
  l.total = o;
  return l;
}

// Packed keys: best [B] then second best [B] (the second array is used by
// the top-2 searches only), each 256-byte aligned.
size_t keys_half_bytes(int64_t B) { return som::align_up(sizeof(uint64_t) * (B ? B : 1), 256); }
size_t keys_bytes(int64_t B) { return 2 * keys_half_bytes(B); }

// Workspace of som_bmu_search: the plan, a validation flag and scratch, the keys.
struct SearchWs {
  PlanLayout plan;
  size_t flag, seen, keys, total;
};

SearchWs search_ws(const Plan& p, int64_t B, int64_t nnz, bool validate) {
  SearchWs w{};
  w.plan = plan_layout(p, nnz);
  size_t o = w.plan.total;
  w.flag = take(o, sizeof(int32_t) * 4);
  w.seen = validate ? take(o, sizeof(int32_t) * B) : 0;
  w.keys = take(o, keys_bytes(B));
  w.total = o;
  return w;
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

hipError_t build_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                      const int32_t* perm, const Plan& p, void* plan, const PlanLayout& l,
                      hipStream_t stream) {
  if (p.kernel == 1 || p.kernel == 3)
    return som::launch_tile_plan(indptr, indices, B, F, perm, static_cast<int>(p.D), at<int32_t>(plan, l.offset),
                                 at<int32_t>(plan, l.count), at<int32_t>(plan, l.feat),
                                 at<uint32_t>(plan, l.extra), stream, p.stage_masks);
  return som::launch_group_plan(indptr, indices, B, F, perm, static_cast<int>(p.D),
                                at<int32_t>(plan, l.offset), at<int32_t>(plan, l.count),
                                at<int32_t>(plan, l.feat), at<int32_t>(plan, l.extra), stream);
}

som_status run_planned(const void* W, int weights, int64_t F, int64_t N, int64_t ldw, const float* norms,
                       const int32_t* indptr, int64_t B, const int32_t* perm, const void* plan,
                       const PlanLayout& l, int32_t* bmu, float* dist, int32_t* bmu2, float* dist2,
                       const Plan& p, uint64_t* keys, hipStream_t stream) {
  som::SearchArgs a{};
  a.W = W;
  a.weights = weights;
  a.F = F;
  a.N = N;
  a.ldw = ldw;
  a.norms = norms;
  a.indptr = indptr;
  a.perm = perm;
  a.B = B;
  a.kernel = p.kernel;
  a.T = p.T;
  a.K = p.K;
  a.group = p.group;
  a.mask_mode = p.mask_mode;
  a.chunk_slices = p.chunk_slices;
  a.rotate = p.rotate ? 1 : 0;
  a.slice = p.NB;
  a.ntiles = p.nunits;
  a.nchunks = p.nchunks;
  a.tile_base = 0;
  a.tile_end = p.nunits;
  a.schedule = p.schedule;
  if (p.kernel == 1 || p.kernel == 3) {
    a.tile_offset = at<int32_t>(plan, l.offset);
    a.tile_count = at<int32_t>(plan, l.count);
    a.union_feat = at<int32_t>(plan, l.feat);
    a.union_mask = at<uint32_t>(plan, l.extra);
  } else {
    a.group_offset = at<int32_t>(plan, l.offset);
    a.group_count = at<int32_t>(plan, l.count);
    a.group_feat = at<int32_t>(plan, l.feat);
    a.entry_pos = at<int32_t>(plan, l.extra);
  }
  a.keys = keys;
  a.bmu = bmu;
  a.dist = dist;
  if (bmu2) {
    a.keys2 = keys + keys_half_bytes(B) / sizeof(uint64_t);
    a.bmu2 = bmu2;
    a.dist2 = dist2;
  }
  hipError_t e = som::launch_search(a, stream);
  if (e != hipSuccess) return hip_fail(e, "search launch");
  e = som::launch_merge(a, stream);
  if (e != hipSuccess) return hip_fail(e, "decode launch");
  return ok();
}

}  // namespace

extern "C" {

int32_t som_abi_version(void) { return 15; }

const char* som_last_error(void) { return g_error.c_str(); }

int64_t som_codebook_ldw(int64_t N) {
  if (N < 1) return 0;
  int64_t ldw = (N + 63) / 64 * 64;
  if (ldw % 512 == 0) ldw += 64;
  return ldw;
}

static som_status norms_impl(const void* W, int weights, int64_t F, int64_t N, int64_t ldw, float* norms,
                             hipStream_t stream) {
  som_status s = check_codebook(W, weights, F, N, ldw);
  if (s != SOM_OK) return s;
  if (!norms) return fail(SOM_ERR_INVALID_ARG, "norms is NULL");
  hipError_t e = som::launch_norms(W, weights, F, N, ldw, norms, stream);
  if (e != hipSuccess) return hip_fail(e, "norms launch");
  return ok();
}

som_status som_codebook_norms(const float* W, int64_t F, int64_t N, int64_t ldw, float* norms,
                              hipStream_t stream) {
  return norms_impl(W, som::kWeightsF32, F, N, ldw, norms, stream);
}

som_status som_codebook_norms_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw, float* norms,
                                  hipStream_t stream) {
  return norms_impl(W, som::kWeightsF16, F, N, ldw, norms, stream);
}

// Workspace of a search that plans internally: the automatic tile size
// depends on the storage type of the entry point called, so the size covers
// both (an fp16 tile plan has more, smaller tiles).
static size_t search_ws_bytes(int64_t N, int64_t B, int64_t nnz, const som_bmu_opts* opts) {
  size_t need = 0;
  for (int w : {som::kWeightsF32, som::kWeightsF16}) {
    Plan p;
    if (make_plan(N, B, opts, &p, w, w) != SOM_OK) continue;
    const size_t t = search_ws(p, B, nnz, opts && opts->validate).total;
    need = t > need ? t : need;
  }
  return need;
}

size_t som_bmu_workspace_bytes(int64_t F, int64_t N, int64_t B, int64_t nnz, const som_bmu_opts* opts) {
  if (F < 1 || N < 1 || B < 0 || nnz < 0) return 0;
  Plan p;
  if (make_plan(N, B, opts, &p, som::kWeightsF32, som::kWeightsF32) != SOM_OK) return 0;
  return search_ws_bytes(N, B, nnz, opts);
}

static som_status search_impl(const void* W, int weights, int64_t F, int64_t N, int64_t ldw,
                              const float* norms, const int32_t* indptr, const int32_t* indices, int64_t B,
                              int64_t nnz, const int32_t* perm, int32_t* bmu, float* dist, int32_t* bmu2,
                              float* dist2, bool top2, const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  som_status s = check_codebook(W, weights, F, N, ldw);
  if (s != SOM_OK) return s;
  if (!norms) return fail(SOM_ERR_INVALID_ARG, "norms is NULL");
  s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (B > 0 && (!bmu || !dist)) return fail(SOM_ERR_INVALID_ARG, "bmu or dist is NULL");
  if (top2 && B > 0 && (!bmu2 || !dist2)) return fail(SOM_ERR_INVALID_ARG, "bmu2 or dist2 is NULL");
  Plan p;
  s = make_plan(N, B, opts, &p, weights, weights);
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
  hipError_t e = build_plan(indptr, indices, B, F, perm, p, ws, w.plan, stream);
  if (e != hipSuccess) return hip_fail(e, "plan launch");
  return run_planned(W, weights, F, N, ldw, norms, indptr, B, perm, ws, w.plan, bmu, dist, top2 ? bmu2 : nullptr,
                     dist2, p, at<uint64_t>(ws, w.keys), stream);
}

som_status som_bmu_search(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                          const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                          const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  return search_impl(W, som::kWeightsF32, F, N, ldw, norms, indptr, indices, B, nnz, perm, bmu, dist, nullptr,
                     nullptr, false, opts, ws, ws_bytes, stream);
}

// ---------------------------------------------------------------------------
// Allocation-free search: the workspace of som_bmu_search (plan and packed
// keys) lives in a file-scope device array instead of a caller's buffer.
// ---------------------------------------------------------------------------

}  // extern "C"

// One copy per GPU, held from the library's load until the process ends.  In
// host code `scratch` names a host-side stand-in: its device address is
// looked up (hipGetSymbolAddress) once per device and only that address is
// ever passed to kernels.
static __device__ __align__(256) unsigned char scratch[SOM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device (looked up on the first
// call on that device, with the device current).
som_status noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(SOM_ERR_INVALID_ARG, "current device index beyond 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(SOM_ERR_HIP, "hipGetSymbolAddress(scratch) returned no address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SOM_OK;
}

}  // namespace

extern "C" {

som_status som_bmu_search_noalloc(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                                  const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                                  const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                                  hipStream_t stream) {
  // every check and the size limit come before any HIP call
  som_status s = check_codebook(W, som::kWeightsF32, F, N, ldw);
  if (s != SOM_OK) return s;
  if (!norms) return fail(SOM_ERR_INVALID_ARG, "norms is NULL");
  s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (B > 0 && (!bmu || !dist)) return fail(SOM_ERR_INVALID_ARG, "bmu or dist is NULL");
  if (opts && opts->validate)
    return fail(SOM_ERR_INVALID_ARG, "validate synchronises the stream: not available on the allocation-free search");
  Plan p;
  s = make_plan(N, B, opts, &p, som::kWeightsF32, som::kWeightsF32);
  if (s != SOM_OK) return s;
  const size_t need = search_ws(p, B, nnz, false).total;
  if (need > SOM_NOALLOC_SCRATCH_BYTES)
    return fail(SOM_ERR_INVALID_ARG, "this batch needs " + std::to_string(need) +
                                         " bytes of workspace, more than the " +
                                         std::to_string(SOM_NOALLOC_SCRATCH_BYTES) +
                                         " the allocation-free search holds: split the batch or use som_bmu_search");
  if (B == 0) return ok();
  void* ws = nullptr;
  s = noalloc_scratch(&ws);
  if (s != SOM_OK) return s;
  // the plan and keys are rewritten in full by each call (the keys by their
  // own initialisation kernel), so nothing left by an earlier call is read
  return search_impl(W, som::kWeightsF32, F, N, ldw, norms, indptr, indices, B, nnz, perm, bmu, dist, nullptr,
                     nullptr, false, opts, ws, SOM_NOALLOC_SCRATCH_BYTES, stream);
}

som_status som_bmu_search_top2(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                               const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                               const int32_t* perm, int32_t* bmu, float* dist, int32_t* bmu2, float* dist2,
                               const som_bmu_opts* opts, void* ws, size_t ws_bytes, hipStream_t stream) {
  return search_impl(W, som::kWeightsF32, F, N, ldw, norms, indptr, indices, B, nnz, perm, bmu, dist, bmu2,
                     dist2, true, opts, ws, ws_bytes, stream);
}

som_status som_bmu_search_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                              const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                              const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                              void* ws, size_t ws_bytes, hipStream_t stream) {
  return search_impl(W, som::kWeightsF16, F, N, ldw, norms, indptr, indices, B, nnz, perm, bmu, dist, nullptr,
                     nullptr, false, opts, ws, ws_bytes, stream);
}

som_status som_bmu_search_top2_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                                   const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                                   const int32_t* perm, int32_t* bmu, float* dist, int32_t* bmu2,
                                   float* dist2, const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  return search_impl(W, som::kWeightsF16, F, N, ldw, norms, indptr, indices, B, nnz, perm, bmu, dist, bmu2,
                     dist2, true, opts, ws, ws_bytes, stream);
}



size_t som_plan_bytes(int64_t B, int64_t nnz, const som_bmu_opts* opts) {
  if (B < 0 || nnz < 0) return 0;
  Plan p;
  const int st = opts_storage(opts);
  if (make_plan(1, B, opts, &p, st, st) != SOM_OK) return 0;
  return plan_layout(p, nnz).total;
}

som_status som_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                    int64_t nnz, const int32_t* perm, const som_bmu_opts* opts, void* plan,
                    size_t plan_bytes, hipStream_t stream) {
  som_status s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  if (opts && opts->validate) return fail(SOM_ERR_INVALID_ARG, "validate applies to som_bmu_search only");
  Plan p;
  const int st = opts_storage(opts);
  s = make_plan(1, B, opts, &p, st, st);
  if (s != SOM_OK) return s;
  const PlanLayout l = plan_layout(p, nnz);
  if (B == 0) return ok();
  if (!plan) return fail(SOM_ERR_WORKSPACE, "plan is NULL");
  if (!aligned(plan, 256)) return fail(SOM_ERR_INVALID_ARG, "plan must be 256-byte aligned");
  if (plan_bytes < l.total)
    return fail(SOM_ERR_WORKSPACE, "plan buffer too small: need " + std::to_string(l.total) + " bytes");
  hipError_t e = build_plan(indptr, indices, B, F, perm, p, plan, l, stream);
  if (e != hipSuccess) return hip_fail(e, "plan launch");
  return ok();
}

size_t som_bmu_search_planned_workspace_bytes(int64_t N, int64_t B, const som_bmu_opts* opts) {
  if (N < 1 || B < 0) return 0;
  Plan p;
  if (make_plan(N, B, opts, &p, opts_storage(opts), opts_storage(opts)) != SOM_OK) return 0;
  return keys_bytes(B);
}

static som_status planned_impl(const void* W, int weights, int64_t F, int64_t N, int64_t ldw,
                               const float* norms, const int32_t* indptr, int64_t B, int64_t nnz,
                               const int32_t* perm, const void* plan, size_t plan_bytes, int32_t* bmu,
                               float* dist, int32_t* bmu2, float* dist2, bool top2, const som_bmu_opts* opts,
                               void* ws, size_t ws_bytes, hipStream_t stream) {
  som_status s = check_codebook(W, weights, F, N, ldw);
  if (s != SOM_OK) return s;
  if (!norms) return fail(SOM_ERR_INVALID_ARG, "norms is NULL");
  if (B < 0 || B >= kI32Max) return fail(SOM_ERR_INVALID_ARG, "B must be in [0, 2^31 - 1)");
  if (nnz < 0 || nnz > kI32Max) return fail(SOM_ERR_INVALID_ARG, "nnz must be in [0, 2^31)");
  if (opts && opts->validate) return fail(SOM_ERR_INVALID_ARG, "validate is not available on a planned search");
  Plan p;
  s = make_plan(N, B, opts, &p, weights, opts_storage(opts));
  if (s != SOM_OK) return s;
  const PlanLayout l = plan_layout(p, nnz);
  if (B == 0) return ok();
  if (!indptr || !bmu || !dist || !plan) return fail(SOM_ERR_INVALID_ARG, "a required pointer is NULL");
  if (top2 && (!bmu2 || !dist2)) return fail(SOM_ERR_INVALID_ARG, "bmu2 or dist2 is NULL");
  if (!aligned(plan, 256)) return fail(SOM_ERR_INVALID_ARG, "plan must be 256-byte aligned");
  if (plan_bytes < l.total)
    return fail(SOM_ERR_INVALID_ARG, "plan buffer smaller than this batch's plan: need " + std::to_string(l.total) + " bytes");
  if (!ws) return fail(SOM_ERR_WORKSPACE, "ws is NULL");
  if (!aligned(ws, 256)) return fail(SOM_ERR_INVALID_ARG, "ws must be 256-byte aligned");
  if (ws_bytes < keys_bytes(B))
    return fail(SOM_ERR_WORKSPACE, "workspace too small: need " + std::to_string(keys_bytes(B)) + " bytes");
  return run_planned(W, weights, F, N, ldw, norms, indptr, B, perm, plan, l, bmu, dist, top2 ? bmu2 : nullptr, dist2,
                     p, static_cast<uint64_t*>(ws), stream);
}

som_status som_bmu_search_planned(const float* W, int64_t F, int64_t N, int64_t ldw,
                                  const float* norms, const int32_t* indptr, int64_t B,
                                  int64_t nnz, const int32_t* perm, const void* plan,
                                  size_t plan_bytes, int32_t* bmu, float* dist,
                                  const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                                  hipStream_t stream) {
  return planned_impl(W, som::kWeightsF32, F, N, ldw, norms, indptr, B, nnz, perm, plan, plan_bytes, bmu, dist,
                      nullptr, nullptr, false, opts, ws, ws_bytes, stream);
}

som_status som_bmu_search_top2_planned(const float* W, int64_t F, int64_t N, int64_t ldw,
                                       const float* norms, const int32_t* indptr, int64_t B,
                                       int64_t nnz, const int32_t* perm, const void* plan,
                                       size_t plan_bytes, int32_t* bmu, float* dist, int32_t* bmu2,
                                       float* dist2, const som_bmu_opts* opts, void* ws,
                                       size_t ws_bytes, hipStream_t stream) {
  return planned_impl(W, som::kWeightsF32, F, N, ldw, norms, indptr, B, nnz, perm, plan, plan_bytes, bmu, dist,
                      bmu2, dist2, true, opts, ws, ws_bytes, stream);
}

som_status som_bmu_search_planned_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw,
                                      const float* norms, const int32_t* indptr, int64_t B,
                                      int64_t nnz, const int32_t* perm, const void* plan,
                                      size_t plan_bytes, int32_t* bmu, float* dist,
                                      const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                                      hipStream_t stream) {
  return planned_impl(W, som::kWeightsF16, F, N, ldw, norms, indptr, B, nnz, perm, plan, plan_bytes, bmu, dist,
                      nullptr, nullptr, false, opts, ws, ws_bytes, stream);
}

som_status som_bmu_search_top2_planned_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw,
                                           const float* norms, const int32_t* indptr, int64_t B,
                                           int64_t nnz, const int32_t* perm, const void* plan,
                                           size_t plan_bytes, int32_t* bmu, float* dist, int32_t* bmu2,
                                           float* dist2, const som_bmu_opts* opts, void* ws,
                                           size_t ws_bytes, hipStream_t stream) {
  return planned_impl(W, som::kWeightsF16, F, N, ldw, norms, indptr, B, nnz, perm, plan, plan_bytes, bmu, dist,
                      bmu2, dist2, true, opts, ws, ws_bytes, stream);
}



som_status som_tile_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                         int64_t nnz, const int32_t* perm, int32_t tile_docs, int32_t* tile_offset,
                         int32_t* tile_count, int32_t* union_feat, uint32_t* union_mask,
                         hipStream_t stream) {
  som_status s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  const int T = tile_docs;
  if (T != 1 && T != 2 && T != 4 && T != 8 && T != 16 && T != 32 && T != 64 && T != 128 && T != 256)
    return fail(SOM_ERR_INVALID_ARG, "tile_docs must be 1, 2, 4, 8, 16, 32, 64, 128 or 256");
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

som_status som_group_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                          int64_t nnz, const int32_t* perm, int32_t group_docs,
                          int32_t* group_offset, int32_t* group_count, int32_t* group_feat,
                          int32_t* entry_pos, hipStream_t stream) {
  som_status s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  if (group_docs < 1 || group_docs > 65536) return fail(SOM_ERR_INVALID_ARG, "group_docs must be in [1, 65536]");
  if ((B + group_docs - 1) / group_docs >= kMaxTiles)
    return fail(SOM_ERR_INVALID_ARG, "batch too large for one launch: too many groups");
  if (B == 0) return ok();
  if (!group_offset || !group_count || (nnz > 0 && (!group_feat || !entry_pos)))
    return fail(SOM_ERR_INVALID_ARG, "an output array is NULL");
  hipError_t e = som::launch_group_plan(indptr, indices, B, F, perm, group_docs, group_offset,
                                        group_count, group_feat, entry_pos, stream);
  if (e != hipSuccess) return hip_fail(e, "group plan launch");
  return ok();
}

size_t som_cluster_workspace_bytes(int64_t B, int64_t F, int64_t nnz) {
  if (B < 0 || F < 1 || nnz < 0 || B >= kI32Max) return 0;
  const int64_t n2 = som::cluster_sort_size(B);
  size_t o = 0;
  take(o, sizeof(int32_t) * F);    // df
  take(o, sizeof(uint64_t) * n2);  // signature keys (padded to a power of two)
  take(o, sizeof(uint32_t) * n2);  // input positions
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
  const int64_t n2 = som::cluster_sort_size(B);
  size_t o = 0;
  const size_t o_df = take(o, sizeof(int32_t) * F);
  const size_t o_keys = take(o, sizeof(uint64_t) * n2);
  const size_t o_vals = take(o, sizeof(uint32_t) * n2);
  hipError_t e = som::launch_cluster(indptr, indices, B, F, nnz, perm, at<int32_t>(ws, o_df),
                                     at<uint64_t>(ws, o_keys), at<uint32_t>(ws, o_vals), stream);
  if (e != hipSuccess) return hip_fail(e, "cluster launch");
  return ok();
}

// ---------------------------------------------------------------------------
// Unfused comparator
// ---------------------------------------------------------------------------

struct UnfusedWs {
  PlanLayout plan;
  size_t score, total;
};

static UnfusedWs unfused_ws(const Plan& p, int64_t N, int64_t nnz, int64_t block_docs) {
  UnfusedWs w{};
  w.plan = plan_layout(p, nnz);
  size_t o = w.plan.total;
  w.score = take(o, sizeof(float) * static_cast<size_t>(block_docs) * static_cast<size_t>(N));
  w.total = o;
  return w;
}

static som_status unfused_plan(int64_t N, int64_t B, const som_bmu_opts* opts, int64_t block_docs, Plan* p) {
  // the comparator is built on kernel 1: the automatic kernel resolves to it
  som_bmu_opts o{};
  if (opts) o = *opts;
  if (o.kernel == 0) o.kernel = 1;
  som_status s = make_plan(N, B, &o, p, som::kWeightsF32, som::kWeightsF32);
  if (s != SOM_OK) return s;
  if (p->kernel != 1) return fail(SOM_ERR_INVALID_ARG, "the unfused comparator uses kernel 1");
  if (o.sweep == 2) return fail(SOM_ERR_INVALID_ARG, "the unfused comparator sweeps in ascending order (sweep 0 or 1)");
  p->rotate = false;  // its block launches cover subsets of the tiles
  if (opts && opts->validate) return fail(SOM_ERR_INVALID_ARG, "validate is not available on the unfused comparator");
  if (block_docs < p->T || block_docs % p->T != 0)
    return fail(SOM_ERR_INVALID_ARG, "block_docs must be a positive multiple of the tile size");
  if (block_docs > (int64_t(1) << 40) / N) return fail(SOM_ERR_INVALID_ARG, "block_docs * N too large");
  return SOM_OK;
}

size_t som_bmu_search_unfused_workspace_bytes(int64_t F, int64_t N, int64_t B, int64_t nnz,
                                              const som_bmu_opts* opts, int64_t block_docs) {
  if (F < 1 || N < 1 || B < 0 || nnz < 0) return 0;
  Plan p;
  if (unfused_plan(N, B, opts, block_docs, &p) != SOM_OK) return 0;
  return unfused_ws(p, N, nnz, block_docs).total;
}

som_status som_bmu_search_unfused(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                                  const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                                  const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                                  int64_t block_docs, void* ws, size_t ws_bytes, hipStream_t stream) {
  som_status s = check_codebook(W, som::kWeightsF32, F, N, ldw);
  if (s != SOM_OK) return s;
  if (!norms) return fail(SOM_ERR_INVALID_ARG, "norms is NULL");
  s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (B > 0 && (!bmu || !dist)) return fail(SOM_ERR_INVALID_ARG, "bmu or dist is NULL");
  Plan p;
  s = unfused_plan(N, B, opts, block_docs, &p);
  if (s != SOM_OK) return s;
  const UnfusedWs w = unfused_ws(p, N, nnz, block_docs);
  if (B == 0) return ok();
  if (!ws) return fail(SOM_ERR_WORKSPACE, "ws is NULL");
  if (!aligned(ws, 256)) return fail(SOM_ERR_INVALID_ARG, "ws must be 256-byte aligned");
  if (ws_bytes < w.total)
    return fail(SOM_ERR_WORKSPACE, "workspace too small: need " + std::to_string(w.total) + " bytes");
  hipError_t e = build_plan(indptr, indices, B, F, perm, p, ws, w.plan, stream);
  if (e != hipSuccess) return hip_fail(e, "plan launch");
  som::SearchArgs a{};
  a.W = W;
  a.weights = som::kWeightsF32;
  a.F = F;
  a.N = N;
  a.ldw = ldw;
  a.norms = norms;
  a.indptr = indptr;
  a.perm = perm;
  a.B = B;
  a.kernel = 1;
  a.T = p.T;
  a.K = p.K;
  a.group = p.group;
  a.mask_mode = p.mask_mode;
  a.chunk_slices = p.chunk_slices;
  a.rotate = p.rotate ? 1 : 0;
  a.ntiles = p.nunits;
  a.nchunks = p.nchunks;
  a.tile_offset = at<int32_t>(ws, w.plan.offset);
  a.tile_count = at<int32_t>(ws, w.plan.count);
  a.union_feat = at<int32_t>(ws, w.plan.feat);
  a.union_mask = at<uint32_t>(ws, w.plan.extra);
  a.score = at<float>(ws, w.score);
  a.bmu = bmu;
  a.dist = dist;
  e = som::launch_unfused(a, block_docs, stream);
  if (e != hipSuccess) return hip_fail(e, "unfused launch");
  return ok();
}

// ---------------------------------------------------------------------------
// Batch-SOM update
// ---------------------------------------------------------------------------

som_status som_update_accumulate(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                                 const int32_t* bmu, int64_t F, int64_t N, uint32_t* acc, int64_t ld_acc,
                                 uint32_t* count, hipStream_t stream) {
  som_status s = check_batch(indptr, indices, B, nnz);
  if (s != SOM_OK) return s;
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  if (N < 1 || N > kI32Max) return fail(SOM_ERR_INVALID_ARG, "N must be in [1, 2^31)");
  if (ld_acc < N) return fail(SOM_ERR_INVALID_ARG, "ld_acc must be >= N");
  if (B == 0) return ok();
  if (!bmu || !acc || !count) return fail(SOM_ERR_INVALID_ARG, "bmu, acc or count is NULL");
  if (!aligned(acc, 4) || !aligned(count, 4)) return fail(SOM_ERR_INVALID_ARG, "acc and count must be 4-byte aligned");
  hipError_t e = som::launch_update_accumulate(indptr, indices, B, bmu, F, N, acc, ld_acc, count, stream);
  if (e != hipSuccess) return hip_fail(e, "accumulate launch");
  return ok();
}

static int update_radius(double sigma) { return sigma > 0 ? static_cast<int>(std::ceil(3.0 * sigma)) : 0; }

struct UpdateWs {
  size_t taps, den_tmp, den, chunk, total;
  int64_t planes;
};

static UpdateWs update_ws(int64_t F, int64_t N) {
  UpdateWs w{};
  size_t o = 0;
  w.taps = take(o, sizeof(float) * (som::kUpdateMaxRadius + 1));
  w.den_tmp = take(o, sizeof(float) * N);
  w.den = take(o, sizeof(float) * N);
  w.planes = static_cast<int64_t>(som::update_chunk_planes(F, N));
  w.chunk = take(o, sizeof(float) * static_cast<size_t>(w.planes) * N);
  w.total = o;
  return w;
}

size_t som_update_workspace_bytes(int64_t F, int64_t N) {
  if (F < 1 || N < 1 || F > kI32Max || N > kI32Max) return 0;
  return update_ws(F, N).total;
}

static som_status finish_impl(void* W, int weights, int64_t F, int64_t ldw, int32_t rows, int32_t cols, double sigma,
                              const uint32_t* acc, int64_t ld_acc, const uint32_t* count, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  if (!W || !acc || !count) return fail(SOM_ERR_INVALID_ARG, "W, acc or count is NULL");
  if (F < 1 || F > kI32Max) return fail(SOM_ERR_INVALID_ARG, "F must be in [1, 2^31)");
  if (rows < 1 || cols < 1 || rows > som::kUpdateMaxRows || cols > som::kUpdateMaxCols)
    return fail(SOM_ERR_INVALID_ARG, "rows must be in [1, 1024] and cols in [1, 16384]");
  const int64_t N = static_cast<int64_t>(rows) * cols;
  if (ldw < N || ld_acc < N) return fail(SOM_ERR_INVALID_ARG, "ldw and ld_acc must be >= rows * cols");
  if (!(sigma >= 0) || !std::isfinite(sigma)) return fail(SOM_ERR_INVALID_ARG, "sigma must be finite and >= 0");
  const int R = sigma * 3.0 > som::kUpdateMaxRadius ? som::kUpdateMaxRadius + 1 : update_radius(sigma);
  if (R > som::kUpdateMaxRadius) return fail(SOM_ERR_INVALID_ARG, "sigma too large: ceil(3 sigma) must be <= 4096");
  if (!aligned(W, weights == som::kWeightsF16 ? 2 : 4) || !aligned(acc, 4) || !aligned(count, 4))
    return fail(SOM_ERR_INVALID_ARG, "W, acc or count misaligned");
  const UpdateWs w = update_ws(F, N);
  if (!ws) return fail(SOM_ERR_WORKSPACE, "ws is NULL");
  if (!aligned(ws, 256)) return fail(SOM_ERR_INVALID_ARG, "ws must be 256-byte aligned");
  if (ws_bytes < w.total)
    return fail(SOM_ERR_WORKSPACE, "workspace too small: need " + std::to_string(w.total) + " bytes");
  hipError_t e = som::launch_update_finish(W, weights, F, ldw, rows, cols, sigma, R, acc, ld_acc, count,
                                           at<float>(ws, w.taps), at<float>(ws, w.den_tmp), at<float>(ws, w.den),
                                           at<float>(ws, w.chunk), w.planes, stream);
  if (e != hipSuccess) return hip_fail(e, "update launch");
  return ok();
}

som_status som_update_finish(float* W, int64_t F, int64_t ldw, int32_t rows, int32_t cols, double sigma,
                             const uint32_t* acc, int64_t ld_acc, const uint32_t* count, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  return finish_impl(W, som::kWeightsF32, F, ldw, rows, cols, sigma, acc, ld_acc, count, ws, ws_bytes, stream);
}

som_status som_update_finish_f16(uint16_t* W, int64_t F, int64_t ldw, int32_t rows, int32_t cols, double sigma,
                                 const uint32_t* acc, int64_t ld_acc, const uint32_t* count, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
  return finish_impl(W, som::kWeightsF16, F, ldw, rows, cols, sigma, acc, ld_acc, count, ws, ws_bytes, stream);
}

som_status som_probe_read(const void* buf, int64_t bytes, int32_t passes, uint32_t* sink, hipStream_t stream) {
  if (!buf || !sink) return fail(SOM_ERR_INVALID_ARG, "buf or sink is NULL");
  if (bytes < 16 || bytes % 16 != 0) return fail(SOM_ERR_INVALID_ARG, "bytes must be a positive multiple of 16");
  if (!aligned(buf, 16) || !aligned(sink, 4)) return fail(SOM_ERR_INVALID_ARG, "buf must be 16-byte aligned");
  if (passes < 1) return fail(SOM_ERR_INVALID_ARG, "passes must be >= 1");
  hipError_t e = som::launch_read_probe(buf, bytes, passes, sink, stream);
  if (e != hipSuccess) return hip_fail(e, "probe launch");
  return ok();
}

som_status som_probe_lds(int32_t iters, uint32_t* sink, int64_t* bytes, hipStream_t stream) {
  if (!sink || !bytes) return fail(SOM_ERR_INVALID_ARG, "sink or bytes is NULL");
  if (!aligned(sink, 4)) return fail(SOM_ERR_INVALID_ARG, "sink must be 4-byte aligned");
  if (iters < 4 || iters % 4 != 0 || iters > (1 << 24))
    return fail(SOM_ERR_INVALID_ARG, "iters must be a multiple of 4 in [4, 2^24]");
  hipError_t e = som::launch_lds_probe(iters, sink, bytes, stream);
  if (e != hipSuccess) return hip_fail(e, "LDS probe launch");
  return ok();
}

}  // extern "C"
