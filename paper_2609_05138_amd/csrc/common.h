// Internal declarations shared by the HIP translation units of libsom.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace som {

// Packed argmin key: the high 32 bits are the distance mapped to an unsigned
// integer whose order matches the float order, the low 32 bits the neuron
// index.  The unsigned 64-bit minimum of two keys is then the smaller
// distance, and on equal distances the lower index -- associative and
// commutative, so the reduction order never changes the answer.
__device__ __forceinline__ uint32_t ordered_bits(float d) {
  uint32_t u = __float_as_uint(d);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_ordered_bits(uint32_t u) {
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u);
}

__device__ __forceinline__ uint64_t pack_key(float d, uint32_t j) {
  return (static_cast<uint64_t>(ordered_bits(d)) << 32) | j;
}

constexpr uint64_t kNoKey = ~0ull;

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------------------
// Launchers (each enqueues on `stream` and returns the launch status).
// ---------------------------------------------------------------------------

// Codebook storage types (SearchArgs::weights, launch_norms).
constexpr int kWeightsF32 = 0;
constexpr int kWeightsF16 = 1;

hipError_t launch_norms(const void* W, int weights, int64_t F, int64_t N, int64_t ldw, float* norms,
                        hipStream_t stream);

// CSR (and optional permutation) checks; sets *flag (device int) nonzero on failure.
hipError_t launch_validate(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                           int64_t nnz, const int32_t* perm, int32_t* seen, int32_t* flag,
                           hipStream_t stream);

// Tile plan: tile_offset[ntiles+1] (exclusive scan of per-tile nonzeros),
// tile_count[ntiles], union_feat / union_mask (see som_tile_plan).  With
// stage_masks (tiles of 64, 128 or 256 documents: the shared-union search's
// document-major form) each tile's region is rounded up to whole 16-entry
// stages and each stage's masks are stored document-major: 16-bit word s of
// the stage (at the stage's first mask word) holds bit r set iff document s
// holds entry r of the stage.
hipError_t launch_tile_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                            const int32_t* perm, int T, int32_t* tile_offset, int32_t* tile_count,
                            int32_t* union_feat, uint32_t* union_mask, hipStream_t stream,
                            bool stage_masks = false);

// Document-group plan (for the documents-on-lanes search): per group of D
// consecutive documents of the tiled order, the sorted feature union and the
// union position of every nonzero.
hipError_t launch_group_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                             const int32_t* perm, int D, int32_t* group_offset, int32_t* group_count,
                             int32_t* group_feat, int32_t* entry_pos, hipStream_t stream);

// Block index -> (tile or tile-group index, neuron slice) of a kernel-1/3
// launch over a grid of nx (a multiple of 8) x nslices workgroups, dealt to
// the XCDs round-robin in linear order.  XCD x owns the contiguous tile range
// [x * nx/8, (x+1) * nx/8); it visits the neuron slices in chunks of q, and
// inside a chunk its tiles in turn with the chunk's slices back to back (the
// last chunk may hold fewer than q slices).  q = 1 is slice-major order.
__host__ __device__ inline void chunked_block(uint64_t lin, uint64_t nx, uint64_t nslices, uint64_t q,
                                              uint64_t* unit, uint64_t* slice) {
  const uint64_t xcd = lin % 8, j = lin / 8, per = nx / 8;
  const uint64_t full = nslices / q, rest = nslices - full * q;
  const uint64_t chunk = j / (per * q);
  const uint64_t r = chunk < full ? j - chunk * per * q : j - full * per * q;
  const uint64_t qq = chunk < full ? q : rest;
  *unit = xcd * per + r / qq;
  *slice = chunk * q + r % qq;
}

// Phase periods of the rotated sweeps (see search.hip): kernel 3 with
// super-tiles of S waves of T documents, in workgroups per XCD; kernel 1
// with T-document tiles, G per workgroup, in tiles per XCD.
hipError_t st_phase_wgs(int T, int S, int32_t* wgs);
hipError_t k1_phase_tiles(int T, int G, int mask_mode, int32_t* tiles);

struct SearchArgs {
  const void* W;    // fp32 or fp16 [F][ldw] (see `weights`)
  int weights;      // kWeightsF32 or kWeightsF16 (kernel 1 only)
  int64_t F, N, ldw;
  const float* norms;
  const int32_t* indptr;
  const int32_t* perm;
  int64_t B;
  int T;            // documents per tile (kernel 3: per wave)
  int K;            // neurons per lane (4 or 8); a slice is 64 * K neurons
  int group;        // tiles (waves) per workgroup, all on the same slice
                    // (kernel 3: waves per super-tile of group * T documents)
  int mask_mode;    // 0 = branch-free fma by the membership bit, 1 = scalar branches
  int64_t ntiles;
  int64_t nchunks;  // neuron slices = ceil(N / (64 * K))
  int64_t tile_base = 0;  // kernel 1 searches tiles [tile_base, tile_end) of the plan
  int64_t tile_end = 0;
  // kernel 3, round-synchronised launches (round_wgs > 0): one launch per
  // (neuron slice, round); XCD x searches super-tiles x * xcd_span +
  // round_base + [0, round_wgs) of slice slice_base
  int32_t schedule = 0;   // 1 = one launch over every slice, 2 = rounds
  int32_t round_wgs = 0;
  int64_t round_base = 0;
  int64_t xcd_span = 0;
  int64_t slice_base = 0;
  // kernels 1 and 3 (one launch over every slice): neuron slices per schedule
  // chunk; the grid's workgroups walk the chunks in turn, and inside a chunk
  // each XCD's tiles with their chunk slices back to back (1 = slice-major)
  int32_t chunk_slices = 1;
  // kernels 1 and 3 (one launch of one-slice chunks; kernel 3
  // document-major): 1 = rotated sweep; phase_wgs is its phase period, in
  // workgroups (kernel 3) or tiles (kernel 1) per XCD, set by the launch
  int32_t rotate = 0;
  int32_t phase_wgs = 0;
  float* score = nullptr;  // unfused comparator: distances of tiled-order documents
                           // [tile_base * T, ...) go to score[(p - tile_base * T) * N + j]
  const int32_t* tile_offset;
  const int32_t* tile_count;
  const int32_t* union_feat;
  const uint32_t* union_mask;
  uint64_t* keys;   // [B] packed (distance, index) minima, tiled order
  uint64_t* keys2;  // [B] second-smallest keys, or nullptr when only the BMU is wanted
  // documents-on-lanes search (kernel 2)
  int kernel;       // 1 = neurons on lanes (tile masks), 2 = documents on lanes (groups),
                    // 3 = shared-union super-tiles (tile plan with group * T / 32 mask words)
  int slice;        // kernel 2: neurons per slice (32 or 64)
  const int32_t* group_offset;
  const int32_t* group_count;
  const int32_t* group_feat;
  const int32_t* entry_pos;
  int32_t* bmu;
  float* dist;
  int32_t* bmu2;    // with keys2: second-best unit (-1 if none) and its distance (+inf)
  float* dist2;
};

hipError_t launch_search(const SearchArgs& a, hipStream_t stream);
// Kernels 1 and 3 over an fp16 codebook (their own translation unit).
hipError_t launch_search_k1_f16(const SearchArgs& a, hipStream_t stream);
hipError_t launch_search_st_f16(const SearchArgs& a, hipStream_t stream);
// Unfused comparator: kernel 1 writes the distance block of block_docs
// documents at a time into `score`, then a wave-per-row argmin reduces it.
hipError_t launch_unfused(SearchArgs a, int64_t block_docs, hipStream_t stream);
// Initialises the keys, then runs the fused search; launch_merge decodes the
// keys into results in input order.
hipError_t launch_merge(const SearchArgs& a, hipStream_t stream);

// Batch-SOM update (update.hip).
constexpr int kUpdateMaxRows = 1024;   // column-blur strip: rows x 32 fp32 in LDS
constexpr int kUpdateMaxCols = 16384;  // row blur: one grid row in LDS
constexpr int kUpdateMaxRadius = 4096;
size_t update_chunk_planes(int64_t F, int64_t N);
hipError_t launch_update_accumulate(const int32_t* indptr, const int32_t* indices, int64_t B, const int32_t* bmu,
                                    int64_t F, int64_t N, uint32_t* acc, int64_t ld_acc, uint32_t* count,
                                    hipStream_t stream);
hipError_t launch_update_finish(void* W, int weights, int64_t F, int64_t ldw, int rows, int cols, double sigma, int R,
                                const uint32_t* acc, int64_t ld_acc, const uint32_t* count, float* taps,
                                float* den_tmp, float* den, float* chunk, int64_t chunk_planes,
                                hipStream_t stream);

// Read-bandwidth probe (probe.hip): `passes` grid-stride reads of buf.
hipError_t launch_read_probe(const void* buf, int64_t bytes, int32_t passes, uint32_t* sink, hipStream_t stream);
hipError_t launch_lds_probe(int32_t iters, uint32_t* sink, int64_t* bytes, hipStream_t stream);

// Clustering: df histogram, signatures and a bitonic sort of n2 =
// cluster_sort_size(B) (a power of two >= B) (key, position) pairs.
int64_t cluster_sort_size(int64_t B);
hipError_t launch_cluster(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                          int64_t nnz, int32_t* perm, int32_t* df, uint64_t* keys, uint32_t* vals,
                          hipStream_t stream);

}  // namespace som
