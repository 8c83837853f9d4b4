/*
 * som.h -- C ABI of the best-matching-unit (BMU) search for sparse binary
 * documents against a feature-major codebook, on one AMD Instinct MI355X
 * (gfx950).
 *
 * The search (paper, Section 3 "Background: the design being tuned"): for
 * each document x, a binary vector with feature set S, return the neuron j
 * closest to x in squared Euclidean distance,
 *
 *     d_j = ||x - w_j||^2 = |S| + ||w_j||^2 - 2 * sum_{f in S} W[f][j],
 *
 * with the codebook stored feature-major (each feature's weights contiguous
 * across neurons, W[f * ldw + j]), which turns the search into a tiled
 * sparse-dense product whose argmin is fused into the product (same
 * section).  Ties go to the lowest neuron index.
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers owned by the caller unless stated.  The
 *    library allocates nothing and keeps no pointer after it returns.
 *  - Work is enqueued asynchronously on `stream` (0 = the legacy default
 *    stream); buffers must stay alive until that work completes.
 *  - Argument errors are detected on the host before any HIP call and
 *    return SOM_ERR_INVALID_ARG (or SOM_ERR_WORKSPACE); nothing is enqueued
 *    then.  A failed launch returns SOM_ERR_HIP.  som_last_error() holds a
 *    message for the last failure on the calling thread.
 *  - No entry point throws, aborts or exits.
 *  - Documents are CSR: indptr int32[B+1] with indptr[0] == 0 and
 *    indptr[B] == nnz, indices int32[nnz] strictly ascending within each row
 *    (a binary vector lists each feature once) and in [0, F).  Empty rows
 *    are allowed.  Malformed CSR is undefined behaviour unless
 *    opts->validate is set, in which case it is detected on the device and
 *    reported as SOM_ERR_INVALID_CSR before any search work runs.
 *  - Non-finite weights are undefined behaviour.
 */
#ifndef SOM_H
#define SOM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum som_status {
  SOM_OK = 0,
  SOM_ERR_INVALID_ARG = 1, /* bad size, null pointer, misaligned or bad layout */
  SOM_ERR_INVALID_CSR = 2, /* only with opts->validate: unsorted, duplicate or out-of-range ids */
  SOM_ERR_WORKSPACE = 3,   /* ws too small (see som_*_workspace_bytes) */
  SOM_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
} som_status;

/* Tuning knobs of the search.  A zero-initialised struct (or NULL) selects
 * the defaults.  Only `sweep` changes a result, and only in rounding: with
 * the ascending sweep every document's dot product is summed in ascending
 * feature order whatever the other knobs, so outputs are bit-identical
 * across all their settings and all kernels; the rotated sweep (the default
 * of kernels 1 and 3) sums in a rotated order that is fixed for a given
 * batch, perm, opts and device.
 *
 * Automatic choices (measured on MI355X at map sizes 32^2 to 512^2, F =
 * 2,048 to 20,000, batches up to 1M documents): rotated union sweeps
 * (`sweep`) wherever available; for an fp32 codebook kernel 3 with
 * 64-document super-tiles and the document-major dispatch; for fp16,
 * or when a knob only kernel 1 has is set (tile_docs of 32 or less,
 * lane_neurons, group_tiles), kernel 1 with tiles of 16 documents for fp32
 * and 8 for fp16, and four tiles per workgroup for fp32 tiles of 16
 * documents when N >= 131,072.  The automatic choices depend on the storage
 * type: a search that plans internally uses its own (fp32 or fp16);
 * som_plan, som_plan_bytes and the planned searches use opts->storage, so a
 * plan and its search always agree on the geometry.
 *
 * kernel 1, neurons on lanes: a wave holds a tile of T documents (Section
 *   4.1) against 64*K neurons (K per lane, 128-bit loads, Section 4.3) and
 *   sweeps the tile's union once, adding each row into the documents whose
 *   membership bit is set;
 * kernel 2, documents on lanes: a workgroup holds a group of 64*G documents,
 *   one per lane, against a narrow slice of NB neurons; the group's feature
 *   union (the tile union with a tile of 64*G documents) streams through LDS
 *   and each lane adds the rows of its own document's features;
 * kernel 3, shared-union super-tiles: a workgroup holds a super-tile of D
 *   documents (tile_docs: 64, 128 or 256) against 256 neurons (fp32) or 512
 *   (fp16); the super-tile's union (Section 4.1 with a tile of D documents)
 *   is fetched once per workgroup with 128-bit loads into LDS, and each wave
 *   (8 documents; 16 for D = 256 with an fp32 codebook) adds the rows its
 *   documents hold.
 *   Its plan is the tile plan with D-document tiles (with mask_mode 2, the
 *   default, each 16-entry stage's masks stored document-major); a plan
 *   built with the same tile_docs and mask_mode serves both storage types.
 * Every kernel cuts the neuron axis into slices whose minima are merged
 * (Section 4.2) and fuses the argmin (Section 3). */
typedef struct som_bmu_opts {
  int32_t kernel;        /* 0 = auto (see above), 1 = neurons on lanes, 2 = documents on lanes,
                            3 = shared-union super-tiles */
  int32_t tile_docs;     /* kernel 1: T = 0 (auto: 16 for fp32, 8 for fp16), 1, 2, 4, 8, 16 or 32;
                            kernel 3: D = 0 (auto: 64), 64, 128 or 256 (256: fp32 only) */
  int32_t lane_neurons;  /* kernel 1: K = 0 (auto: 4 for fp32, 8 for fp16), 4 or 8; T = 32 needs 4 */
  int32_t group_tiles;   /* kernel 1: tiles per workgroup, 0 (auto: see above), 1, 2, 4 or 8;
                            kernel 2: waves per workgroup G, 0 (auto), 4, 8 or 16 */
  int32_t mask_mode;     /* kernel 1: 0 = auto, 1 = branch-free multiply by the membership
                            bit, 2 = one scalar branch per document; kernel 3: 0 = auto (2),
                            1 = row-major: one visit per row the wave needs, with a scalar
                            branch tree over the wave's documents, 2 = document-major: per
                            document, the stage entries it holds, read from the plan's
                            per-stage document words */
  int32_t slice_neurons; /* kernel 2: NB = 0 (auto), 32 or 64 */
  int32_t validate;      /* 1 = check the CSR batch on the device first (synchronises `stream`) */
  int32_t storage;       /* 0 = fp32, 1 = fp16: the codebook storage type whose automatic tile
                            size som_plan, som_plan_bytes and the planned searches resolve
                            (searches that plan internally use their own type) */
  int32_t schedule;      /* kernel 3: 0 = auto (1), 1 = one launch over every neuron slice,
                            2 = round-synchronised launches: per slice, one launch per round of
                            as many super-tiles as the device holds at once, so that they sweep
                            their ascending unions side by side; kernels 1 and 2: 0 or 1 */
  int32_t neuron_chunk;  /* kernels 1 and 3 (schedule 1): neurons per schedule chunk (Section 4.2,
                            "Neuron-axis chunking"), 0 = auto (one slice, 64 * K neurons) or a
                            multiple of the slice width.  The launch visits the neuron axis chunk
                            by chunk; inside a chunk each XCD takes its tiles in turn and runs a
                            tile's slices of the chunk back to back.  Chunks wider than the map
                            cover it whole. */
  int32_t sweep;         /* order of each union sweep: 0 = auto (2 where available, else 1),
                            1 = ascending feature order, 2 = rotated (kernel 1, or kernel 3 with
                            mask_mode 2, as one launch of one-slice chunks: schedule 1 and
                            neuron_chunk 0 or one slice; else SOM_ERR_INVALID_ARG): each tile
                            (kernel 3: super-tile) starts its union at an entry (a stage) given
                            by its place in its XCD's share of the launch and wraps round, so
                            that the tiles an XCD runs at once sweep the same feature range
                            together and share its L2 (on the topic workload measured 19%
                            faster with kernel 3 and 17% with fp16 kernel 1; within 1.3% on
                            the Zipf maps).  A document's dot product is then summed in that
                            order, which depends on the plan, the launch's tile grid and the
                            device's CU count, not on the codebook, its storage type or the
                            neuron range: results are reproducible on one device type, fp16
                            and fp32 searches of one plan use the same order, and column
                            ranges compose exactly, but results may differ from the ascending
                            sweep's in the last bits of dist (and, at exact or near ties, in
                            bmu). */
} som_bmu_opts;

/* Version of this ABI (bumped on any incompatible change). */
int32_t som_abi_version(void);

/* Message describing the last failure on the calling thread; never NULL,
 * "" when the last call succeeded.  Valid until the thread's next call. */
const char* som_last_error(void);

/* ||w_j||^2 for j < N (Section 3; the per-epoch "norms" pass of Table 4).
 *   W      fp32 [F][ldw], feature-major, 16-byte aligned, ldw >= N, ldw % 4 == 0
 *   norms  fp32 [N] output: each sum of squares is accumulated in fp64 in a
 *          fixed order and rounded to fp32 once (deterministic).
 * Errors: SOM_ERR_INVALID_ARG for F < 1, N < 1, bad ldw/alignment or NULL. */
som_status som_codebook_norms(const float* W, int64_t F, int64_t N, int64_t ldw, float* norms,
                              hipStream_t stream);

/* Recommended row stride ldw (in floats) of a feature-major codebook of N
 * neurons; host-only, enqueues nothing.  The search reads each feature row
 * in 1 KB slices (256 neurons), the same slice of every row at once.  The L2
 * of each XCD interleaves its 16 channels on 128-byte lines, so with a row
 * stride that is a multiple of 2 KB every row's slice falls on the same 8
 * channels and only half of the L2 holds the slice.  The recommended stride
 * is N rounded up to a multiple of 64 floats (256-byte aligned rows), plus
 * 64 floats when that is a multiple of 512, which rotates consecutive rows
 * across all channels.  Any ldw >= N with ldw % 4 == 0 stays valid; this is
 * a layout choice for speed only.  Returns 0 for N < 1. */
int64_t som_codebook_ldw(int64_t N);

/* Bytes of device workspace som_bmu_search (or som_bmu_search_f16) needs
 * for these sizes and options (0 if the arguments are invalid); with
 * automatic tile sizes it covers both storage types. */
size_t som_bmu_workspace_bytes(int64_t F, int64_t N, int64_t B, int64_t nnz,
                               const som_bmu_opts* opts);

/* BMU of each document of a CSR batch (Section 3; the tiled sweep of Section
 * 4.1, the chunked neuron axis of Section 4.2; the argmin is fused, never
 * materialising the document x neuron score block).
 *   W       fp32 [F][ldw] feature-major codebook (as for som_codebook_norms)
 *   norms   fp32 [N] from som_codebook_norms of the same W
 *   indptr  int32 [B+1], indices int32 [nnz]: the batch (see conventions)
 *   perm    int32 [B] or NULL: tile order.  Position p of the tiled order
 *           holds input document perm[p] (a permutation of 0..B-1, e.g. from
 *           som_cluster_order); NULL = input order.  Results are always in
 *           input order.
 *   bmu     int32 [B] output: argmin_j d_j (lowest index on exact ties)
 *   dist    fp32 [B] output: d_bmu, the squared distance |S| + ||w||^2 - 2 dot
 *           evaluated in fp32 (dot summed in the order opts->sweep names)
 *   ws      device workspace of at least som_bmu_workspace_bytes(...) bytes,
 *           256-byte aligned
 * B == 0 is a valid no-op.  One call is one launch, which takes at most
 * 65,535 neuron slices (N <= 65,535 * 64 * K: 16,776,960 neurons at the fp32
 * default of 4 per lane; kernel 2 slices are opts->slice_neurons wide) and
 * fewer than 2^24 tiles or groups (ceil(B / T)); larger sizes return
 * SOM_ERR_INVALID_ARG: split the batch, or the neuron axis.  No row is read
 * beyond its first round_up(N, 4) elements (8 for fp16), so a column range
 * [r0, r0 + n) of W is searched as W + r0 and norms + r0 with the same ldw
 * and N = n (r0 a multiple of 4, of 8 for fp16).  Adding r0 to bmu and
 * keeping each document's smaller distance, the earlier range's on a tie,
 * gives the whole search's bmu and dist exactly. */
som_status som_bmu_search(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                          const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                          const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                          void* ws, size_t ws_bytes, hipStream_t stream);

/* som_bmu_search without a workspace argument and without any allocation,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The
 * workspace comes from a static device array of SOM_NOALLOC_SCRATCH_BYTES
 * (64 MiB) that each GPU the library runs on holds until the process ends;
 * the call itself allocates nothing and needs
 * som_bmu_workspace_bytes(F, N, B, nnz, opts) <= SOM_NOALLOC_SCRATCH_BYTES
 * (e.g. batches of 65,536 documents of 80 features), else it returns
 * SOM_ERR_INVALID_ARG before any HIP call.  Its first call on a device
 * looks up the array's address there (with that device current).
 * Arguments, results and errors as for som_bmu_search with an fp32
 * codebook; opts->validate must be 0 (validation synchronises).  Every call
 * on one GPU uses that GPU's one array: calls whose work overlaps on a GPU
 * (different streams, or threads) race and must be serialised by the
 * caller; calls in one stream order are safe. */
#define SOM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
som_status som_bmu_search_noalloc(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                                  const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                                  const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                                  hipStream_t stream);

/* Best AND second-best unit of each document in the same fused pass (the
 * paper's kernel keeps the second-best unit because the topographic error,
 * on which both of its stopping rules depend, needs it: Section 6.2, Table 5;
 * Section 7.2, Table 8).  Arguments as for som_bmu_search, plus
 *   bmu2    int32 [B] output: argmin over j != bmu[i] of d_j (lowest index on
 *           exact ties, so with two neurons at the minimum distance, bmu is
 *           the lower and bmu2 the higher index); -1 when N == 1
 *   dist2   fp32 [B] output: d_bmu2 as for dist; +inf when N == 1
 * bmu and dist are identical to som_bmu_search's.  Each neuron slice folds
 * its own two smallest packed keys into the document's (best, second) pair
 * with two 64-bit atomic minima; the pair is exact whatever their order.
 * The workspace size is the same as for som_bmu_search. */
som_status som_bmu_search_top2(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                               const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                               const int32_t* perm, int32_t* bmu, float* dist, int32_t* bmu2,
                               float* dist2, const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/* The two stages of som_bmu_search, for callers that search one batch against
 * several codebook versions (a training loop): the plan depends only on the
 * batch, perm and opts, never on the codebook.
 *   som_plan            builds the plan into `plan` (device memory of at least
 *                       som_plan_bytes(B, nnz, opts) bytes, 256-byte aligned)
 *   som_bmu_search_planned  searches with it; indptr, perm and opts must be those
 *                       the plan was built with, and F at least som_plan's (the
 *                       plan's feature ids index codebook rows unchecked); ws
 *                       holds the per-document
 *                       packed minima, best and second best
 *                       (som_bmu_search_planned_workspace_bytes, 16 B per
 *                       document) */
size_t som_plan_bytes(int64_t B, int64_t nnz, const som_bmu_opts* opts);
som_status som_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                    int64_t nnz, const int32_t* perm, const som_bmu_opts* opts, void* plan,
                    size_t plan_bytes, hipStream_t stream);
size_t som_bmu_search_planned_workspace_bytes(int64_t N, int64_t B, const som_bmu_opts* opts);
som_status som_bmu_search_planned(const float* W, int64_t F, int64_t N, int64_t ldw,
                                  const float* norms, const int32_t* indptr, int64_t B,
                                  int64_t nnz, const int32_t* perm, const void* plan,
                                  size_t plan_bytes, int32_t* bmu, float* dist,
                                  const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                                  hipStream_t stream);
/* som_bmu_search_top2 on a plan from som_plan (same rules as
 * som_bmu_search_planned; the plan does not depend on the top-2 choice). */
som_status som_bmu_search_top2_planned(const float* W, int64_t F, int64_t N, int64_t ldw,
                                       const float* norms, const int32_t* indptr, int64_t B,
                                       int64_t nnz, const int32_t* perm, const void* plan,
                                       size_t plan_bytes, int32_t* bmu, float* dist, int32_t* bmu2,
                                       float* dist2, const som_bmu_opts* opts, void* ws,
                                       size_t ws_bytes, hipStream_t stream);

/* Tile plan of kernel 1 (Section 4.1), written to explicit arrays: for each
 * tile of T consecutive documents of the tiled order (perm as in
 * som_bmu_search; the last tile may be short) the sorted union of their
 * features and, per union entry, a T-bit membership mask (bit s set iff the
 * tile's s-th document contains the feature).  This is also the content of
 * kernel 3's plan (tiles of its D documents).
 *   tile_docs   T in {1, 2, 4, 8, 16, 32, 64, 128, 256}
 *   tile_offset int32 [ntiles+1] output, ntiles = ceil(B / T): tile t's union
 *               is stored at [tile_offset[t], tile_offset[t] + tile_count[t]);
 *               tile_offset[t] is the number of nonzeros of tiles < t
 *   tile_count  int32 [ntiles] output: |U_t|
 *   union_feat  int32 [nnz] output (entries past each tile's count are unused)
 *   union_mask  uint32 [nnz * MW] output, MW = ceil(T / 32) words per entry:
 *               bit s of entry u is bit s % 32 of union_mask[u * MW + s / 32]
 *               (kernel 3's own plan, by default, rearranges these bits per
 *               16-entry stage and document; this entry point writes them
 *               entry by entry)
 * Needs no workspace. */
som_status som_tile_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                         int64_t nnz, const int32_t* perm, int32_t tile_docs, int32_t* tile_offset,
                         int32_t* tile_count, int32_t* union_feat, uint32_t* union_mask,
                         hipStream_t stream);

/* Group plan of kernel 2, written to explicit arrays: for each group of D
 * consecutive documents of the tiled order (the last may be short) the sorted
 * union of their features and, for every nonzero, the position of its feature
 * in its group's union.
 *   group_docs   D, 1 .. 65536
 *   group_offset int32 [ngroups+1] output, ngroups = ceil(B / D) (as tile_offset)
 *   group_count  int32 [ngroups] output: union size
 *   group_feat   int32 [nnz] output: the unions, group g at group_offset[g]
 *   entry_pos    int32 [nnz] output, indexed like `indices`
 * Needs no workspace. */
som_status som_group_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                          int64_t nnz, const int32_t* perm, int32_t group_docs,
                          int32_t* group_offset, int32_t* group_count, int32_t* group_feat,
                          int32_t* entry_pos, hipStream_t stream);

/* Tile-membership clustering (Section 4.2: documents that share descriptors
 * are placed in the same tile, shrinking each tile's union).  The paper
 * gives no algorithm; this is the label-free reading: df(f) = number of
 * documents of the batch containing f; a document's signature is (s1, s2),
 * its two features of highest df (ties to the lower id, F for a missing
 * one); documents are ordered by (s1, s2, input position).
 *   perm  int32 [B] output: perm[p] = input index of the document at position p
 *   ws    at least som_cluster_workspace_bytes(B, F, nnz) bytes
 * Deterministic; B == 0 is a no-op. */
size_t som_cluster_workspace_bytes(int64_t B, int64_t F, int64_t nnz);
som_status som_cluster_order(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                             int64_t nnz, int32_t* perm, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/* ---------------------------------------------------------------------------
 * fp16 codebook storage, fp32 accumulation (the paper's kernel stores two
 * bytes per weight, Section 4.2, and loads them as half-precision pairs,
 * Section 4.3).  W holds IEEE-754
 * binary16 bit patterns, feature-major [F][ldw], 16-byte aligned, with
 * ldw >= N and ldw % 8 == 0 (som_codebook_ldw(N) satisfies both).  Every
 * other argument, output and error is as for the fp32 function of the same
 * name.  The results are those of the fp32 functions on the codebook whose
 * weights are the fp16 values widened exactly to fp32: norms are the rounded
 * weights' norms (fp64 accumulate, rounded once), and every document's dot
 * product sums the widened weights in the order opts->sweep names, so fp16
 * and fp32 searches of the same (fp16-representable) codebook with the same
 * kernel and knobs are bit-identical; across the automatic kernels (3 for
 * fp32, 1 for fp16, both rotating) they are with the ascending sweep
 * (sweep = 1).  Search knobs: kernels 1 (the automatic one for
 * fp16) and 3; lane_neurons 0 or 8 (a 512-neuron slice, one 128-bit load of
 * 8 weights per lane per row); tile_docs up to 16 for kernel 1, 64 or 128
 * for kernel 3.  Plans from som_plan are shared with the fp32 search.
 * ------------------------------------------------------------------------- */
som_status som_codebook_norms_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw, float* norms,
                                  hipStream_t stream);
som_status som_bmu_search_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                              const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                              const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                              void* ws, size_t ws_bytes, hipStream_t stream);
som_status som_bmu_search_top2_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                                   const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                                   const int32_t* perm, int32_t* bmu, float* dist, int32_t* bmu2,
                                   float* dist2, const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                                   hipStream_t stream);
som_status som_bmu_search_planned_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw,
                                      const float* norms, const int32_t* indptr, int64_t B,
                                      int64_t nnz, const int32_t* perm, const void* plan,
                                      size_t plan_bytes, int32_t* bmu, float* dist,
                                      const som_bmu_opts* opts, void* ws, size_t ws_bytes,
                                      hipStream_t stream);
som_status som_bmu_search_top2_planned_f16(const uint16_t* W, int64_t F, int64_t N, int64_t ldw,
                                           const float* norms, const int32_t* indptr, int64_t B,
                                           int64_t nnz, const int32_t* perm, const void* plan,
                                           size_t plan_bytes, int32_t* bmu, float* dist, int32_t* bmu2,
                                           float* dist2, const som_bmu_opts* opts, void* ws,
                                           size_t ws_bytes, hipStream_t stream);

/* Unfused comparator (an ablation, not the method): the same search with the
 * argmin NOT fused into the product, the design the paper's fused kernel is
 * measured against (Section 3: the comparison computes the sparse-dense
 * product, materialises the score block, then reduces it with a separate
 * argmin pass; Section 4.4).  Kernel 1's union sweep writes the distance block
 * of block_docs documents at a time (fp32 [block_docs][N], in ws), then one
 * wave per document reduces its row.  The distances are the fused search's
 * fp32 values, so bmu and dist are bit-identical to som_bmu_search's with the
 * same opts and the ascending sweep (sweep = 1).  Kernel 1 (also when
 * opts->kernel is 0; sweep 0 or 1) and an fp32 codebook
 * only; block_docs a positive multiple of the tile size.  ws: som_bmu_search_unfused_workspace_bytes
 * (plan + score block). */
size_t som_bmu_search_unfused_workspace_bytes(int64_t F, int64_t N, int64_t B, int64_t nnz,
                                              const som_bmu_opts* opts, int64_t block_docs);
som_status som_bmu_search_unfused(const float* W, int64_t F, int64_t N, int64_t ldw, const float* norms,
                                  const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                                  const int32_t* perm, int32_t* bmu, float* dist, const som_bmu_opts* opts,
                                  int64_t block_docs, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Batch-SOM update (the step after the search: the best-matching unit and its
 * neighbours are updated, Section 3; Section 6.1, Table 4 splits it into a
 * scatter into accumulators, a neighbourhood blur, a write-back and a norms
 * refresh).  The paper leaves the neighbourhood function and its schedule to
 * its companion paper; this library's reading is the textbook batch map:
 * neuron j sits at row j / cols, column j % cols of a rows x cols grid; the
 * neighbourhood of width sigma is h(i, j) = exp(-(dr^2 + dc^2) / (2 sigma^2))
 * for |dr| <= R and |dc| <= R, R = ceil(3 sigma), 0 beyond (sigma = 0: h is
 * the identity); an epoch's new codebook is
 *     W[f][j] = sum_i h(i, j) acc[f][i] / sum_i h(i, j) count[i]
 * wherever the denominator is positive, and unchanged elsewhere.
 * ------------------------------------------------------------------------- */

/* Accumulate one searched batch: for every document d with bmu[d] in [0, N),
 * count[bmu[d]] += 1 and acc[f * ld_acc + bmu[d]] += 1 for each of its
 * features f in [0, F) (other ids are ignored).  uint32 atomics: exact and
 * independent of order.  The caller zeroes acc [F][ld_acc] and count [N] at
 * the start of an epoch and calls this once per batch (after the search of
 * that batch, with its bmu output).  B == 0 is a no-op. */
som_status som_update_accumulate(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t nnz,
                                 const int32_t* bmu, int64_t F, int64_t N, uint32_t* acc, int64_t ld_acc,
                                 uint32_t* count, hipStream_t stream);

/* End of an epoch: blur the accumulators over the neighbourhood (separable:
 * a row pass, then a column pass fused with the division) and write the new
 * weights into W [F][ldw] in place (N = rows * cols <= ldw; rows <= 1024,
 * cols <= 16384, sigma finite with ceil(3 sigma) <= 4096).  acc and count are
 * read only.  Sums are fp32 in a fixed tap order (deterministic); the taps
 * are exp() evaluated in fp64 and rounded to fp32 once.  Refresh the norms
 * afterwards with som_codebook_norms[_f16].  ws: som_update_workspace_bytes
 * (F, N) bytes, 256-byte aligned (about 256 MB of it is a chunk of blurred
 * feature planes; the features are processed in chunks). */
size_t som_update_workspace_bytes(int64_t F, int64_t N);
som_status som_update_finish(float* W, int64_t F, int64_t ldw, int32_t rows, int32_t cols, double sigma,
                             const uint32_t* acc, int64_t ld_acc, const uint32_t* count, void* ws,
                             size_t ws_bytes, hipStream_t stream);
/* The same for an fp16 codebook (IEEE binary16 bit patterns; the new weights
 * are rounded to nearest from the fp32 quotient). */
som_status som_update_finish_f16(uint16_t* W, int64_t F, int64_t ldw, int32_t rows, int32_t cols, double sigma,
                                 const uint32_t* acc, int64_t ld_acc, const uint32_t* count, void* ws,
                                 size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Measurement aid: read-bandwidth probe.  Reads `bytes` (a multiple of 16) of
 * device memory at `buf` (16-byte aligned) `passes` times with coalesced
 * 128-bit loads, every workgroup of an XCD re-reading the same part of the
 * buffer (so a buffer of a few MB per XCD is served by the L2s after the
 * first pass, a larger one by the memory-side cache or HBM) and moving to
 * another CU of that XCD between passes (so the vector L1s do not serve the
 * re-reads).  `sink` (4 bytes of device memory) is written only for one
 * value of the folded data; its content is meaningless.  Time the call with
 * events on `stream`: bytes * passes / time is the read rate.  Nothing is
 * allocated; buf is never written.
 * ------------------------------------------------------------------------- */
som_status som_probe_read(const void* buf, int64_t bytes, int32_t passes, uint32_t* sink, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Measurement aid: LDS read probe.  Launches four 512-thread workgroups per
 * CU (the residency of the shared-union search kernel), each holding a 32 KB
 * LDS buffer; every wave reads `iters` 1 KB rows of it (64 lanes x 128 bits,
 * another row each read) and folds each into four adds.  `iters`: a multiple
 * of 4 in [4, 2^24].  `sink` (4 bytes of device memory) is written only for
 * one value of the folded data.  On success `*bytes` (host memory) holds the
 * bytes the launch reads from LDS: time the call with events on `stream`,
 * *bytes / time is the LDS read rate.  Nothing is allocated.
 * ------------------------------------------------------------------------- */
som_status som_probe_lds(int32_t iters, uint32_t* sink, int64_t* bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SOM_H */
