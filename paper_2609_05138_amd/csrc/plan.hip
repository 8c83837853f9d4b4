// Tile plan (paper, Section 4.1): a tile of T documents forms the sorted
// union of the distinct features its documents contain, so that each union
// feature's codebook row is swept once for the whole tile.  Per union entry
// the plan also records a T-bit membership mask (bit s: the tile's s-th
// document contains the feature), which the search uses to add the row only
// into the accumulators of the documents that hold it.
//
// Layout produced (all int32 unless noted):
//   tile_offset[t]  = number of nonzeros in tiles < t (exclusive scan); the
//                     union of tile t is stored from there, and since
//                     |U_t| <= nnz(t) it never overlaps tile t + 1
//   tile_count[t]   = |U_t|
//   union_feat[.]   = ascending feature ids, union_mask[. * MW + w] (uint32)
//                     = word w of the entry's mask
//
// Construction: one workgroup per tile marks a bitmap of T-bit masks indexed
// by feature (a window of up to 32768 / MW features in LDS), then compacts the
// nonzero entries in ascending order with a workgroup prefix sum.  Integer
// work, bit-exact by construction.
#include "common.h"

namespace som {
namespace {

constexpr int kPlanThreads = 256;
constexpr int kPlanWindow = 32768;  // features per LDS window (128 KB of masks)

__device__ __forceinline__ int64_t tile_doc(const int32_t* perm, int64_t p) {
  return perm ? static_cast<int64_t>(perm[p]) : p;
}

// Nonzeros of each tile, rounded up to a multiple of `round` (the space a
// tile's union may take: |U_t| <= nnz(t)).
__global__ void __launch_bounds__(256)
k_tile_nnz(const int32_t* __restrict__ indptr, const int32_t* __restrict__ perm, int64_t B, int T,
           int64_t ntiles, int32_t* __restrict__ tile_nnz, int round) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= ntiles) return;
  int32_t s = 0;
  for (int k = 0; k < T; ++k) {
    const int64_t p = t * T + k;
    if (p < B) {
      const int64_t d = tile_doc(perm, p);
      s += indptr[d + 1] - indptr[d];
    }
  }
  tile_nnz[t] = (s + round - 1) / round * round;
}

// Exclusive scan of n values in place into out[0..n] (out[n] = total), one
// workgroup of 1024 threads; each thread scans a contiguous run.
__global__ void __launch_bounds__(1024)
k_scan(const int32_t* __restrict__ in, int64_t n, int32_t* __restrict__ out) {
  __shared__ int32_t sums[1024];
  const int tid = threadIdx.x;
  const int64_t per = (n + 1023) / 1024;
  const int64_t a = tid * per;
  const int64_t b = a + per < n ? a + per : n;
  int32_t s = 0;
  for (int64_t i = a; i < b; ++i) s += in[i];
  sums[tid] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int32_t v = tid >= off ? sums[tid - off] : 0;
    __syncthreads();
    sums[tid] += v;
    __syncthreads();
  }
  int32_t run = tid ? sums[tid - 1] : 0;
  for (int64_t i = a; i < b; ++i) {
    const int32_t v = in[i];
    out[i] = run;
    run += v;
  }
  if (tid == 1023) out[n] = sums[1023];
}

// Workgroup exclusive prefix sum of one value per thread (256 threads).
__device__ int32_t block_exclusive_scan(int32_t v, int32_t* tmp, int32_t* total) {
  const int tid = threadIdx.x;
  tmp[tid] = v;
  __syncthreads();
  for (int off = 1; off < kPlanThreads; off <<= 1) {
    const int32_t x = tid >= off ? tmp[tid - off] : 0;
    __syncthreads();
    tmp[tid] += x;
    __syncthreads();
  }
  const int32_t incl = tmp[tid];
  *total = tmp[kPlanThreads - 1];
  __syncthreads();
  return incl - v;
}

__global__ void __launch_bounds__(kPlanThreads)
k_plan(const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
       const int32_t* __restrict__ perm, int64_t B, int64_t F, int T, int MW, int window,
       const int32_t* __restrict__ tile_offset, int32_t* __restrict__ tile_count,
       int32_t* __restrict__ union_feat, uint32_t* __restrict__ union_mask) {
  extern __shared__ uint32_t bits[];  // [window][MW]
  __shared__ int32_t tmp[kPlanThreads];
  const int tid = threadIdx.x;
  const int64_t t = blockIdx.x;
  const int64_t out0 = tile_offset[t];
  int32_t written = 0;
  for (int64_t w0 = 0; w0 < F; w0 += window) {
    const int wlen = static_cast<int>(F - w0 < window ? F - w0 : window);
    for (int i = tid; i < wlen * MW; i += kPlanThreads) bits[i] = 0u;
    __syncthreads();
    for (int k = 0; k < T; ++k) {
      const int64_t p = t * T + k;
      if (p >= B) break;
      const int64_t d = tile_doc(perm, p);
      const int32_t a = indptr[d], b = indptr[d + 1];
      for (int32_t i = a + tid; i < b; i += kPlanThreads) {
        const int64_t f = indices[i];
        if (f >= w0 && f < w0 + wlen) atomicOr(&bits[(f - w0) * MW + (k >> 5)], 1u << (k & 31));
      }
    }
    __syncthreads();
    // each thread compacts a contiguous run of the window, in order
    const int per = (wlen + kPlanThreads - 1) / kPlanThreads;
    const int a = tid * per;
    const int b = a + per < wlen ? a + per : wlen;
    int32_t cnt = 0;
    for (int i = a; i < b; ++i) {
      uint32_t any = 0u;
      for (int w = 0; w < MW; ++w) any |= bits[i * MW + w];
      cnt += any != 0u;
    }
    int32_t total;
    int32_t pos = block_exclusive_scan(cnt, tmp, &total);
    for (int i = a; i < b; ++i) {
      uint32_t any = 0u;
      for (int w = 0; w < MW; ++w) any |= bits[i * MW + w];
      if (any) {
        const int64_t o = out0 + written + pos;
        union_feat[o] = static_cast<int32_t>(w0 + i);
        for (int w = 0; w < MW; ++w) union_mask[o * MW + w] = bits[i * MW + w];
        ++pos;
      }
    }
    written += total;
    __syncthreads();
  }
  if (tid == 0) tile_count[t] = written;
}

// Document-group plan: a group is D consecutive documents of the tiled
// order.  For each group: the sorted union of its features (group_feat, at
// group_offset[g], group_count[g] entries) and, for every nonzero of its
// documents, the position of that nonzero's feature inside the group's union
// (entry_pos, indexed like `indices`).  Positions increase along a document
// because both its features and the union are sorted.
__global__ void __launch_bounds__(kPlanThreads)
k_gplan(const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
        const int32_t* __restrict__ perm, int64_t B, int64_t F, int D, int window,
        const int32_t* __restrict__ group_offset, int32_t* __restrict__ group_count,
        int32_t* __restrict__ group_feat, int32_t* __restrict__ entry_pos) {
  extern __shared__ uint32_t rank[];  // [window]: 0 = absent, else 1 + union position
  __shared__ int32_t tmp[kPlanThreads];
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  constexpr int kWaves = kPlanThreads / 64;
  const int64_t g = blockIdx.x;
  const int64_t out0 = group_offset[g];
  int32_t written = 0;
  for (int64_t w0 = 0; w0 < F; w0 += window) {
    const int wlen = static_cast<int>(F - w0 < window ? F - w0 : window);
    for (int i = tid; i < wlen; i += kPlanThreads) rank[i] = 0u;
    __syncthreads();
    for (int k = wave; k < D; k += kWaves) {
      const int64_t p = g * D + k;
      if (p >= B) break;
      const int64_t d = tile_doc(perm, p);
      for (int32_t i = indptr[d] + lane; i < indptr[d + 1]; i += 64) {
        const int64_t f = indices[i];
        if (f >= w0 && f < w0 + wlen) rank[f - w0] = 1u;
      }
    }
    __syncthreads();
    const int per = (wlen + kPlanThreads - 1) / kPlanThreads;
    const int a = tid * per;
    const int b = a + per < wlen ? a + per : wlen;
    int32_t cnt = 0;
    for (int i = a; i < b; ++i) cnt += rank[i] != 0u;
    int32_t total;
    int32_t pos = block_exclusive_scan(cnt, tmp, &total);
    for (int i = a; i < b; ++i) {
      if (rank[i]) {
        const int32_t at = written + pos;
        group_feat[out0 + at] = static_cast<int32_t>(w0 + i);
        rank[i] = static_cast<uint32_t>(at) + 1u;
        ++pos;
      }
    }
    __syncthreads();
    for (int k = wave; k < D; k += kWaves) {
      const int64_t p = g * D + k;
      if (p >= B) break;
      const int64_t d = tile_doc(perm, p);
      for (int32_t i = indptr[d] + lane; i < indptr[d + 1]; i += 64) {
        const int64_t f = indices[i];
        if (f >= w0 && f < w0 + wlen) entry_pos[i] = static_cast<int32_t>(rank[f - w0]) - 1;
      }
    }
    written += total;
    __syncthreads();
  }
  if (tid == 0) group_count[g] = written;
}

// CSR checks: rows non-decreasing in indptr, ids in [0, F) and strictly
// ascending within a row; optional permutation must hit every index once.
__global__ void __launch_bounds__(256)
k_validate(const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices, int64_t B,
           int64_t F, int64_t nnz, const int32_t* __restrict__ perm, int32_t* __restrict__ seen,
           int32_t* __restrict__ flag) {
  const int64_t d = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (d == 0 && (indptr[0] != 0 || indptr[B] != nnz)) atomicOr(flag, 1);
  if (d >= B) return;
  const int32_t a = indptr[d], b = indptr[d + 1];
  if (a > b || a < 0 || b > nnz) {
    atomicOr(flag, 2);
    return;
  }
  int64_t prev = -1;
  for (int32_t i = a; i < b; ++i) {
    const int64_t f = indices[i];
    if (f < 0 || f >= F || f <= prev) {
      atomicOr(flag, 4);
      break;
    }
    prev = f;
  }
  if (perm) {
    const int64_t q = perm[d];
    if (q < 0 || q >= B) {
      atomicOr(flag, 8);
    } else if (atomicAdd(&seen[q], 1) != 0) {
      atomicOr(flag, 16);
    }
  }
}

// Stage masks of the shared-union search: each tile's union (its region
// rounded up to whole stages of kStage entries) is cut into stages, and the
// stage's kStage x T membership bits are rewritten in place from entry-major
// (entry u: MW words, bit s = document s) to document-major (document s: one
// 16-bit word, bit r = entry r of the stage; entries past |U_t| are empty).
// Both forms take 16 * MW words.  One workgroup of T threads per tile, one
// document per thread; the stage's words pass through LDS, so every read of
// a stage precedes its rewrite.
constexpr int kStage = 16;

__global__ void __launch_bounds__(256)
k_stage_masks(const int32_t* __restrict__ tile_offset, const int32_t* __restrict__ tile_count, int T,
              uint32_t* __restrict__ union_mask) {
  __shared__ uint32_t blk[kStage * 8];  // kStage entries x at most 8 words
  const int MW = T / 32;
  const int d = threadIdx.x;
  const int64_t t = blockIdx.x;
  const int64_t u0 = tile_offset[t];
  const int32_t cnt = tile_count[t];
  for (int32_t g = 0; g * kStage < cnt; ++g) {
    uint32_t* m = union_mask + (u0 + static_cast<int64_t>(g) * kStage) * MW;
    for (int i = d; i < kStage * MW; i += T) blk[i] = g * kStage + i / MW < cnt ? m[i] : 0u;
    __syncthreads();
    uint32_t word = 0u;
#pragma unroll
    for (int r = 0; r < kStage; ++r) word |= ((blk[r * MW + (d >> 5)] >> (d & 31)) & 1u) << r;
    reinterpret_cast<uint16_t*>(m)[d] = static_cast<uint16_t>(word);
    __syncthreads();
  }
}

__global__ void k_fill_i32(int32_t* __restrict__ p, int64_t n, int32_t v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

}  // namespace

hipError_t launch_group_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                             const int32_t* perm, int D, int32_t* group_offset, int32_t* group_count,
                             int32_t* group_feat, int32_t* entry_pos, hipStream_t stream) {
  const int64_t ngroups = (B + D - 1) / D;
  hipLaunchKernelGGL(k_tile_nnz, dim3(static_cast<uint32_t>((ngroups + 255) / 256)), dim3(256), 0,
                     stream, indptr, perm, B, D, ngroups, group_count, 1);
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, stream, group_count, ngroups, group_offset);
  const int window = static_cast<int>(F < kPlanWindow ? F : kPlanWindow);
  const size_t lds = sizeof(uint32_t) * static_cast<size_t>(window);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_gplan),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_gplan, dim3(static_cast<uint32_t>(ngroups)), dim3(kPlanThreads), lds, stream,
                     indptr, indices, perm, B, F, D, window, group_offset, group_count, group_feat,
                     entry_pos);
  return hipGetLastError();
}

hipError_t launch_validate(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                           int64_t nnz, const int32_t* perm, int32_t* seen, int32_t* flag,
                           hipStream_t stream) {
  hipLaunchKernelGGL(k_fill_i32, dim3(1), dim3(64), 0, stream, flag, int64_t(1), 0);
  if (perm) {
    hipLaunchKernelGGL(k_fill_i32, dim3(static_cast<uint32_t>((B + 255) / 256)), dim3(256), 0,
                       stream, seen, B, 0);
  }
  const int64_t groups = (B + 255) / 256;
  hipLaunchKernelGGL(k_validate, dim3(static_cast<uint32_t>(groups > 0 ? groups : 1)), dim3(256),
                     0, stream, indptr, indices, B, F, nnz, perm, seen, flag);
  return hipGetLastError();
}

hipError_t launch_tile_plan(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                            const int32_t* perm, int T, int32_t* tile_offset, int32_t* tile_count,
                            int32_t* union_feat, uint32_t* union_mask, hipStream_t stream, bool stage_masks) {
  const int64_t ntiles = (B + T - 1) / T;
  if (stage_masks && (T < 64 || T > 256 || T % 32 != 0)) return hipErrorInvalidValue;
  // per-tile nonzeros are staged in tile_count, then scanned into tile_offset
  hipLaunchKernelGGL(k_tile_nnz, dim3(static_cast<uint32_t>((ntiles + 255) / 256)), dim3(256), 0,
                     stream, indptr, perm, B, T, ntiles, tile_count, stage_masks ? kStage : 1);
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, stream, tile_count, ntiles, tile_offset);
  const int MW = (T + 31) / 32;
  const int window = static_cast<int>(F < kPlanWindow / MW ? F : kPlanWindow / MW);
  const size_t lds = sizeof(uint32_t) * static_cast<size_t>(window) * MW;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_plan),
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     static_cast<int>(lds));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_plan, dim3(static_cast<uint32_t>(ntiles)), dim3(kPlanThreads), lds, stream,
                     indptr, indices, perm, B, F, T, MW, window, tile_offset, tile_count, union_feat,
                     union_mask);
  if (stage_masks)
    hipLaunchKernelGGL(k_stage_masks, dim3(static_cast<uint32_t>(ntiles)), dim3(static_cast<uint32_t>(T)), 0,
                       stream, tile_offset, tile_count, T, union_mask);
  return hipGetLastError();
}

}  // namespace som
