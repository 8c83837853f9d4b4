// Tile-membership clustering (paper, Section 4.2): place documents that
// share descriptors in the same tile so that each tile's feature union
// shrinks.  The paper gives no algorithm; this is a label-free reading:
//   df(f)  = number of documents of the batch containing f
//   (s1,s2)= a document's two features of highest df (ties to the lower id;
//            F stands in for a missing feature)
//   order  = the documents sorted by (s1, s2, input position).
// Integer work; deterministic.  Every kernel here is the library's own: an
// LDS-windowed df histogram, one signature per document, and a bitonic
// sorting network over (signature, input position) pairs.  Since the input
// position makes every pair distinct, the network's (unstable) sort yields
// exactly the stable order by signature.
#include "common.h"

namespace som {
namespace {

constexpr int kHistWindow = 32768;   // features per LDS histogram window (128 KB)
constexpr int kHistItems = 1 << 18;  // indices per workgroup

__global__ void __launch_bounds__(256)
k_df_lds(const int32_t* __restrict__ indices, int64_t nnz, int64_t w0, int wlen, int32_t* __restrict__ df) {
  __shared__ int32_t h[kHistWindow];
  for (int i = threadIdx.x; i < wlen; i += 256) h[i] = 0;
  __syncthreads();
  const int64_t a = static_cast<int64_t>(blockIdx.x) * kHistItems;
  const int64_t b = a + kHistItems < nnz ? a + kHistItems : nnz;
  for (int64_t i = a + threadIdx.x; i < b; i += 256) {
    const int64_t f = indices[i] - w0;
    if (f >= 0 && f < wlen) atomicAdd(&h[f], 1);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < wlen; i += 256)
    if (h[i]) atomicAdd(&df[w0 + i], h[i]);
}

__global__ void k_zero_i32(int32_t* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// Signature key of each document at position d < B: key (s1 << bits) | s2,
// value d; positions B .. n2-1 are padding that sorts after every document.
// kSigLanes lanes share a document: each keeps the top two of its share of
// the features under the order (df descending, id ascending), packed as
// ((df + 1) << 32) | ~id so that the larger key ranks first (0 = none), and
// the lanes merge their pairs with shuffles.  Features of a document are
// distinct, so no two non-empty keys are equal and the merge is exact.
constexpr int kSigLanes = 8;

__global__ void __launch_bounds__(256)
k_signature(const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices, int64_t B, int64_t n2,
            int64_t F, int bits, const int32_t* __restrict__ df, uint64_t* __restrict__ keys,
            uint32_t* __restrict__ vals) {
  const int64_t d = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kSigLanes;
  const int sub = threadIdx.x & (kSigLanes - 1);
  if (d >= n2) return;   // a document's lanes leave together
  if (d >= B) {
    if (sub == 0) {
      keys[d] = ~0ull;
      vals[d] = 0xffffffffu;
    }
    return;
  }
  uint64_t k1 = 0, k2 = 0;
  const int32_t e = indptr[d + 1];
  for (int32_t i = indptr[d] + sub; i < e; i += kSigLanes) {
    const uint32_t f = static_cast<uint32_t>(indices[i]);
    const uint64_t k = (static_cast<uint64_t>(df[f] + 1) << 32) | (0xffffffffu - f);
    if (k > k1) {
      k2 = k1;
      k1 = k;
    } else if (k > k2) {
      k2 = k;
    }
  }
#pragma unroll
  for (int off = 1; off < kSigLanes; off <<= 1) {
    const uint64_t o1 = (static_cast<uint64_t>(__shfl_xor(static_cast<uint32_t>(k1 >> 32), off, kSigLanes)) << 32) |
                        __shfl_xor(static_cast<uint32_t>(k1), off, kSigLanes);
    const uint64_t o2 = (static_cast<uint64_t>(__shfl_xor(static_cast<uint32_t>(k2 >> 32), off, kSigLanes)) << 32) |
                        __shfl_xor(static_cast<uint32_t>(k2), off, kSigLanes);
    // top two of two ranked pairs: the larger first, then the larger of the
    // smaller first and both seconds
    const uint64_t hi = k1 > o1 ? k1 : o1;
    const uint64_t lo = k1 > o1 ? o1 : k1;
    const uint64_t s = k2 > o2 ? k2 : o2;
    k1 = hi;
    k2 = lo > s ? lo : s;
  }
  if (sub == 0) {
    const int64_t s1 = k1 ? static_cast<int64_t>(0xffffffffu - static_cast<uint32_t>(k1)) : F;
    const int64_t s2 = k2 ? static_cast<int64_t>(0xffffffffu - static_cast<uint32_t>(k2)) : F;
    keys[d] = (static_cast<uint64_t>(s1) << bits) | static_cast<uint64_t>(s2);
    vals[d] = static_cast<uint32_t>(d);
  }
}

int key_bits(int64_t F) {
  int b = 1;
  while ((int64_t(1) << b) <= F) ++b;  // values 0..F inclusive
  return b;
}

// ---------------------------------------------------------------------------
// Bitonic sort of n2 (a power of two) pairs (key, val), ascending in the
// pair order.  Step (k, j) compares element i with i ^ j for every i whose
// bit j is clear, in ascending direction when bit k of i is clear and
// descending otherwise; k runs over 2, 4, .., n2 and, for each k, j over
// k/2, k/4, .., 1.  Steps with j < kLocal stay inside aligned blocks of
// kLocal elements and run in LDS (one launch for a run of them); wider
// steps run over global memory, up to three of them per launch.
// ---------------------------------------------------------------------------
constexpr int kLocal = 2048;           // elements per LDS block
constexpr int kLocalThreads = kLocal / 2;

__device__ __forceinline__ bool pair_greater(uint64_t ka, uint32_t va, uint64_t kb, uint32_t vb) {
  return ka > kb || (ka == kb && va > vb);
}

// Steps (k, j) for k = k_lo .. k_hi and, for each k, j from (k == k_lo ?
// j_first : k/2) down to 1, on blocks of `blk` elements (blk = min(kLocal,
// n2), blk / 2 threads per block, one compared pair per thread and step).
__global__ void __launch_bounds__(kLocalThreads)
k_bitonic_local(uint64_t* __restrict__ keys, uint32_t* __restrict__ vals, int64_t blk, int64_t k_lo, int64_t k_hi,
                int64_t j_first) {
  __shared__ uint64_t sk[kLocal];
  __shared__ uint32_t sv[kLocal];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * blk;
  const int t = threadIdx.x;
  for (int64_t i = t; i < blk; i += blockDim.x) {
    sk[i] = keys[base + i];
    sv[i] = vals[base + i];
  }
  __syncthreads();
  for (int64_t k = k_lo; k <= k_hi; k <<= 1) {
    for (int64_t j = (k == k_lo ? j_first : k >> 1); j > 0; j >>= 1) {
      // thread t's pair: insert a clear bit j into t (j is a power of two)
      const int64_t i = ((t & ~(j - 1)) << 1) | (t & (j - 1));
      const int64_t l = i + j;
      const bool asc = ((base + i) & k) == 0;
      const uint64_t ka = sk[i], kb = sk[l];
      const uint32_t va = sv[i], vb = sv[l];
      if (pair_greater(ka, va, kb, vb) == asc) {
        sk[i] = kb;
        sv[i] = vb;
        sk[l] = ka;
        sv[l] = va;
      }
      __syncthreads();
    }
  }
  for (int64_t i = t; i < blk; i += blockDim.x) {
    keys[base + i] = sk[i];
    vals[base + i] = sv[i];
  }
}

// One step (k, j) with j >= kLocal over all n2 elements: thread t compares
// the pair (i, i + j), i being t with a clear bit j inserted.
__global__ void __launch_bounds__(256)
k_bitonic_global(uint64_t* __restrict__ keys, uint32_t* __restrict__ vals, int64_t n2, int64_t k, int64_t j) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= n2 / 2) return;
  const int64_t i = ((t & ~(j - 1)) << 1) | (t & (j - 1));
  const int64_t l = i + j;
  const bool asc = (i & k) == 0;
  const uint64_t ka = keys[i], kb = keys[l];
  const uint32_t va = vals[i], vb = vals[l];
  if (pair_greater(ka, va, kb, vb) == asc) {
    keys[i] = kb;
    vals[i] = vb;
    keys[l] = ka;
    vals[l] = va;
  }
}

// Steps (k, j), (k, j/2), .., (k, j/2^(L-1)) in one launch, all with
// j/2^(L-1) >= kLocal: thread t holds the R = 2^L elements base + m*q
// (q = j/2^(L-1), m = 0 .. R-1; base is t with L clear bits inserted at q),
// which those steps pair only among themselves, in registers.  The elements
// span 2j <= k, so they share bit k and one direction.
template <int L>
__global__ void __launch_bounds__(256)
k_bitonic_global_multi(uint64_t* __restrict__ keys, uint32_t* __restrict__ vals, int64_t n2, int64_t k, int64_t j) {
  constexpr int R = 1 << L;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= n2 / R) return;
  const int64_t q = j >> (L - 1);
  const int64_t base = ((t & ~(q - 1)) << L) | (t & (q - 1));
  const bool asc = (base & k) == 0;
  uint64_t kk[R];
  uint32_t vv[R];
#pragma unroll
  for (int m = 0; m < R; ++m) {
    kk[m] = keys[base + m * q];
    vv[m] = vals[base + m * q];
  }
#pragma unroll
  for (int s = L - 1; s >= 0; --s) {
#pragma unroll
    for (int m = 0; m < R; ++m) {
      const int d = 1 << s;
      if (m & d) continue;
      if (pair_greater(kk[m], vv[m], kk[m + d], vv[m + d]) == asc) {
        const uint64_t tk = kk[m];
        const uint32_t tv = vv[m];
        kk[m] = kk[m + d];
        vv[m] = vv[m + d];
        kk[m + d] = tk;
        vv[m + d] = tv;
      }
    }
  }
#pragma unroll
  for (int m = 0; m < R; ++m) {
    keys[base + m * q] = kk[m];
    vals[base + m * q] = vv[m];
  }
}

__global__ void __launch_bounds__(256)
k_perm_out(const uint32_t* __restrict__ vals, int64_t B, int32_t* __restrict__ perm) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < B) perm[i] = static_cast<int32_t>(vals[i]);
}

}  // namespace

int64_t cluster_sort_size(int64_t B) {
  int64_t n2 = 1;
  while (n2 < B) n2 <<= 1;
  return n2;
}

hipError_t launch_cluster(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                          int64_t nnz, int32_t* perm, int32_t* df, uint64_t* keys, uint32_t* vals,
                          hipStream_t stream) {
  hipLaunchKernelGGL(k_zero_i32, dim3(static_cast<uint32_t>((F + 255) / 256)), dim3(256), 0, stream, df, F);
  if (nnz > 0) {
    const uint32_t groups = static_cast<uint32_t>((nnz + kHistItems - 1) / kHistItems);
    for (int64_t w0 = 0; w0 < F; w0 += kHistWindow) {
      const int wlen = static_cast<int>(F - w0 < kHistWindow ? F - w0 : kHistWindow);
      hipLaunchKernelGGL(k_df_lds, dim3(groups), dim3(256), 0, stream, indices, nnz, w0, wlen, df);
    }
  }
  const int bits = key_bits(F);
  const int64_t n2 = cluster_sort_size(B);
  hipLaunchKernelGGL(k_signature, dim3(static_cast<uint32_t>((n2 * kSigLanes + 255) / 256)), dim3(256), 0, stream,
                     indptr, indices, B, n2, F, bits, df, keys, vals);
  if (n2 >= 2) {
    const int64_t blk = n2 < kLocal ? n2 : kLocal;
    const uint32_t nblk = static_cast<uint32_t>(n2 / blk);
    // every step with k <= blk inside the blocks
    hipLaunchKernelGGL(k_bitonic_local, dim3(nblk), dim3(static_cast<uint32_t>(blk / 2)), 0, stream, keys, vals,
                       blk, int64_t(2), blk, int64_t(1));
    for (int64_t k = 2 * blk; k <= n2; k <<= 1) {
      // the wide steps three (or two) at a time, the last odd one alone
      int64_t j = k >> 1;
      while (j >= blk) {
        if (j >= 4 * blk) {
          hipLaunchKernelGGL(k_bitonic_global_multi<3>, dim3(static_cast<uint32_t>((n2 / 8 + 255) / 256)), dim3(256),
                             0, stream, keys, vals, n2, k, j);
          j >>= 3;
        } else if (j >= 2 * blk) {
          hipLaunchKernelGGL(k_bitonic_global_multi<2>, dim3(static_cast<uint32_t>((n2 / 4 + 255) / 256)), dim3(256),
                             0, stream, keys, vals, n2, k, j);
          j >>= 2;
        } else {
          hipLaunchKernelGGL(k_bitonic_global, dim3(static_cast<uint32_t>((n2 / 2 + 255) / 256)), dim3(256), 0,
                             stream, keys, vals, n2, k, j);
          j >>= 1;
        }
      }
      hipLaunchKernelGGL(k_bitonic_local, dim3(nblk), dim3(static_cast<uint32_t>(blk / 2)), 0, stream, keys, vals,
                         blk, k, k, blk >> 1);
    }
  }
  hipLaunchKernelGGL(k_perm_out, dim3(static_cast<uint32_t>((B + 255) / 256)), dim3(256), 0, stream, vals, B, perm);
  return hipGetLastError();
}

}  // namespace som
