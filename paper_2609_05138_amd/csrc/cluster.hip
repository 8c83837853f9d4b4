// Tile-membership clustering (paper, Section 4.2): place documents that
// share descriptors in the same tile so that each tile's feature union
// shrinks.  The paper gives no algorithm; this is a label-free reading:
//   df(f)  = number of documents of the batch containing f
//   (s1,s2)= a document's two features of highest df (ties to the lower id;
//            F stands in for a missing feature)
//   order  = stable sort of the documents by (s1, s2), i.e. by
//            (s1, s2, input position).
// Integer work; deterministic.  The stable key sort is a library radix
// sort (hipCUB); the histogram and signatures are our kernels.
#include <hipcub/hipcub.hpp>

#include "common.h"

namespace som {
namespace {

constexpr int kHistWindow = 16384;   // features per LDS histogram window
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

__global__ void k_iota(int32_t* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = static_cast<int32_t>(i);
}

// Signature key of each document: (s1 << bits) | s2.
__global__ void __launch_bounds__(256)
k_signature(const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices, int64_t B,
            int64_t F, int bits, const int32_t* __restrict__ df, uint64_t* __restrict__ keys) {
  const int64_t d = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (d >= B) return;
  int64_t s1 = F, s2 = F;
  int32_t c1 = -1, c2 = -1;  // df of s1, s2
  for (int32_t i = indptr[d]; i < indptr[d + 1]; ++i) {
    const int64_t f = indices[i];
    const int32_t c = df[f];
    // rank by (-df, f); features arrive in ascending f, so "greater df" wins
    if (c > c1) {
      s2 = s1; c2 = c1;
      s1 = f; c1 = c;
    } else if (c > c2) {
      s2 = f; c2 = c;
    }
  }
  keys[d] = (static_cast<uint64_t>(s1) << bits) | static_cast<uint64_t>(s2);
}

int key_bits(int64_t F) {
  int b = 1;
  while ((int64_t(1) << b) <= F) ++b;  // values 0..F inclusive
  return b;
}

}  // namespace

size_t cluster_sort_temp_bytes(int64_t B, int64_t F) {
  size_t bytes = 0;
  const hipError_t e = hipcub::DeviceRadixSort::SortPairs(nullptr, bytes, static_cast<const uint64_t*>(nullptr),
                                     static_cast<uint64_t*>(nullptr), static_cast<const int32_t*>(nullptr),
                                     static_cast<int32_t*>(nullptr), static_cast<int>(B), 0,
                                     2 * key_bits(F));
  return e == hipSuccess ? bytes : 0;
}

hipError_t launch_cluster(const int32_t* indptr, const int32_t* indices, int64_t B, int64_t F,
                          int64_t nnz, int32_t* perm, int32_t* df, uint64_t* keys,
                          uint64_t* keys_sorted, int32_t* iota, void* sort_temp,
                          size_t sort_temp_bytes, hipStream_t stream) {
  hipLaunchKernelGGL(k_zero_i32, dim3(static_cast<uint32_t>((F + 255) / 256)), dim3(256), 0, stream, df, F);
  if (nnz > 0) {
    const uint32_t groups = static_cast<uint32_t>((nnz + kHistItems - 1) / kHistItems);
    for (int64_t w0 = 0; w0 < F; w0 += kHistWindow) {
      const int wlen = static_cast<int>(F - w0 < kHistWindow ? F - w0 : kHistWindow);
      hipLaunchKernelGGL(k_df_lds, dim3(groups), dim3(256), 0, stream, indices, nnz, w0, wlen, df);
    }
  }
  const int bits = key_bits(F);
  hipLaunchKernelGGL(k_signature, dim3(static_cast<uint32_t>((B + 255) / 256)), dim3(256), 0, stream,
                     indptr, indices, B, F, bits, df, keys);
  hipLaunchKernelGGL(k_iota, dim3(static_cast<uint32_t>((B + 255) / 256)), dim3(256), 0, stream, iota, B);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  size_t tb = sort_temp_bytes;
  return hipcub::DeviceRadixSort::SortPairs(sort_temp, tb, keys, keys_sorted, iota, perm,
                                            static_cast<int>(B), 0, 2 * bits, stream);
}

}  // namespace som
