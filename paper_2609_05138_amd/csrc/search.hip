// Fused BMU search (paper, Section 3; levers of Section 4).
//
// One workgroup handles one tile of T documents against one chunk of
// neurons (Section 4.2, neuron-axis chunking).  Each wave owns 64*K
// consecutive-by-lane neurons of the chunk (K per lane, read as K/4 128-bit
// loads, Section 4.3) and keeps the T x K partial dot products in VGPRs.
// It sweeps the tile's feature union once (Section 4.1): every union row
// slice is loaded once and added into the accumulators of exactly the
// documents whose membership bit is set, so each document's dot product is
// summed in ascending feature order whatever T, the chunking or the tile
// order (bit-identical results across them).  The argmin is fused
// (Section 3): distances d = (|S| + ||w_j||^2) - 2*dot are formed in
// registers, reduced per lane, across the wave with shuffles and across the
// workgroup's waves with an LDS atomic minimum on packed (distance, index)
// keys; one key per (chunk, document) goes to the partial array, and a
// merge kernel takes the minimum over chunks and writes results in input
// order.
//
// The grid is (tiles, chunks) with tiles fastest, so workgroups are dispatched
// chunk-major: the whole device sweeps one neuron chunk at a time and the
// chunk's columns stay resident in the caches.
#include "common.h"

namespace som {
namespace {

template <int T, int K>
__device__ __forceinline__ void add_row(float (&acc)[T][K], const float4 (&w)[K / 4], uint32_t m) {
#pragma unroll
  for (int s = 0; s < T; ++s) {
    if (m & (1u << s)) {  // wave-uniform: a scalar branch, no divergence
#pragma unroll
      for (int q = 0; q < K / 4; ++q) {
        acc[s][4 * q + 0] += w[q].x;
        acc[s][4 * q + 1] += w[q].y;
        acc[s][4 * q + 2] += w[q].z;
        acc[s][4 * q + 3] += w[q].w;
      }
    }
  }
}

template <int K>
__device__ __forceinline__ void load_row(float4 (&w)[K / 4], const float* row, const bool (&in)[K / 4]) {
#pragma unroll
  for (int q = 0; q < K / 4; ++q)
    w[q] = in[q] ? *reinterpret_cast<const float4*>(row + 256 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t k) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(k), off, 64);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(k >> 32), off, 64);
    const uint64_t o = (static_cast<uint64_t>(hi) << 32) | lo;
    k = o < k ? o : k;
  }
  return k;
}

template <int T, int K, int WAVES, int U>
__global__ void __launch_bounds__(WAVES * 64)
k_search(SearchArgs a) {
  constexpr int Q = K / 4;
  constexpr int64_t WN = 64 * K;
  constexpr int64_t CN = WAVES * WN;
  __shared__ unsigned long long red[T];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t t = blockIdx.x;  // tile: fastest-varying, so the grid runs chunk-major
  const int64_t c = blockIdx.y;  // neuron chunk
  if (threadIdx.x < T) red[threadIdx.x] = kNoKey;

  const int64_t n0 = c * CN + wave * WN;  // first neuron of this wave
  float acc[T][K];
#pragma unroll
  for (int s = 0; s < T; ++s)
#pragma unroll
    for (int k = 0; k < K; ++k) acc[s][k] = 0.f;

  bool in[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) in[q] = n0 + 256 * q + 4 * lane < a.ldw;

  if (n0 < a.N) {
    const int32_t u0 = a.tile_offset[t];
    const int32_t cnt = a.tile_count[t];
    const int32_t* __restrict__ uf = a.union_feat + u0;
    const uint32_t* __restrict__ um = a.union_mask + u0;
    const float* __restrict__ Wl = a.W + n0 + 4 * lane;
    int32_t u = 0;
    for (; u + U <= cnt; u += U) {
      float4 w[U][Q];
      uint32_t m[U];
#pragma unroll
      for (int r = 0; r < U; ++r) {
        const int64_t f = __builtin_amdgcn_readfirstlane(uf[u + r]);
        m[r] = __builtin_amdgcn_readfirstlane(um[u + r]);
        load_row<K>(w[r], Wl + f * a.ldw, in);
      }
#pragma unroll
      for (int r = 0; r < U; ++r) add_row<T, K>(acc, w[r], m[r]);
    }
    for (; u < cnt; ++u) {
      float4 w[Q];
      const int64_t f = __builtin_amdgcn_readfirstlane(uf[u]);
      const uint32_t m = __builtin_amdgcn_readfirstlane(um[u]);
      load_row<K>(w, Wl + f * a.ldw, in);
      add_row<T, K>(acc, w, m);
    }
  }
  __syncthreads();  // red[] initialised

  if (n0 < a.N) {
    float nrm[K];
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t j = n0 + 256 * q + 4 * lane + e;
        nrm[4 * q + e] = j < a.N ? a.norms[j] : 0.f;
      }
#pragma unroll
    for (int s = 0; s < T; ++s) {
      const int64_t p = t * T + s;
      if (p >= a.B) break;
      const int64_t d = a.perm ? static_cast<int64_t>(a.perm[p]) : p;
      const float nnz = static_cast<float>(a.indptr[d + 1] - a.indptr[d]);
      float best = 0.f;
      uint32_t bj = 0xffffffffu;
#pragma unroll
      for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t j = n0 + 256 * q + 4 * lane + e;
          if (j < a.N) {
            const float dj = fmaf(-2.f, acc[s][4 * q + e], nnz + nrm[4 * q + e]);
            if (bj == 0xffffffffu || dj < best) {  // ascending j: strict < keeps the lowest
              best = dj;
              bj = static_cast<uint32_t>(j);
            }
          }
        }
      uint64_t key = bj == 0xffffffffu ? kNoKey : pack_key(best, bj);
      key = wave_min_u64(key);
      if (lane == 0) atomicMin(&red[s], static_cast<unsigned long long>(key));
    }
  }
  __syncthreads();
  if (threadIdx.x < T) {
    const int64_t p = t * T + threadIdx.x;
    if (p < a.B) a.partial[c * (a.ntiles * T) + p] = red[threadIdx.x];
  }
}

__global__ void __launch_bounds__(256) k_merge(SearchArgs a) {
  const int64_t p = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (p >= a.B) return;
  const int64_t P = a.ntiles * a.T;
  uint64_t best = kNoKey;
  for (int64_t c = 0; c < a.nchunks; ++c) {
    const uint64_t k = a.partial[c * P + p];
    best = k < best ? k : best;
  }
  const int64_t d = a.perm ? static_cast<int64_t>(a.perm[p]) : p;
  a.bmu[d] = static_cast<int32_t>(static_cast<uint32_t>(best));
  a.dist[d] = from_ordered_bits(static_cast<uint32_t>(best >> 32));
}

template <int T, int K, int WAVES>
hipError_t launch_tkw(const SearchArgs& a, hipStream_t stream) {
  constexpr int U = T <= 8 ? 4 : 2;
  const dim3 grid(static_cast<uint32_t>(a.ntiles), static_cast<uint32_t>(a.nchunks));
  hipLaunchKernelGGL((k_search<T, K, WAVES, U>), grid, dim3(WAVES * 64), 0, stream, a);
  return hipGetLastError();
}

template <int T, int K>
hipError_t launch_tk(const SearchArgs& a, hipStream_t stream) {
  switch (a.waves) {
    case 1: return launch_tkw<T, K, 1>(a, stream);
    case 2: return launch_tkw<T, K, 2>(a, stream);
    case 4: return launch_tkw<T, K, 4>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_search(const SearchArgs& a, hipStream_t stream) {
  switch (a.T) {
    case 1: return launch_tk<1, 8>(a, stream);
    case 2: return launch_tk<2, 8>(a, stream);
    case 4: return launch_tk<4, 8>(a, stream);
    case 8: return launch_tk<8, 8>(a, stream);
    case 16: return launch_tk<16, 8>(a, stream);
    case 32: return launch_tk<32, 4>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_merge(const SearchArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_merge, dim3(static_cast<uint32_t>((a.B + 255) / 256)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace som
