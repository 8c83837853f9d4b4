// Fused BMU search, kernel 2 (documents on lanes), the key array
// initialisation and decode, and the dispatch of the three kernels (paper,
// Section 3; kernel 1 is in search_k1.h, kernel 3 in search_st.h).
#include "search_st.h"

namespace som {
namespace {

// Documents on lanes (the neuron axis cut into narrow slices).
//
// A workgroup of G waves owns a group of D = 64*G consecutive documents of
// the tiled order, one document per lane, and one slice of NB neurons (32 or
// 64: a slice's rows for all 20,000 features are 2.5-5 MB, the size of one
// XCD's L2, so with slice-major dispatch every row is fetched from HBM about
// once per XCD).  The group's feature union (the tile union of Section 4.1
// with a tile of D documents) is streamed through a double-buffered LDS
// window of kRows row slices, loaded with coalesced 128-bit loads; each lane
// then walks its own document's features that fall in the window (their
// union positions come from the plan, in ascending order) and adds the NB
// weights of each into its NB accumulators.  Each document's dot product is
// therefore summed in ascending feature order, exactly as in the
// neurons-on-lanes kernel: results are bit-identical between the two.  The
// lane's best neuron over the slice is folded into the document's packed key
// with an atomic minimum, skipped when the key already holds a better value.
template <int NB>
struct DocsCfg {
  static constexpr int kQ = NB / 4;              // float4 per row slice
  static constexpr int kStride = kQ + 1;         // LDS row stride in float4 (bank spread)
  static constexpr int kRows = NB == 32 ? 448 : 224;  // rows per window (2 windows < 160 KB)
};

template <int NB, int G>
__global__ void __launch_bounds__(G * 64)
k_search_docs(SearchArgs a) {
  using C = DocsCfg<NB>;
  constexpr int kQ = C::kQ, kStride = C::kStride, kRows = C::kRows;
  constexpr int kThreads = G * 64;
  constexpr int kTpr = kQ;                        // staging threads per row
  constexpr int kRpp = kThreads / kTpr;           // rows per staging pass
  constexpr int kPasses = (kRows + kRpp - 1) / kRpp;
  __shared__ float4 rows[2][kRows * kStride];

  const int tid = threadIdx.x;
  const int64_t g = blockIdx.x;
  const int64_t c = blockIdx.y;
  const int64_t n0 = c * NB;
  const int64_t D = static_cast<int64_t>(kThreads);
  const int64_t p = g * D + tid;                  // this lane's document (tiled order)
  const bool valid = p < a.B;
  const int64_t d = valid ? (a.perm ? static_cast<int64_t>(a.perm[p]) : p) : 0;
  const int32_t e0 = valid ? a.indptr[d] : 0;
  const int32_t e1 = valid ? a.indptr[d + 1] : 0;
  const int32_t cnt = a.group_count[g];
  const int32_t goff = a.group_offset[g];
  const int32_t nw = (cnt + kRows - 1) / kRows;
  const int64_t ldw = a.ldw;

  // staging role: row r = pass * kRpp + tid / kTpr, float4 q = tid % kTpr;
  // columns past the last neuron re-read the last float4 holding one, so no
  // load leaves [0, round_up(N, 4)) of its row
  const int sq = tid % kTpr;
  const int sr = tid / kTpr;
  const int64_t nv = (a.N + 3) / 4 * 4;
  const int64_t scol = n0 + 4 * sq < nv ? n0 + 4 * sq : nv - 4;
  const float* __restrict__ Wc = static_cast<const float*>(a.W) + scol;
  float4 stage[kPasses];
#pragma unroll
  for (int k = 0; k < kPasses; ++k) stage[k] = make_float4(0.f, 0.f, 0.f, 0.f);

  float acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) acc[j] = 0.f;

  constexpr int32_t kEnd = 0x7fffffff;
  int32_t ptr = e0;
  int32_t pos = ptr < e1 ? a.entry_pos[ptr] : kEnd;

// staging of window w into registers, then into LDS buffer `buf`
#define SOM_DOCS_PREFETCH(w)                                                   \
  _Pragma("unroll") for (int k = 0; k < kPasses; ++k) {                        \
    const int r = k * kRpp + sr;                                               \
    const int32_t u = (w) * kRows + r;                                         \
    const int64_t f = (r < kRows && u < cnt) ? a.group_feat[goff + u] : 0;     \
    stage[k] = *reinterpret_cast<const float4*>(Wc + f * ldw);                 \
  }
#define SOM_DOCS_STORE(buf)                                                    \
  _Pragma("unroll") for (int k = 0; k < kPasses; ++k) {                        \
    const int r = k * kRpp + sr;                                               \
    if (r < kRows) rows[buf][r * kStride + sq] = stage[k];                     \
  }

  if (nw > 0) {
    SOM_DOCS_PREFETCH(0)
    SOM_DOCS_STORE(0)
  }
  __syncthreads();
  for (int32_t w = 0; w < nw; ++w) {
    if (w + 1 < nw) { SOM_DOCS_PREFETCH(w + 1) }
    const int32_t wbase = w * kRows;
    const int32_t wend = wbase + kRows;
    const float4* __restrict__ buf = rows[w & 1];
    while (pos < wend) {
      const int32_t nxt = ptr + 1 < e1 ? a.entry_pos[ptr + 1] : kEnd;
      const float4* rp = buf + (pos - wbase) * kStride;
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        const float4 v = rp[q];
        acc[4 * q + 0] += v.x;
        acc[4 * q + 1] += v.y;
        acc[4 * q + 2] += v.z;
        acc[4 * q + 3] += v.w;
      }
      pos = nxt;
      ++ptr;
    }
    if (w + 1 < nw) { SOM_DOCS_STORE((w + 1) & 1) }
    __syncthreads();
  }
#undef SOM_DOCS_PREFETCH
#undef SOM_DOCS_STORE

  if (!valid) return;
  const float nnz = static_cast<float>(e1 - e0);
  if (a.keys2) {  // best and second best
    uint64_t k1 = kNoKey, k2 = kNoKey;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int64_t gj = n0 + j;
      if (gj < a.N) top2_insert(pack_key(fmaf(-2.f, acc[j], nnz + a.norms[gj]), static_cast<uint32_t>(gj)), k1, k2);
    }
    // a stale read of `best` only filters: if k1 is not below it, the true
    // best is below k1 too, so the displaced key would be k1 itself
    uint64_t* kb = a.keys + p;
    const uint64_t displaced =
        k1 < *kb ? top2_displaced(kb, k1) : k1;
    const uint64_t cand = displaced < k2 ? displaced : k2;
    uint64_t* ks = a.keys2 + p;
    if (cand < *ks) atomicMin(reinterpret_cast<unsigned long long*>(ks), static_cast<unsigned long long>(cand));
    return;
  }
  float best = 0.f;
  uint32_t bj = 0xffffffffu;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int64_t gj = n0 + j;
    if (gj < a.N) {
      const float dj = fmaf(-2.f, acc[j], nnz + a.norms[gj]);
      if (bj == 0xffffffffu || dj < best) {  // ascending j: strict < keeps the lowest
        best = dj;
        bj = static_cast<uint32_t>(gj);
      }
    }
  }
  const uint64_t key = pack_key(best, bj);
  unsigned long long* kp = reinterpret_cast<unsigned long long*>(a.keys + p);
  if (key < *kp) atomicMin(kp, static_cast<unsigned long long>(key));
}

__global__ void __launch_bounds__(256) k_keys_init(uint64_t* __restrict__ keys, uint64_t* __restrict__ keys2,
                                                   int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) {
    keys[i] = kNoKey;
    if (keys2) keys2[i] = kNoKey;
  }
}

// Decode each document's key into (bmu, dist) in input order.
__global__ void __launch_bounds__(256) k_decode(SearchArgs a) {
  const int64_t p = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (p >= a.B) return;
  const uint64_t best = a.keys[p];
  const int64_t d = a.perm ? static_cast<int64_t>(a.perm[p]) : p;
  a.bmu[d] = static_cast<int32_t>(static_cast<uint32_t>(best));
  a.dist[d] = from_ordered_bits(static_cast<uint32_t>(best >> 32));
  if (a.keys2) {
    const uint64_t second = a.keys2[p];
    a.bmu2[d] = second == kNoKey ? -1 : static_cast<int32_t>(static_cast<uint32_t>(second));
    a.dist2[d] = second == kNoKey ? __builtin_inff() : from_ordered_bits(static_cast<uint32_t>(second >> 32));
  }
}

// Unfused comparator, second pass: one wave per row of the distance block
// (one document), lanes striding the row with 128-bit loads; each lane keeps
// its first minimum in ascending j, then the wave reduces packed keys, so the
// lowest index wins ties exactly as in the fused search.
__global__ void __launch_bounds__(256)
k_argmin_rows(const float* __restrict__ score, int64_t N, int64_t p0, int64_t rows, const int32_t* __restrict__ perm,
              int32_t* __restrict__ bmu, float* __restrict__ dist) {
  const int lane = threadIdx.x & 63;
  const int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const float* row = score + r * N;
  float best = 0.f;
  uint32_t bj = 0xffffffffu;
  const int64_t n4 = N / 4 * 4;
  for (int64_t j = 4 * lane; j < n4; j += 256) {
    const float4 v = *reinterpret_cast<const float4*>(row + j);
    const float x[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (bj == 0xffffffffu || x[e] < best) {
        best = x[e];
        bj = static_cast<uint32_t>(j + e);
      }
  }
  for (int64_t j = n4 + lane; j < N; j += 64)
    if (bj == 0xffffffffu || row[j] < best) {
      best = row[j];
      bj = static_cast<uint32_t>(j);
    }
  uint64_t key = bj == 0xffffffffu ? kNoKey : pack_key(best, bj);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(key), off, 64);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(key >> 32), off, 64);
    const uint64_t o = (static_cast<uint64_t>(hi) << 32) | lo;
    key = o < key ? o : key;
  }
  if (lane == 0) {
    const int64_t p = p0 + r;
    const int64_t d = perm ? static_cast<int64_t>(perm[p]) : p;
    bmu[d] = static_cast<int32_t>(static_cast<uint32_t>(key));
    dist[d] = from_ordered_bits(static_cast<uint32_t>(key >> 32));
  }
}

template <int NB, int G>
hipError_t launch_docs_ng(const SearchArgs& a, hipStream_t stream) {
  const int64_t ngroups = (a.B + 64 * G - 1) / (64 * G);
  const dim3 grid(static_cast<uint32_t>(ngroups), static_cast<uint32_t>(a.nchunks));
  hipLaunchKernelGGL((k_search_docs<NB, G>), grid, dim3(G * 64), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_docs(const SearchArgs& a, hipStream_t stream) {
  if (a.slice == 32) {
    switch (a.group) {
      case 4: return launch_docs_ng<32, 4>(a, stream);
      case 8: return launch_docs_ng<32, 8>(a, stream);
      case 16: return launch_docs_ng<32, 16>(a, stream);
      default: return hipErrorInvalidValue;
    }
  }
  if (a.slice == 64) {
    switch (a.group) {
      case 4: return launch_docs_ng<64, 4>(a, stream);
      case 8: return launch_docs_ng<64, 8>(a, stream);
      case 16: return launch_docs_ng<64, 16>(a, stream);
      default: return hipErrorInvalidValue;
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_k1(const SearchArgs& a, hipStream_t stream) {
  if (a.weights == kWeightsF16) return launch_search_k1_f16(a, stream);
  switch (a.T) {
    case 1: return a.K == 4 ? launch_tk<float, 1, 4>(a, stream) : launch_tk<float, 1, 8>(a, stream);
    case 2: return a.K == 4 ? launch_tk<float, 2, 4>(a, stream) : launch_tk<float, 2, 8>(a, stream);
    case 4: return a.K == 4 ? launch_tk<float, 4, 4>(a, stream) : launch_tk<float, 4, 8>(a, stream);
    case 8: return a.K == 4 ? launch_tk<float, 8, 4>(a, stream) : launch_tk<float, 8, 8>(a, stream);
    case 16: return a.K == 4 ? launch_tk<float, 16, 4>(a, stream) : launch_tk<float, 16, 8>(a, stream);
    case 32: return launch_tk<float, 32, 4>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

// Phase period of kernel 3's rotated sweep, in workgroups per XCD: 3/2 of
// the workgroups one XCD holds at once (its CUs times the occupancy per CU).
// Measured on the topic workload (1M documents, 512^2 map) over 3/4 to 3
// times that count, 5/4 to 3/2 were fastest.  It is taken from the fp32
// kernel of the super-tile's shape for both storage types, so that the fp16
// and fp32 searches of one plan sum in the same order.
hipError_t st_phase_wgs(int T, int S, int32_t* wgs) {
  constexpr int P = 16, NSLOT = 2;
  const void* fn = nullptr;
  if (T == 8 && S == 8) fn = reinterpret_cast<const void*>(k_search_st<float, 8, 4, 8, P, NSLOT, kStDocRotated>);
  if (T == 8 && S == 16) fn = reinterpret_cast<const void*>(k_search_st<float, 8, 4, 16, P, NSLOT, kStDocRotated>);
  if (T == 16 && S == 16) fn = reinterpret_cast<const void*>(k_search_st<float, 16, 4, 16, P, NSLOT, kStDocRotated>);
  if (!fn) return hipErrorInvalidValue;
  int per_cu = 0, dev = 0, cus = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, S * 64, 0);
  if (e != hipSuccess) return e;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int M = 3 * per_cu * cus / static_cast<int>(2 * kXcds);
  *wgs = M > 0 ? M : 1;
  return hipSuccess;
}

// Phase period of kernel 1's rotated sweep, in tiles per XCD: 3/2 of the
// tiles (one per wave) one XCD holds at once, from the fp32 kernel of the
// tile shape for both storage types, as for kernel 3.
template <int T, int G>
const void* k1_f32_kernel(int mask_mode) {
  constexpr int U = T >= 16 ? 2 : 8;  // fp32 rows per batch (launch_tkg)
  return mask_mode == kMaskBranch ? reinterpret_cast<const void*>(k_search<float, T, 4, G, U, kMaskBranch>)
                                  : reinterpret_cast<const void*>(k_search<float, T, 4, G, U, kMaskFma>);
}
template <int T>
const void* k1_f32_kernel_g(int G, int mask_mode) {
  switch (G) {
    case 1: return k1_f32_kernel<T, 1>(mask_mode);
    case 2: return k1_f32_kernel<T, 2>(mask_mode);
    case 4: return k1_f32_kernel<T, 4>(mask_mode);
    case 8: return k1_f32_kernel<T, 8>(mask_mode);
    default: return nullptr;
  }
}

hipError_t k1_phase_tiles(int T, int G, int mask_mode, int32_t* tiles) {
  const void* fn = T == 1 ? k1_f32_kernel_g<1>(G, mask_mode)
                 : T == 2 ? k1_f32_kernel_g<2>(G, mask_mode)
                 : T == 4 ? k1_f32_kernel_g<4>(G, mask_mode)
                 : T == 8 ? k1_f32_kernel_g<8>(G, mask_mode)
                 : T == 16 ? k1_f32_kernel_g<16>(G, mask_mode)
                 : T == 32 ? k1_f32_kernel_g<32>(G, mask_mode) : nullptr;
  if (!fn) return hipErrorInvalidValue;
  int per_cu = 0, dev = 0, cus = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, G * 64, 0);
  if (e != hipSuccess) return e;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int M = 3 * per_cu * G * cus / static_cast<int>(2 * kXcds);
  *tiles = M > 0 ? M : 1;
  return hipSuccess;
}

hipError_t launch_k3(const SearchArgs& a, hipStream_t stream) {
  if (a.weights == kWeightsF16) return launch_search_st_f16(a, stream);
  if (a.K != 4) return hipErrorInvalidValue;
  // waves of 8 documents for 64- and 128-document super-tiles, of 16 for 256
  // (a workgroup holds at most 16 waves)
  if (a.T == 8) {
    switch (a.group) {
      case 8: return launch_st<float, 8, 4, 8>(a, stream);
      case 16: return launch_st<float, 8, 4, 16>(a, stream);
      default: return hipErrorInvalidValue;
    }
  }
  if (a.T == 16 && a.group == 16) return launch_st<float, 16, 4, 16>(a, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_search(const SearchArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_keys_init, dim3(static_cast<uint32_t>((a.B + 255) / 256)), dim3(256), 0, stream,
                     a.keys, a.keys2, a.B);
  if (a.kernel == 2) return launch_docs(a, stream);
  if (a.kernel == 3) return launch_k3(a, stream);
  return launch_k1(a, stream);
}

hipError_t launch_unfused(SearchArgs a, int64_t block_docs, hipStream_t stream) {
  const int64_t tiles_per_block = block_docs / a.T;
  for (int64_t t0 = 0; t0 < a.ntiles; t0 += tiles_per_block) {
    a.tile_base = t0;
    a.tile_end = t0 + tiles_per_block < a.ntiles ? t0 + tiles_per_block : a.ntiles;
    hipError_t e = launch_k1(a, stream);
    if (e != hipSuccess) return e;
    const int64_t p0 = t0 * a.T;
    const int64_t rows = (a.tile_end * a.T < a.B ? a.tile_end * a.T : a.B) - p0;
    hipLaunchKernelGGL(k_argmin_rows, dim3(static_cast<uint32_t>((rows + 3) / 4)), dim3(256), 0, stream, a.score,
                       a.N, p0, rows, a.perm, a.bmu, a.dist);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_merge(const SearchArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_decode, dim3(static_cast<uint32_t>((a.B + 255) / 256)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace som
