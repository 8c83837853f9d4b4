// Fused BMU search (paper, Section 3; levers of Section 4).
//
// Work unit: one wave = one tile of T documents x one neuron slice of 64*K
// neurons (K per lane, read as K/4 128-bit loads, Section 4.3).  The wave
// keeps the T x K partial dot products in VGPRs and sweeps the tile's
// feature union once (Section 4.1): each union row slice is loaded once and
// added into the accumulators of exactly the documents whose membership bit
// is set, so every document's dot product is summed in ascending feature
// order whatever T, the slicing or the tile order (bit-identical results).
// The argmin is fused (Section 3): distances (|S| + ||w_j||^2) - 2*dot are
// formed in registers and reduced per lane, then across the wave with
// shuffles; the wave folds its result into the document's packed
// (distance, index) key with one 64-bit atomic minimum, so the neuron-axis
// chunks (Section 4.2) are merged without materialising any score block.
//
// A workgroup holds G waves on G different tiles of the SAME slice, and the
// grid is (tile groups, slices) with tile groups fastest: workgroups are
// dispatched slice-major, so the whole device sweeps one narrow neuron
// slice at a time and that slice's hot rows stay resident in each XCD's L2.
#include "common.h"

namespace som {
namespace {

// Add one union row slice into the accumulators of the documents whose
// membership bit is set.  Two equivalent forms (both add the row in the same
// order, so their results are bit-identical):
//   kMaskFma:    acc[s] = fma(w, b_s, acc[s]) with b_s = 1.0 or 0.0 taken from
//                the wave-uniform mask -- branch-free, T*K VALU per row;
//   kMaskBranch: wave-uniform scalar branches (a group-of-four test, then one
//                per document), popcount*K VALU.
enum MaskMode { kMaskFma = 0, kMaskBranch = 1 };


template <int T, int K, int MODE>
__device__ __forceinline__ void add_row(float (&acc)[T][K], const float4 (&w)[K / 4], uint32_t m) {
  if (MODE == kMaskFma) {
#pragma unroll
    for (int s = 0; s < T; ++s) {
      const float b = (m >> s) & 1u ? 1.f : 0.f;
#pragma unroll
      for (int q = 0; q < K / 4; ++q) {
        acc[s][4 * q + 0] = fmaf(w[q].x, b, acc[s][4 * q + 0]);
        acc[s][4 * q + 1] = fmaf(w[q].y, b, acc[s][4 * q + 1]);
        acc[s][4 * q + 2] = fmaf(w[q].z, b, acc[s][4 * q + 2]);
        acc[s][4 * q + 3] = fmaf(w[q].w, b, acc[s][4 * q + 3]);
      }
    }
  } else {
    // one scalar test per group of four documents first: most rows of a
    // tile of eight or more documents belong to one or two of them
#pragma unroll
    for (int g = 0; g < T; g += 4) {
      if (T >= 8 && ((m >> g) & 0xfu) == 0u) continue;
#pragma unroll
      for (int s = g; s < (g + 4 < T ? g + 4 : T); ++s) {
        if (m & (1u << s)) {
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
  }
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

// The two smallest of all lanes' (k1 < k2) pairs: merging two sorted pairs
// keeps min(a1, b1) and min(max(a1, b1), min(a2, b2)).  Keys are distinct
// (the low word is the neuron index), so the result is exact.
__device__ __forceinline__ void wave_top2_u64(uint64_t& k1, uint64_t& k2) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o1 = (static_cast<uint64_t>(__shfl_xor(static_cast<uint32_t>(k1 >> 32), off, 64)) << 32) |
                        __shfl_xor(static_cast<uint32_t>(k1), off, 64);
    const uint64_t o2 = (static_cast<uint64_t>(__shfl_xor(static_cast<uint32_t>(k2 >> 32), off, 64)) << 32) |
                        __shfl_xor(static_cast<uint32_t>(k2), off, 64);
    const uint64_t lo = k1 < o1 ? k1 : o1;
    const uint64_t hi = k1 < o1 ? o1 : k1;
    const uint64_t m2 = k2 < o2 ? k2 : o2;
    k1 = lo;
    k2 = hi < m2 ? hi : m2;
  }
}

// Insert a candidate key into a lane's sorted (k1 < k2) pair.
__device__ __forceinline__ void top2_insert(uint64_t key, uint64_t& k1, uint64_t& k2) {
  // selects only (a branchy form makes the compiler keep the pair in scratch)
  const uint64_t lo = key < k1 ? key : k1;
  const uint64_t hi = key < k1 ? k1 : key;
  k2 = hi < k2 ? hi : k2;
  k1 = lo;
}

// atomicMin on `best`, returning max(previous value, k1): the key this
// update pushes towards the second place.
__device__ __forceinline__ uint64_t top2_displaced(uint64_t* best, uint64_t k1) {
  const uint64_t old = atomicMin(reinterpret_cast<unsigned long long*>(best), static_cast<unsigned long long>(k1));
  return old > k1 ? old : k1;
}

// Fold one slice's (k1 < k2) into a document's global pair (best, second).
// The displaced value max(old best, k1) and k2 are the only keys of this
// slice that can be the global second: whichever of the two slices holding
// the global first and second updates `best` later pushes the other into
// `second`, whatever the order of the atomics, so the final pair is exact.
__device__ __forceinline__ void top2_merge(uint64_t* best, uint64_t* second, uint64_t k1, uint64_t k2) {
  const uint64_t displaced = top2_displaced(best, k1);
  const uint64_t cand = displaced < k2 ? displaced : k2;
  if (cand != kNoKey) atomicMin(reinterpret_cast<unsigned long long*>(second), static_cast<unsigned long long>(cand));
}

// Each wave stages its tile's union list in its own LDS window, kEntryChunk
// entries (feature id, mask) at a time, then issues its row loads from
// scalar registers.  The window is padded with (row 0, empty mask) entries
// so the row pipeline never branches on the list length.
constexpr int kEntryChunk = 512;

// Accelerator complex dies (XCDs) of an MI355X, each with its own L2.
constexpr uint32_t kXcds = 8;

template <int T, int K, int G, int U, int MODE>
__global__ void __launch_bounds__(G * 64)
k_search(SearchArgs a) {
  constexpr int Q = K / 4;
  constexpr int64_t WN = 64 * K;
  static_assert(kEntryChunk % (2 * U) == 0, "row batches must tile a window");
  __shared__ int2 ent_all[G][kEntryChunk + 2 * U];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // Workgroups are handed to the XCDs round-robin (workgroup i of a launch
  // runs on XCD i mod 8) and gridDim.x is a multiple of 8, so every XCD sees
  // the same residues in every slice row; give each XCD one contiguous range
  // of tile groups instead, so that neighbouring tiles of the (clustered)
  // tiled order, which share features, share that XCD's L2.
  const uint32_t per_xcd = gridDim.x / kXcds;
  const uint32_t wg = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  const int64_t t = static_cast<int64_t>(wg) * G + wave;         // this wave's tile
  const int64_t c = blockIdx.y;                                  // neuron slice
  if (t >= a.ntiles) return;                                     // no barriers below
  int2* ent = ent_all[wave];
  if (lane < 2 * U) ent[kEntryChunk + lane] = make_int2(0, 0);

  const int64_t n0 = c * WN;
  float acc[T][K];
#pragma unroll
  for (int s = 0; s < T; ++s)
#pragma unroll
    for (int k = 0; k < K; ++k) acc[s][k] = 0.f;

  // byte offsets of this lane's float4s inside a row slice; lanes past the
  // row end re-read the row's last float4 (in bounds; never reported)
  uint32_t offb[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int64_t o = 256 * q + 4 * lane;
    offb[q] = static_cast<uint32_t>(4 * (n0 + o < a.ldw ? o : a.ldw - 4 - n0));
  }
  const int32_t u0 = a.tile_offset[t];
  const int32_t cnt = a.tile_count[t];
  const float* __restrict__ Wn = a.W + n0;
  const int64_t ldw = a.ldw;

  float4 wa[U][Q], wb[U][Q];
  uint32_t ma[U], mb[U];
  auto fetch = [&](float4 (&w)[U][Q], uint32_t (&m)[U], int i) {
#pragma unroll
    for (int r = 0; r < U; ++r) {
      const int2 e = ent[i + r];
      const int32_t f32 = __builtin_amdgcn_readfirstlane(e.x);
      m[r] = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(e.y));
      const char* row = reinterpret_cast<const char*>(Wn + static_cast<int64_t>(f32) * ldw);
#pragma unroll
      for (int q = 0; q < Q; ++q) w[r][q] = *reinterpret_cast<const float4*>(row + offb[q]);
    }
  };
  auto process = [&](const float4 (&w)[U][Q], const uint32_t (&m)[U]) {
#pragma unroll
    for (int r = 0; r < U; ++r) add_row<T, K, MODE>(acc, w[r], m[r]);
  };

  for (int32_t base = 0; base < cnt; base += kEntryChunk) {
    // one wave reads and writes its own window: program order suffices
    for (int i = lane; i < kEntryChunk; i += 64) {
      const int32_t idx = base + i;
      ent[i] = idx < cnt ? make_int2(a.union_feat[u0 + idx], static_cast<int>(a.union_mask[u0 + idx]))
                         : make_int2(0, 0);
    }
    const int32_t rem = cnt - base;
    const int n = rem < kEntryChunk ? rem : kEntryChunk;
    // two batches of U rows in flight: load batch i+1 while adding batch i;
    // loads past n read the zero padding (row 0, empty mask).  Scheduling
    // barriers keep each batch's loads ahead of the adds of the previous one.
    fetch(wa, ma, 0);
    for (int i = 0; i < n; i += 2 * U) {
      fetch(wb, mb, i + U);
      __builtin_amdgcn_sched_barrier(0);
      process(wa, ma);
      __builtin_amdgcn_sched_barrier(0);
      fetch(wa, ma, i + 2 * U);
      __builtin_amdgcn_sched_barrier(0);
      process(wb, mb);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

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
    if (a.keys2) {  // best and second best (wave-uniform branch)
      uint64_t k1 = kNoKey, k2 = kNoKey;
#pragma unroll
      for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t j = n0 + 256 * q + 4 * lane + e;
          if (j < a.N)
            top2_insert(pack_key(fmaf(-2.f, acc[s][4 * q + e], nnz + nrm[4 * q + e]), static_cast<uint32_t>(j)),
                        k1, k2);
        }
      wave_top2_u64(k1, k2);
      if (lane == 0) top2_merge(a.keys + p, a.keys2 + p, k1, k2);
      continue;
    }
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
    if (lane == 0) atomicMin(reinterpret_cast<unsigned long long*>(a.keys + p), static_cast<unsigned long long>(key));
  }
}

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
  // columns past the row end re-read the row's last float4 (in bounds)
  const int sq = tid % kTpr;
  const int sr = tid / kTpr;
  const int64_t scol = n0 + 4 * sq < ldw ? n0 + 4 * sq : ldw - 4;
  const float* __restrict__ Wc = a.W + scol;
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

template <int T, int K, int G>
hipError_t launch_tkg(const SearchArgs& a, hipStream_t stream) {
  constexpr int U = K == 4 ? 8 : 4;
  // tile groups rounded up to a multiple of the XCD count (see k_search)
  const int64_t groups = (a.ntiles + G - 1) / G;
  const dim3 grid(static_cast<uint32_t>((groups + kXcds - 1) / kXcds * kXcds), static_cast<uint32_t>(a.nchunks));
  if (a.mask_mode == kMaskBranch)
    hipLaunchKernelGGL((k_search<T, K, G, U, kMaskBranch>), grid, dim3(G * 64), 0, stream, a);
  else
    hipLaunchKernelGGL((k_search<T, K, G, U, kMaskFma>), grid, dim3(G * 64), 0, stream, a);
  return hipGetLastError();
}

template <int T, int K>
hipError_t launch_tk(const SearchArgs& a, hipStream_t stream) {
  switch (a.group) {
    case 1: return launch_tkg<T, K, 1>(a, stream);
    case 2: return launch_tkg<T, K, 2>(a, stream);
    case 4: return launch_tkg<T, K, 4>(a, stream);
    case 8: return launch_tkg<T, K, 8>(a, stream);
    default: return hipErrorInvalidValue;
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

hipError_t launch_search(const SearchArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_keys_init, dim3(static_cast<uint32_t>((a.B + 255) / 256)), dim3(256), 0, stream,
                     a.keys, a.keys2, a.B);
  if (a.kernel == 2) return launch_docs(a, stream);
  switch (a.T) {
    case 1: return a.K == 4 ? launch_tk<1, 4>(a, stream) : launch_tk<1, 8>(a, stream);
    case 2: return a.K == 4 ? launch_tk<2, 4>(a, stream) : launch_tk<2, 8>(a, stream);
    case 4: return a.K == 4 ? launch_tk<4, 4>(a, stream) : launch_tk<4, 8>(a, stream);
    case 8: return a.K == 4 ? launch_tk<8, 4>(a, stream) : launch_tk<8, 8>(a, stream);
    case 16: return a.K == 4 ? launch_tk<16, 4>(a, stream) : launch_tk<16, 8>(a, stream);
    case 32: return launch_tk<32, 4>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_merge(const SearchArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_decode, dim3(static_cast<uint32_t>((a.B + 255) / 256)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace som
