// Kernel 1 of the fused BMU search (paper, Section 3; levers of Section 4),
// templated on the codebook's storage type (fp32, or fp16 as in the paper's
// own kernel, Sections 4.2 and 4.3); accumulation is fp32 either way.
//
// Work unit: one wave = one tile of T documents x one neuron slice of 64*K
// neurons (K per lane, read with 128-bit loads, Section 4.3).  The wave
// keeps the T x K partial dot products in VGPRs and sweeps the tile's
// feature union once (Section 4.1): each union row slice is loaded once,
// widened to fp32, and added into the accumulators of exactly the documents
// whose membership bit is set, so every document's dot product is summed in
// ascending feature order whatever T, the slicing or the tile order
// (bit-identical results).  The argmin is fused (Section 3): distances
// (|S| + ||w_j||^2) - 2*dot are formed in registers and reduced per lane,
// then across the wave with shuffles; the wave folds its result into the
// document's packed (distance, index) key with one 64-bit atomic minimum, so
// the neuron-axis chunks (Section 4.2) are merged without materialising any
// score block.
//
// A workgroup holds G waves on G different tiles of the SAME slice, and the
// grid is (tile groups, slices) with tile groups fastest: workgroups are
// dispatched slice-major, so the whole device sweeps one narrow neuron
// slice at a time and that slice's hot rows stay resident in each XCD's L2.
//
// Included by the translation units that instantiate it (one per storage
// type); everything here has internal linkage.
#pragma once

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

// Elements of the storage type in one 128-bit load.
template <typename WT>
struct Storage;
template <>
struct Storage<float> {
  static constexpr int kE = 4;
};
template <>
struct Storage<_Float16> {
  static constexpr int kE = 8;
};

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float8 __attribute__((ext_vector_type(8)));
// A native 128-bit vector (HIP's uint4 is a struct whose copies can go through
// private memory when staged in arrays).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Widen one 128-bit load of the storage type to fp32 (exact for fp16).
template <typename WT>
__device__ __forceinline__ void widen(const uint4& raw, float4* out);
template <>
__device__ __forceinline__ void widen<float>(const uint4& raw, float4* out) {
  out[0] = make_float4(__uint_as_float(raw.x), __uint_as_float(raw.y), __uint_as_float(raw.z),
                       __uint_as_float(raw.w));
}
template <>
__device__ __forceinline__ void widen<_Float16>(const uint4& raw, float4* out) {
  const half8 h = __builtin_bit_cast(half8, raw);
  const float8 f = __builtin_convertvector(h, float8);
  out[0] = make_float4(f[0], f[1], f[2], f[3]);
  out[1] = make_float4(f[4], f[5], f[6], f[7]);
}
template <typename WT>
__device__ __forceinline__ void widen_v(const u32x4& raw, float4* out);
template <>
__device__ __forceinline__ void widen_v<float>(const u32x4& raw, float4* out) {
  out[0] = make_float4(__uint_as_float(raw.x), __uint_as_float(raw.y), __uint_as_float(raw.z),
                       __uint_as_float(raw.w));
}
template <>
__device__ __forceinline__ void widen_v<_Float16>(const u32x4& raw, float4* out) {
  const half8 h = __builtin_bit_cast(half8, raw);
  const float8 f = __builtin_convertvector(h, float8);
  out[0] = make_float4(f[0], f[1], f[2], f[3]);
  out[1] = make_float4(f[4], f[5], f[6], f[7]);
}

// Fused epilogue (Section 3): the T documents at tiled positions p0 .. p0+T-1
// against this wave's slice of 64*K neurons starting at n0.  Distances
// (|S| + ||w_j||^2) - 2*dot are formed in registers, reduced per lane (ascending
// j, strict < keeps the lowest index), then across the wave with shuffles, and
// folded into the document's packed key with one 64-bit atomic minimum (or, for
// the top-2 search, into the (best, second) pair; for the unfused comparator,
// written to the distance block instead).
template <typename WT, int T, int K>
__device__ __forceinline__ void epilogue(const SearchArgs& a, const float (&acc)[T][K], int64_t p0, int64_t n0,
                                         int lane) {
  constexpr int E = Storage<WT>::kE;
  constexpr int Q = K / E;
  float nrm[K];
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int64_t j = n0 + 64 * E * q + E * lane + e;
      nrm[E * q + e] = j < a.N ? a.norms[j] : 0.f;
    }
  // one loop per output form (the choice is wave-uniform), each small enough
  // to unroll fully, so the accumulators stay in registers
  if (a.score) {  // unfused comparator: write the distances, no argmin here
#pragma unroll
    for (int s = 0; s < T; ++s) {
      const int64_t p = p0 + s;
      if (p >= a.B) break;
      const int64_t d = a.perm ? static_cast<int64_t>(a.perm[p]) : p;
      const float nnz = static_cast<float>(a.indptr[d + 1] - a.indptr[d]);
      float* row = a.score + (p - a.tile_base * T) * a.N;
#pragma unroll
      for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int64_t j = n0 + 64 * E * q + E * lane + e;
          if (j < a.N) row[j] = fmaf(-2.f, acc[s][E * q + e], nnz + nrm[E * q + e]);
        }
    }
    return;
  }
  if (a.keys2) {  // best and second best
#pragma unroll
    for (int s = 0; s < T; ++s) {
      const int64_t p = p0 + s;
      if (p >= a.B) break;
      const int64_t d = a.perm ? static_cast<int64_t>(a.perm[p]) : p;
      const float nnz = static_cast<float>(a.indptr[d + 1] - a.indptr[d]);
      uint64_t k1 = kNoKey, k2 = kNoKey;
#pragma unroll
      for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int64_t j = n0 + 64 * E * q + E * lane + e;
          if (j < a.N)
            top2_insert(pack_key(fmaf(-2.f, acc[s][E * q + e], nnz + nrm[E * q + e]), static_cast<uint32_t>(j)),
                        k1, k2);
        }
      wave_top2_u64(k1, k2);
      if (lane == 0) top2_merge(a.keys + p, a.keys2 + p, k1, k2);
    }
    return;
  }
#pragma unroll
  for (int s = 0; s < T; ++s) {
    const int64_t p = p0 + s;
    if (p >= a.B) break;
    const int64_t d = a.perm ? static_cast<int64_t>(a.perm[p]) : p;
    const float nnz = static_cast<float>(a.indptr[d + 1] - a.indptr[d]);
    float best = 0.f;
    uint32_t bj = 0xffffffffu;
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int64_t j = n0 + 64 * E * q + E * lane + e;
        if (j < a.N) {
          const float dj = fmaf(-2.f, acc[s][E * q + e], nnz + nrm[E * q + e]);
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

// Waves per SIMD the register budget must allow: 16-document fp32 tiles fit
// five (at most 96 VGPRs), which the memory-latency-bound loop needs; the
// register allocator is otherwise free to settle just above that line.
template <typename WT, int T, int K>
constexpr int k1_min_waves() {
  return (sizeof(WT) == 4 && T == 16 && K == 4) ? 5 : 1;
}

template <typename WT, int T, int K, int G, int U, int MODE>
__global__ void __launch_bounds__(G * 64) __attribute__((amdgpu_waves_per_eu(k1_min_waves<WT, T, K>())))
k_search(SearchArgs a) {
  constexpr int E = Storage<WT>::kE;  // elements per 128-bit load
  constexpr int Q = K / E;            // loads per lane per row
  constexpr int64_t WN = 64 * K;      // neurons per slice
  static_assert(K % E == 0 && K % 4 == 0, "a lane holds whole 128-bit loads");
  static_assert(kEntryChunk % (2 * U) == 0, "row batches must tile a window");
  __shared__ int2 ent_all[G][kEntryChunk + 2 * U];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // Workgroups are handed to the XCDs round-robin (workgroup i of a launch
  // runs on XCD i mod 8) and gridDim.x is a multiple of 8, so every XCD sees
  // the same residues in every slice row; give each XCD one contiguous range
  // of tile groups instead, so that neighbouring tiles of the (clustered)
  // tiled order, which share features, share that XCD's L2.
  uint64_t wg, c;  // tile group, neuron slice
  if (a.chunk_slices > 1) {
    chunked_block(static_cast<uint64_t>(blockIdx.y) * gridDim.x + blockIdx.x, gridDim.x, gridDim.y,
                  static_cast<uint64_t>(a.chunk_slices), &wg, &c);
  } else {
    const uint32_t per_xcd = gridDim.x / kXcds;
    wg = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    c = blockIdx.y;
  }
  const int64_t t = a.tile_base + static_cast<int64_t>(wg) * G + wave;  // this wave's tile
  if (t >= a.tile_end) return;                                          // no barriers below
  int2* ent = ent_all[wave];
  if (lane < 2 * U) ent[kEntryChunk + lane] = make_int2(0, 0);

  const int64_t n0 = c * WN;
  float acc[T][K];
#pragma unroll
  for (int s = 0; s < T; ++s)
#pragma unroll
    for (int k = 0; k < K; ++k) acc[s][k] = 0.f;

  // Load q of a lane covers neurons n0 + 64*E*q + E*lane + [0, E), which are
  // accumulators E*q .. E*q + E - 1.  Byte offsets inside a row slice; lanes
  // past the last neuron re-read the last group holding one (never reported),
  // so no load leaves [0, round_up(N, E)) of its row.
  // The limit is slice-relative and wave-uniform: 32-bit scalar arithmetic
  // keeps the per-lane cost to one compare and select.
  const int64_t nv = (a.N + E - 1) / E * E;
  const int32_t lim = static_cast<int32_t>(nv - n0 < WN ? nv - n0 : WN);  // valid columns of the slice
  uint32_t offb[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int32_t o = 64 * E * q + E * lane;
    offb[q] = static_cast<uint32_t>(sizeof(WT)) * static_cast<uint32_t>(o < lim ? o : lim - E);
  }
  const int32_t u0 = a.tile_offset[t];
  const int32_t cnt = a.tile_count[t];
  // Rotated sweep: the tile's union is swept from entry e0 on, wrapping round,
  // so that the tiles an XCD runs at once sweep the same part of the feature
  // range together.  e0 is the tile's phase (as in kernel 3): the plan's
  // nonzeros of the XCD's earlier tiles, a proxy for their work, over
  // a.phase_wgs tiles' mean work, mod 1, times the union's size; it depends on
  // the plan and the tile grid only, not on the slice.
  int32_t e0 = 0;
  if (a.rotate && a.chunk_slices <= 1 && cnt > 1) {
    const int64_t per_xcd = gridDim.x / kXcds;  // tile groups per XCD
    const int64_t g0 = (blockIdx.x % kXcds) * per_xcd;
    const int64_t first = a.tile_base + g0 * G;
    const int64_t end = a.tile_base + (g0 + per_xcd) * G < a.tile_end ? a.tile_base + (g0 + per_xcd) * G : a.tile_end;
    const uint64_t o_first = static_cast<uint32_t>(a.tile_offset[first]);
    const uint64_t work = static_cast<uint32_t>(a.tile_offset[end]) - o_first;   // >= cnt > 0
    const uint64_t nx = static_cast<uint64_t>(end - first);
    const uint64_t den = static_cast<uint64_t>(a.phase_wgs) * work;
    const uint64_t num = (static_cast<uint32_t>(u0) - o_first) * nx % den;
    const uint64_t ph = (num << 20) / den;
    e0 = __builtin_amdgcn_readfirstlane(static_cast<int32_t>((ph * static_cast<uint64_t>(cnt)) >> 20));
  }
  const WT* __restrict__ Wn = static_cast<const WT*>(a.W) + n0;
  const int64_t ldw = a.ldw;

  uint4 wa[U][Q], wb[U][Q];
  uint32_t ma[U], mb[U];
  auto fetch = [&](uint4 (&w)[U][Q], uint32_t (&m)[U], int i) {
#pragma unroll
    for (int r = 0; r < U; ++r) {
      const int2 e = ent[i + r];
      const int32_t f32 = __builtin_amdgcn_readfirstlane(e.x);
      m[r] = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(e.y));
      const char* row = reinterpret_cast<const char*>(Wn + static_cast<int64_t>(f32) * ldw);
#pragma unroll
      for (int q = 0; q < Q; ++q) w[r][q] = *reinterpret_cast<const uint4*>(row + offb[q]);
    }
  };
  auto process = [&](const uint4 (&w)[U][Q], const uint32_t (&m)[U]) {
#pragma unroll
    for (int r = 0; r < U; ++r) {
      float4 wf[K / 4];
#pragma unroll
      for (int q = 0; q < Q; ++q) widen<WT>(w[r][q], wf + q * (E / 4));
      add_row<T, K, MODE>(acc, wf, m[r]);
    }
  };

  for (int32_t base = 0; base < cnt; base += kEntryChunk) {
    // one wave reads and writes its own window: program order suffices
    for (int i = lane; i < kEntryChunk; i += 64) {
      const int32_t idx = base + i;
      const int32_t src = idx + e0 < cnt ? idx + e0 : idx + e0 - cnt;   // rotated sweep (e0 = 0: ascending)
      ent[i] = idx < cnt ? make_int2(a.union_feat[u0 + src], static_cast<int>(a.union_mask[u0 + src]))
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

  epilogue<WT, T, K>(a, acc, t * T, n0, lane);
}

template <typename WT, int T, int K, int G>
hipError_t launch_tkg(const SearchArgs& a, hipStream_t stream) {
  // Rows per batch (two batches in flight), chosen by measurement on the
  // 512^2 map: deeper batches raise each wave's loads in flight but cost
  // VGPRs, and the occupancy they take matters more.  fp32 with one 128-bit
  // load per lane per row: 8 rows, 2 from T = 16 on (the accumulators grow;
  // 2 ran a 1M-document batch 3.7 % faster than 4); fp16 (8 weights per
  // load): 4 rows, 2 from T = 16 on; two loads per row: 4.
  constexpr int Q = K / Storage<WT>::kE;
  constexpr int U = Q == 1 ? (sizeof(WT) == 2 ? (T >= 16 ? 2 : 4) : (T >= 16 ? 2 : 8)) : 4;
  // tile groups rounded up to a multiple of the XCD count (see k_search)
  const int64_t groups = (a.tile_end - a.tile_base + G - 1) / G;
  const dim3 grid(static_cast<uint32_t>((groups + kXcds - 1) / kXcds * kXcds), static_cast<uint32_t>(a.nchunks));
  SearchArgs b = a;
  if (a.rotate) {
    const hipError_t e = k1_phase_tiles(T, G, a.mask_mode, &b.phase_wgs);
    if (e != hipSuccess) return e;
  }
  if (a.mask_mode == kMaskBranch)
    hipLaunchKernelGGL((k_search<WT, T, K, G, U, kMaskBranch>), grid, dim3(G * 64), 0, stream, b);
  else
    hipLaunchKernelGGL((k_search<WT, T, K, G, U, kMaskFma>), grid, dim3(G * 64), 0, stream, b);
  return hipGetLastError();
}

template <typename WT, int T, int K>
hipError_t launch_tk(const SearchArgs& a, hipStream_t stream) {
  switch (a.group) {
    case 1: return launch_tkg<WT, T, K, 1>(a, stream);
    case 2: return launch_tkg<WT, T, K, 2>(a, stream);
    case 4: return launch_tkg<WT, T, K, 4>(a, stream);
    case 8: return launch_tkg<WT, T, K, 8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace
}  // namespace som
