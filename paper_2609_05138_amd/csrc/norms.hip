// Codebook norms ||w_j||^2 = sum_f W[f][j]^2 (paper, Section 3; the "norms"
// pass of Table 4).  One streaming pass over the feature-major codebook:
// each lane owns the neurons of one 128-bit load per row (four fp32 or eight
// fp16 weights) and the waves of a workgroup split the rows; squares are
// exact in fp64 and accumulated there in a fixed order, so the result is
// deterministic and rounded to fp32 exactly once.  For an fp16 codebook the
// norms are those of the stored (rounded) weights.  Bound: HBM read
// bandwidth (4 or 2 B per weight).
#include "common.h"

namespace som {
namespace {

constexpr int kNormWaves = 8;   // waves per workgroup, each a residue class of rows
constexpr int kChains = 4;      // independent fp64 chains per lane (loads in flight)

typedef _Float16 nh8 __attribute__((ext_vector_type(8)));

template <typename WT>
struct NormLoad;
template <>
struct NormLoad<float> {
  static constexpr int kE = 4;
  static __device__ __forceinline__ void get(const float* p, double (&v)[4]) {
    const float4 x = *reinterpret_cast<const float4*>(p);
    v[0] = x.x;
    v[1] = x.y;
    v[2] = x.z;
    v[3] = x.w;
  }
};
template <>
struct NormLoad<_Float16> {
  static constexpr int kE = 8;
  static __device__ __forceinline__ void get(const _Float16* p, double (&v)[8]) {
    const nh8 x = *reinterpret_cast<const nh8*>(p);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = static_cast<double>(x[e]);
  }
};

template <typename WT>
__global__ void __launch_bounds__(kNormWaves * 64)
k_norms(const WT* __restrict__ W, int64_t F, int64_t N, int64_t ldw, float* __restrict__ norms) {
  constexpr int E = NormLoad<WT>::kE;
  __shared__ double part[kNormWaves][64][E];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t col = (static_cast<int64_t>(blockIdx.x) * 64 + lane) * E;  // first of E neurons
  double s[kChains][E] = {};
  // only groups holding a neuron j < N are read: no load leaves
  // [0, round_up(N, E)) of its row
  if (col < N) {
    const WT* base = W + col;
    int64_t f = wave;
    // rows f, f + 8, f + 16, f + 24 go to chains 0..3, in increasing f per chain
    for (; f + 3 * kNormWaves < F; f += kChains * kNormWaves) {
      double v[kChains][E];
#pragma unroll
      for (int c = 0; c < kChains; ++c) NormLoad<WT>::get(base + (f + c * kNormWaves) * ldw, v[c]);
#pragma unroll
      for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int e = 0; e < E; ++e) s[c][e] = fma(v[c][e], v[c][e], s[c][e]);
    }
    // at most three rows remain (f, f + 8, f + 16), one per chain
#pragma unroll
    for (int c = 0; c < kChains - 1; ++c) {
      const int64_t fr = f + c * kNormWaves;
      if (fr < F) {
        double v[E];
        NormLoad<WT>::get(base + fr * ldw, v);
#pragma unroll
        for (int e = 0; e < E; ++e) s[c][e] = fma(v[e], v[e], s[c][e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) part[wave][lane][e] = (s[0][e] + s[1][e]) + (s[2][e] + s[3][e]);
  __syncthreads();
  if (wave == 0 && col < N) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      double t = part[0][lane][e];
#pragma unroll
      for (int w = 1; w < kNormWaves; ++w) t += part[w][lane][e];
      if (col + e < N) norms[col + e] = static_cast<float>(t);
    }
  }
}

}  // namespace

hipError_t launch_norms(const void* W, int weights, int64_t F, int64_t N, int64_t ldw, float* norms,
                        hipStream_t stream) {
  if (weights == kWeightsF16) {
    const int64_t groups = ((N + 7) / 8 + 63) / 64;
    hipLaunchKernelGGL(k_norms<_Float16>, dim3(static_cast<uint32_t>(groups)), dim3(kNormWaves * 64), 0, stream,
                       static_cast<const _Float16*>(W), F, N, ldw, norms);
  } else {
    const int64_t groups = ((N + 3) / 4 + 63) / 64;
    hipLaunchKernelGGL(k_norms<float>, dim3(static_cast<uint32_t>(groups)), dim3(kNormWaves * 64), 0, stream,
                       static_cast<const float*>(W), F, N, ldw, norms);
  }
  return hipGetLastError();
}

}  // namespace som
