// Codebook norms ||w_j||^2 = sum_f W[f][j]^2 (paper, Section 3; the "norms"
// pass of Table 4).  One streaming pass over the feature-major codebook:
// each lane owns four consecutive neurons (one 128-bit load per row) and
// the waves of a workgroup split the rows; squares are exact in fp64 and
// accumulated there in a fixed order, so the result is deterministic and
// rounded to fp32 exactly once.  Bound: HBM read bandwidth (4 B per weight).
#include "common.h"

namespace som {
namespace {

constexpr int kNormWaves = 8;   // waves per workgroup, each a residue class of rows
constexpr int kChains = 4;      // independent fp64 chains per lane (loads in flight)

__global__ void __launch_bounds__(kNormWaves * 64)
k_norms(const float* __restrict__ W, int64_t F, int64_t N, int64_t ldw, float* __restrict__ norms) {
  __shared__ double part[kNormWaves][64][4];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t col = (static_cast<int64_t>(blockIdx.x) * 64 + lane) * 4;  // first of 4 neurons
  double s[kChains][4] = {};
  if (col < ldw) {
    const float* base = W + col;
    int64_t f = wave;
    // rows f, f + 8, f + 16, f + 24 go to chains 0..3, in increasing f per chain
    for (; f + 3 * kNormWaves < F; f += kChains * kNormWaves) {
      float4 v[kChains];
#pragma unroll
      for (int c = 0; c < kChains; ++c)
        v[c] = *reinterpret_cast<const float4*>(base + (f + c * kNormWaves) * ldw);
#pragma unroll
      for (int c = 0; c < kChains; ++c) {
        s[c][0] = fma(static_cast<double>(v[c].x), static_cast<double>(v[c].x), s[c][0]);
        s[c][1] = fma(static_cast<double>(v[c].y), static_cast<double>(v[c].y), s[c][1]);
        s[c][2] = fma(static_cast<double>(v[c].z), static_cast<double>(v[c].z), s[c][2]);
        s[c][3] = fma(static_cast<double>(v[c].w), static_cast<double>(v[c].w), s[c][3]);
      }
    }
    // at most three rows remain (f, f + 8, f + 16), one per chain
#pragma unroll
    for (int c = 0; c < kChains - 1; ++c) {
      const int64_t fr = f + c * kNormWaves;
      if (fr < F) {
        const float4 v = *reinterpret_cast<const float4*>(base + fr * ldw);
        s[c][0] = fma(static_cast<double>(v.x), static_cast<double>(v.x), s[c][0]);
        s[c][1] = fma(static_cast<double>(v.y), static_cast<double>(v.y), s[c][1]);
        s[c][2] = fma(static_cast<double>(v.z), static_cast<double>(v.z), s[c][2]);
        s[c][3] = fma(static_cast<double>(v.w), static_cast<double>(v.w), s[c][3]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) part[wave][lane][e] = (s[0][e] + s[1][e]) + (s[2][e] + s[3][e]);
  __syncthreads();
  if (wave == 0 && col < N) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      double t = part[0][lane][e];
#pragma unroll
      for (int w = 1; w < kNormWaves; ++w) t += part[w][lane][e];
      if (col + e < N) norms[col + e] = static_cast<float>(t);
    }
  }
}

}  // namespace

hipError_t launch_norms(const float* W, int64_t F, int64_t N, int64_t ldw, float* norms,
                        hipStream_t stream) {
  const int64_t groups = (ldw / 4 + 63) / 64;
  hipLaunchKernelGGL(k_norms, dim3(static_cast<uint32_t>(groups)), dim3(kNormWaves * 64), 0, stream,
                     W, F, N, ldw, norms);
  return hipGetLastError();
}

}  // namespace som
