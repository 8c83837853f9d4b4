// Batch-SOM update after the search (paper, Section 3: the best-matching
// unit and its neighbours are updated; Section 6.1, Table 4: a scatter into
// accumulators, a neighbourhood blur, a write-back, then the norms refresh).
// The neighbourhood is the reading stated in include/som.h: a Gaussian of
// width sigma on the rows x cols map grid, truncated at R = ceil(3 sigma) along
// each axis, hence separable into a row blur and a column blur.
//
//  k_accumulate   one wave per document: acc[f][bmu] += 1 for its features and
//                 count[bmu] += 1, as uint32 atomics (exact, order-free)
//  k_taps         g[k] = exp(-k^2 / (2 sigma^2)) for k = 0..R, in fp64, rounded
//                 to fp32 once
//  k_blur_rows    one grid row of one feature per workgroup, staged in LDS:
//                 t[r][c] = sum_{k=-R..R} g[|k|] acc[r][c+k]  (fixed tap order)
//  k_blur_cols    a strip of 32 columns of one feature per workgroup, staged
//                 in LDS: v[r][c] = sum_k g[|k|] t[r+k][c]; then either the
//                 blurred counts (den) or the write-back W = v / den where
//                 den > 0 (other units keep their weights)
//  k_blur_fused   R <= 16: both passes on a 64 x 64 tile (plus halo) in LDS,
//                 the same sums term for term; the accumulators are read once
//                 (with the halo) and the codebook written once.
// Bound: HBM (the two-pass path streams 16 B per element, the fused one
// about 9-13 B).
#include "common.h"

namespace som {
namespace {

constexpr int kStrip = 32;  // columns per column-blur workgroup (128 B of fp32)

__global__ void __launch_bounds__(256)
k_accumulate(const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices, int64_t B,
             const int32_t* __restrict__ bmu, int64_t F, int64_t N, uint32_t* __restrict__ acc,
             int64_t ld_acc, uint32_t* __restrict__ count) {
  const int lane = threadIdx.x & 63;
  const int64_t d = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (d >= B) return;
  const int64_t b = bmu[d];
  if (b < 0 || b >= N) return;  // not a unit of this map: ignored
  const int32_t e0 = indptr[d], e1 = indptr[d + 1];
  for (int32_t e = e0 + lane; e < e1; e += 64) {
    const int64_t f = indices[e];
    if (f >= 0 && f < F) atomicAdd(acc + f * ld_acc + b, 1u);
  }
  if (lane == 0) atomicAdd(count + b, 1u);
}

__global__ void k_taps(double sigma, int R, float* __restrict__ g) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k > R) return;
  g[k] = sigma > 0 ? static_cast<float>(exp(-static_cast<double>(k) * k / (2.0 * sigma * sigma))) : 1.f;
}

// in: plane p of the input (uint32 accumulators or fp32), rows x cols with
// row stride `cols` inside a plane of stride ld_in; out: fp32 plane of
// stride ld_out.  Grid (rows, planes): rows fastest, so that concurrent
// workgroups spread over one plane rather than hitting the same offset of
// planes a power-of-two stride apart (the same memory channels).
template <typename IN>
__global__ void __launch_bounds__(256)
k_blur_rows(const IN* __restrict__ in, int64_t ld_in, float* __restrict__ out, int64_t ld_out, int cols, int R,
            const float* __restrict__ g) {
  extern __shared__ float row[];
  const int64_t p = blockIdx.y;
  const int r = blockIdx.x;
  const IN* src = in + p * ld_in + static_cast<int64_t>(r) * cols;
  for (int c = threadIdx.x; c < cols; c += blockDim.x) row[c] = static_cast<float>(src[c]);
  __syncthreads();
  float* dst = out + p * ld_out + static_cast<int64_t>(r) * cols;
  for (int c = threadIdx.x; c < cols; c += blockDim.x) {
    const int lo = c - R < 0 ? -c : -R;
    const int hi = c + R >= cols ? cols - 1 - c : R;
    float s = 0.f;
    for (int k = lo; k <= hi; ++k) s = fmaf(g[k < 0 ? -k : k], row[c + k], s);
    dst[c] = s;
  }
}

// MODE 0: den[j] = v (one plane); MODE 1: write-back into the codebook.
// Grid (strips, planes), strips fastest (see k_blur_rows).
template <typename WT, int MODE>
__global__ void __launch_bounds__(256)
k_blur_cols(const float* __restrict__ t, int64_t ld_t, int rows, int cols, int R, const float* __restrict__ g,
            float* __restrict__ den_out, const float* __restrict__ den, WT* __restrict__ W, int64_t ldw) {
  extern __shared__ float strip[];  // [rows][kStrip]
  const int64_t p = blockIdx.y;
  const int c0 = blockIdx.x * kStrip;
  const int cx = threadIdx.x % kStrip;
  const int ry = threadIdx.x / kStrip;          // 8 row lanes
  const int c = c0 + cx;
  const float* src = t + p * ld_t;
  for (int r = ry; r < rows; r += 256 / kStrip)
    strip[r * kStrip + cx] = c < cols ? src[static_cast<int64_t>(r) * cols + c] : 0.f;
  __syncthreads();
  if (c >= cols) return;
  for (int r = ry; r < rows; r += 256 / kStrip) {
    const int lo = r - R < 0 ? -r : -R;
    const int hi = r + R >= rows ? rows - 1 - r : R;
    float s = 0.f;
    for (int k = lo; k <= hi; ++k) s = fmaf(g[k < 0 ? -k : k], strip[(r + k) * kStrip + cx], s);
    const int64_t j = static_cast<int64_t>(r) * cols + c;
    if (MODE == 0) {
      den_out[j] = s;
    } else {
      const float dj = den[j];
      if (dj > 0.f) W[p * ldw + j] = static_cast<WT>(s / dj);
    }
  }
}

// Fused blur + write-back for small radii: one 64 x 64 tile of one feature
// per workgroup, loaded with its R-wide halo into LDS (cells outside the grid
// are zero and add nothing, so the sums equal the two-pass ones term for
// term); the row pass and the column pass both run in LDS and the codebook
// is written once.  Grid (tiles, features) with tiles fastest: feature planes
// sit a power-of-two stride apart, so workgroups that ran the same tile of
// consecutive features would all hit the same memory channels.
constexpr int kTile = 64;
constexpr int kFusedMaxR = 16;

template <typename WT>
__global__ void __launch_bounds__(256)
k_blur_fused(const uint32_t* __restrict__ acc, int64_t ld_acc, int64_t f0, int rows, int cols, int R,
             const float* __restrict__ g, const float* __restrict__ den, WT* __restrict__ W, int64_t ldw) {
  extern __shared__ float lds[];
  const int E = kTile + 2 * R;                    // tile edge with halo
  float* in = lds;                                // [E][E]
  float* mid = lds + E * E;                       // [E][kTile]
  float* taps = mid + E * kTile;                  // [R + 1]
  const int64_t f = f0 + blockIdx.y;
  const int tiles_x = (cols + kTile - 1) / kTile;
  const int r0 = (blockIdx.x / tiles_x) * kTile;
  const int c0 = (blockIdx.x % tiles_x) * kTile;
  const uint32_t* src = acc + f * ld_acc;
  for (int i = threadIdx.x; i <= R; i += blockDim.x) taps[i] = g[i];
  // Thread (ty, tx) loads columns tx and tx + 64 of rows ty, ty + 4, ...: all
  // of its loads are issued before the first LDS store.
  constexpr int kMaxE = kTile + 2 * kFusedMaxR;
  constexpr int kPasses = kMaxE / 4;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  float v[kPasses][2];
#pragma unroll
  for (int q = 0; q < kPasses; ++q)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int y = ty + 4 * q, x = tx + 64 * h;
      const int r = r0 - R + y, c = c0 - R + x;
      v[q][h] = (y < E && x < E && r >= 0 && r < rows && c >= 0 && c < cols)
                    ? static_cast<float>(src[static_cast<int64_t>(r) * cols + c])
                    : 0.f;
    }
#pragma unroll
  for (int q = 0; q < kPasses; ++q)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int y = ty + 4 * q, x = tx + 64 * h;
      if (y < E && x < E) in[y * E + x] = v[q][h];
    }
  __syncthreads();
  for (int i = threadIdx.x; i < E * kTile; i += blockDim.x) {
    const int y = i / kTile, x = i % kTile;
    const float* row = in + y * E + x;            // taps k = -R..R at row[R + k]
    float s = 0.f;
    for (int k = -R; k <= R; ++k) s = fmaf(taps[k < 0 ? -k : k], row[R + k], s);
    mid[i] = s;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kTile * kTile; i += blockDim.x) {
    const int y = i / kTile, x = i % kTile;
    const int r = r0 + y, c = c0 + x;
    if (r >= rows || c >= cols) continue;
    float s = 0.f;
    for (int k = -R; k <= R; ++k) s = fmaf(taps[k < 0 ? -k : k], mid[(y + R + k) * kTile + x], s);
    const int64_t j = static_cast<int64_t>(r) * cols + c;
    const float dj = den[j];
    if (dj > 0.f) W[f * ldw + j] = static_cast<WT>(s / dj);
  }
}

}  // namespace

size_t update_chunk_planes(int64_t F, int64_t N) {
  int64_t fc = (int64_t(1) << 26) / (N > 0 ? N : 1);  // about 256 MB of fp32 per chunk
  if (fc < 1) fc = 1;
  if (fc > 65535) fc = 65535;  // planes go in grid.y
  if (fc > F) fc = F;
  return static_cast<size_t>(fc);
}

hipError_t launch_update_accumulate(const int32_t* indptr, const int32_t* indices, int64_t B, const int32_t* bmu,
                                    int64_t F, int64_t N, uint32_t* acc, int64_t ld_acc, uint32_t* count,
                                    hipStream_t stream) {
  hipLaunchKernelGGL(k_accumulate, dim3(static_cast<uint32_t>((B + 3) / 4)), dim3(256), 0, stream, indptr, indices,
                     B, bmu, F, N, acc, ld_acc, count);
  return hipGetLastError();
}

hipError_t launch_update_finish(void* W, int weights, int64_t F, int64_t ldw, int rows, int cols, double sigma, int R,
                                const uint32_t* acc, int64_t ld_acc, const uint32_t* count, float* taps,
                                float* den_tmp, float* den, float* chunk, int64_t chunk_planes,
                                hipStream_t stream) {
  const int64_t N = static_cast<int64_t>(rows) * cols;
  hipLaunchKernelGGL(k_taps, dim3(static_cast<uint32_t>(R / 256 + 1)), dim3(256), 0, stream, sigma, R, taps);
  const size_t row_lds = sizeof(float) * static_cast<size_t>(cols);
  const size_t col_lds = sizeof(float) * static_cast<size_t>(rows) * kStrip;
  const uint32_t strips = static_cast<uint32_t>((cols + kStrip - 1) / kStrip);
  {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_blur_rows<uint32_t>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(row_lds));
    if (e != hipSuccess) return e;
  }
  for (auto f : {reinterpret_cast<const void*>(&k_blur_cols<float, 0>), reinterpret_cast<const void*>(&k_blur_cols<float, 1>),
                 reinterpret_cast<const void*>(&k_blur_cols<_Float16, 1>)}) {
    hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(col_lds));
    if (e != hipSuccess) return e;
  }
  // denominators: the blurred counts
  hipLaunchKernelGGL(k_blur_rows<uint32_t>, dim3(static_cast<uint32_t>(rows), 1), dim3(256), row_lds, stream, count,
                     N, den_tmp, N, cols, R, taps);
  hipLaunchKernelGGL((k_blur_cols<float, 0>), dim3(strips, 1), dim3(256), col_lds, stream, den_tmp, N, rows, cols, R,
                     taps, den, nullptr, nullptr, int64_t(0));
  if (R <= kFusedMaxR) {
    // numerators blurred tile by tile in LDS and written back through den
    const int E = kTile + 2 * R;
    const size_t lds = sizeof(float) * (static_cast<size_t>(E) * E + static_cast<size_t>(E) * kTile + R + 1);
    const auto fused = weights == kWeightsF16 ? reinterpret_cast<const void*>(&k_blur_fused<_Float16>)
                                              : reinterpret_cast<const void*>(&k_blur_fused<float>);
    hipError_t e = hipFuncSetAttribute(fused, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (e != hipSuccess) return e;
    const uint32_t tiles = static_cast<uint32_t>(((rows + kTile - 1) / kTile) * ((cols + kTile - 1) / kTile));
    for (int64_t f0 = 0; f0 < F; f0 += 65535) {  // grid.y holds at most 65535 features
      const uint32_t fc = static_cast<uint32_t>(F - f0 < 65535 ? F - f0 : 65535);
      if (weights == kWeightsF16)
        hipLaunchKernelGGL(k_blur_fused<_Float16>, dim3(tiles, fc), dim3(256), lds, stream, acc, ld_acc, f0, rows,
                           cols, R, taps, den, static_cast<_Float16*>(W), ldw);
      else
        hipLaunchKernelGGL(k_blur_fused<float>, dim3(tiles, fc), dim3(256), lds, stream, acc, ld_acc, f0, rows, cols,
                           R, taps, den, static_cast<float*>(W), ldw);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    return hipGetLastError();
  }
  // larger radii: numerators a chunk of features at a time, row pass into the
  // chunk buffer, then the column pass written back through den
  for (int64_t f0 = 0; f0 < F; f0 += chunk_planes) {
    const int64_t fc = F - f0 < chunk_planes ? F - f0 : chunk_planes;
    hipLaunchKernelGGL(k_blur_rows<uint32_t>, dim3(static_cast<uint32_t>(rows), static_cast<uint32_t>(fc)), dim3(256),
                       row_lds, stream, acc + f0 * ld_acc, ld_acc, chunk, N, cols, R, taps);
    if (weights == kWeightsF16)
      hipLaunchKernelGGL((k_blur_cols<_Float16, 1>), dim3(strips, static_cast<uint32_t>(fc)), dim3(256), col_lds,
                         stream, chunk, N, rows, cols, R, taps, nullptr, den,
                         static_cast<_Float16*>(W) + f0 * ldw, ldw);
    else
      hipLaunchKernelGGL((k_blur_cols<float, 1>), dim3(strips, static_cast<uint32_t>(fc)), dim3(256), col_lds,
                         stream, chunk, N, rows, cols, R, taps, nullptr, den, static_cast<float*>(W) + f0 * ldw,
                         ldw);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipGetLastError();
}

}  // namespace som
