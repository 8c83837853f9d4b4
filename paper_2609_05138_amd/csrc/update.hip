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
//  k_blur_stream  R <= 16: one wave per 64-column strip of a feature plane
//                 walks down the rows: row pass from an LDS row buffer,
//                 column pass from an LDS ring of the last 2R+1 results, the
//                 same sums term for term; the accumulators are read once and
//                 the codebook written once.
// Bound: HBM (the two-pass path streams 16 B per element, the streaming one
// 8 B plus a halo of 2R/64 of the reads).
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

// Streaming blur + write-back (R <= kStreamMaxR, one instantiation per
// radius): one wave owns a strip of 64 columns of one feature plane and
// walks down the grid rows.  Step r loads row r of the strip with its R-wide
// halo (cells outside the grid are zero) into the wave's own LDS row buffer
// and forms the row pass t[r][c] = sum_{k=-R..R} g[|k|] acc[r][c+k]; each
// lane keeps the row-pass results of the last 2R+1 rows in registers (the
// step loop is unrolled by a multiple of 2R+1, so a row's slot is a static
// index), from which the column pass of row r - R,
// sum_{k=-R..R} g[|k|] t[r-R+k][c] (zero rows outside the grid: their slots
// still hold zero), is formed; then the write-back through the blurred
// counts.  Both sums take the same terms in the same order as the two-pass
// kernels; the taps sit in registers and every LDS read has an immediate
// offset.  Rows, and the blurred counts of the rows written back, are loaded
// at least kStreamAhead steps before use; a wave
// touches only its own LDS, so there is no workgroup barrier, and every input
// and output element is read or written once.
constexpr int kStreamMaxR = 16;
constexpr int kStreamAhead = 8;

template <typename WT, int R>
__global__ void __launch_bounds__(64)
k_blur_stream(const uint32_t* __restrict__ acc, int64_t ld_acc, int64_t f0, int rows, int cols,
              const float* __restrict__ g, const float* __restrict__ den, WT* __restrict__ W, int64_t ldw) {
  constexpr int H = 2 * R + 1;
  // steps per unrolled block: a multiple of H (so row r's history slot is
  // the static index (r mod H)), and at least kStreamAhead (the prefetch depth)
  constexpr int U = H * ((kStreamAhead + H - 1) / H);
  __shared__ float rb[64 + 2 * R + 1];  // the current row with its halo
  const int lane = threadIdx.x;
  const int64_t f = f0 + blockIdx.y;
  const int c0 = blockIdx.x * 64;
  const int c = c0 + lane;
  const uint32_t* src = acc + f * ld_acc;
  float tp[R + 1];
#pragma unroll
  for (int i = 0; i <= R; ++i) tp[i] = g[i];
  float hr[H];  // row-pass results of the last H rows: row r in slot r mod H
#pragma unroll
  for (int i = 0; i < H; ++i) hr[i] = 0.f;
  // this lane's two input columns: c0 - R + lane, and c0 - R + 64 + lane for
  // the halo's last 2R cells
  const int ca = c0 - R + lane, cb = c0 - R + 64 + lane;
  const bool va = ca >= 0 && ca < cols, vb = lane < 2 * R && cb >= 0 && cb < cols;
  // Raw words in flight, with the blurred count of the row written back at
  // the step that uses them (row r - R): every lane loads unconditionally
  // (cells outside the grid read element 0 instead), and the selects and the
  // conversion happen when the row is used, so no load is waited for in the
  // step that issues it.
  const bool vc = c < cols;
  uint32_t pa[U], pb[U];
  float pd[U];
#define SOM_STREAM_LOAD(r, a, b, d)                                                                 \
  {                                                                                                \
    const bool in_ = (r) < rows;                                                                   \
    const int rd_ = (r) - R;                                                                       \
    a = src[(in_ && va) ? static_cast<int64_t>(r) * cols + ca : 0];                                \
    b = src[(in_ && vb) ? static_cast<int64_t>(r) * cols + cb : 0];                                \
    d = den[(rd_ >= 0 && rd_ < rows && vc) ? static_cast<int64_t>(rd_) * cols + c : 0];            \
  }
#pragma unroll
  for (int u = 0; u < U; ++u) SOM_STREAM_LOAD(u, pa[u], pb[u], pd[u])
  const int steps = rows + R;
  for (int r0 = 0; r0 < steps; r0 += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u;
      if (r >= steps) break;
      const bool in = r < rows;
      const float a = (in && va) ? static_cast<float>(pa[u]) : 0.f;
      const float b = (in && vb) ? static_cast<float>(pb[u]) : 0.f;
      const float dj = pd[u];  // blurred count of row r - R (read only when r >= R and c < cols)
      SOM_STREAM_LOAD(r + U, pa[u], pb[u], pd[u])
      // row pass of row r (zero beyond the last row)
      rb[lane] = a;
      if (lane < 2 * R) rb[64 + lane] = b;
      __builtin_amdgcn_wave_barrier();
      float t = 0.f;
#pragma unroll
      for (int j = 0; j <= 2 * R; ++j) t = fmaf(tp[j < R ? R - j : j - R], rb[lane + j], t);
      __builtin_amdgcn_wave_barrier();
      hr[u % H] = r < rows ? t : 0.f;
      // column pass of row r - R: slots (u+1 .. u+H) mod H hold rows r-2R .. r
      // (slots of rows before the first still hold zero)
      if (r >= R) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j <= 2 * R; ++j) s = fmaf(tp[j < R ? R - j : j - R], hr[(u + 1 + j) % H], s);
        if (vc && dj > 0.f) W[f * ldw + static_cast<int64_t>(r - R) * cols + c] = static_cast<WT>(s / dj);
      }
    }
  }
#undef SOM_STREAM_LOAD
}

template <typename WT, int R>
hipError_t launch_stream_r(const uint32_t* acc, int64_t ld_acc, int64_t F, int rows, int cols, const float* taps,
                           const float* den, WT* W, int64_t ldw, hipStream_t stream) {
  const uint32_t strips64 = static_cast<uint32_t>((cols + 63) / 64);
  for (int64_t f0 = 0; f0 < F; f0 += 65535) {  // grid.y holds at most 65535 features
    const uint32_t fc = static_cast<uint32_t>(F - f0 < 65535 ? F - f0 : 65535);
    hipLaunchKernelGGL((k_blur_stream<WT, R>), dim3(strips64, fc), dim3(64), 0, stream, acc, ld_acc, f0, rows, cols,
                       taps, den, W, ldw);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename WT, int R = 0>
hipError_t launch_stream(int r, const uint32_t* acc, int64_t ld_acc, int64_t F, int rows, int cols, const float* taps,
                         const float* den, WT* W, int64_t ldw, hipStream_t stream) {
  if constexpr (R > kStreamMaxR) {
    return hipErrorInvalidValue;
  } else {
    if (r == R) return launch_stream_r<WT, R>(acc, ld_acc, F, rows, cols, taps, den, W, ldw, stream);
    return launch_stream<WT, R + 1>(r, acc, ld_acc, F, rows, cols, taps, den, W, ldw, stream);
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
  if (R <= kStreamMaxR) {
    // numerators streamed down 64-column strips, written back through den
    if (weights == kWeightsF16)
      return launch_stream<_Float16>(R, acc, ld_acc, F, rows, cols, taps, den, static_cast<_Float16*>(W), ldw, stream);
    return launch_stream<float>(R, acc, ld_acc, F, rows, cols, taps, den, static_cast<float*>(W), ldw, stream);
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
