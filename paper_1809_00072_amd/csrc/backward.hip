// Backward pass of model-in-the-loop re-training (Sec. VI, re-training with RxNN):
// the forward pass runs on the crossbar model, the backward pass in floating
// point through the layer's ideal weights with straight-through DAC and ADC
// and the range constraints of the mapping:
//   dX = (dY W^T) * [0 <= x <= x_max]         (inputs the DAC clips: no gradient)
//   dW = clip(X, 0, x_max)^T dY * [|w| <= w_max]
// For a convolution X is its unrolled patch matrix (patch column
// k = (ci kh + ky) kw + kx, Sec. VI): the patches of the clipped input are
// unrolled, dW = patches^T dY, and dX gathers the patch gradients back onto
// the input pixels.  The patches are stored k-major (colsT[k][bv], bv the
// output pixel), so that the unrolling reads and writes along image rows and
// the gather reads the patch gradients dcolsT = W dY^T along them too.  The
// contractions are plain fp32 GEMMs (rocBLAS); dW's long contraction over
// every output pixel is split into chunks whose partial products a reduction
// kernel sums (and masks).  The range masks, the unrolling, the transpose of
// dY and the gather are the kernels below.
#include <rocblas/rocblas.h>

#include <map>
#include <mutex>

#include "common.h"

namespace rxnn {
namespace {

__global__ __launch_bounds__(256) void k_bw_clip(const float* __restrict__ X, int64_t n,
                                                 float x_max, float* __restrict__ out) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x)
    out[e] = fminf(fmaxf(X[e], 0.0f), x_max);
}

__global__ __launch_bounds__(256) void k_bw_mask_x(float* __restrict__ dX,
                                                   const float* __restrict__ X, int64_t n,
                                                   float x_max) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    const float x = X[e];
    if (!(x >= 0.0f && x <= x_max)) dX[e] = 0.0f;
  }
}

__global__ __launch_bounds__(256) void k_bw_mask_w(float* __restrict__ dW,
                                                   const float* __restrict__ W, int64_t n,
                                                   float wmax_fixed, const float* d_wmax) {
  const float wmax = wmax_fixed > 0.0f ? wmax_fixed : *d_wmax;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x)
    if (!(fabsf(W[e]) <= wmax)) dW[e] = 0.0f;
}

// Output pixel bv -> (img, oy, ox).
struct PixDiv {
  FastDiv wo, ho;
};

// Patches of the clipped input, k-major: colsT[k][bv], bv = (img ho + oy) wo + ox.
// Grid: x over output pixels, y = kernel tap ky kw + kx, z = ci.
__global__ __launch_bounds__(256) void k_bw_im2col(const float* __restrict__ X,
                                                   rxnn_conv_desc cd, PixDiv pd, float x_max,
                                                   float* __restrict__ cols) {
  const int ho = (int)pd.ho.d, wo = (int)pd.wo.d;
  const int Bv = cd.n * ho * wo;
  const int bv = blockIdx.x * 256 + threadIdx.x;
  if (bv >= Bv) return;
  const int tap = blockIdx.y, ci = blockIdx.z;
  const int ky = tap / cd.kw, kx = tap - ky * cd.kw;   // uniform per block
  const int t = (int)div_by((uint32_t)bv, pd.wo);
  const int ox = bv - t * wo;
  const int img = (int)div_by((uint32_t)t, pd.ho);
  const int oy = t - img * ho;
  const int y = oy * cd.stride - cd.pad + ky, x = ox * cd.stride - cd.pad + kx;
  float v = 0.0f;
  if (y >= 0 && y < cd.h && x >= 0 && x < cd.w)
    v = fminf(fmaxf(X[(((int64_t)img * cd.c_in + ci) * cd.h + y) * cd.w + x], 0.0f), x_max);
  cols[(int64_t)(ci * cd.kh * cd.kw + tap) * Bv + bv] = v;
}

// dY (n, c_out, ho, wo) -> rows[bv][q], through 64 x 64 tiles in LDS.
__global__ __launch_bounds__(256) void k_bw_rows(const float* __restrict__ dY, int Bv, int Q,
                                                 FastDiv hw, float* __restrict__ rows) {
  __shared__ float tile[64][65];
  const int bv0 = blockIdx.x * 64;
  const int q0 = blockIdx.y * 64;
  const int t = threadIdx.x & 63, u = threadIdx.x >> 6;
  {
    const int bv = bv0 + t;   // pixels bv0 + t of channel q0 + i: contiguous in NCHW
    const int img = (int)div_by((uint32_t)bv, hw), pix = bv - img * (int)hw.d;
    for (int i = u; i < 64; i += 4) {
      const int q = q0 + i;
      if (bv < Bv && q < Q) tile[i][t] = dY[((int64_t)img * Q + q) * hw.d + pix];
    }
  }
  __syncthreads();
  for (int i = u; i < 64; i += 4) {   // row bv0 + i, columns q0 + t
    const int bv = bv0 + i;
    const int q = q0 + t;
    if (bv < Bv && q < Q) rows[(int64_t)bv * Q + q] = tile[t][i];
  }
}

// dX[img][ci][y][x] = sum over the taps whose patch reads (y, x) of the patch
// gradient dcolsT[k][bv], masked where the DAC clipped the input.  Grid: x
// over the pixels of one channel plane, y = ci, z = img.  A tap reads (y, x)
// from output pixel ((y + pad - ky) / stride, (x + pad - kx) / stride) when
// both divisions are exact and in range.
template <bool S1>
__global__ __launch_bounds__(256) void k_bw_col2im(const float* __restrict__ dcols,
                                                   const float* __restrict__ X, rxnn_conv_desc cd,
                                                   int ho, int wo, FastDiv wdiv, FastDiv sdiv,
                                                   float x_max, float* __restrict__ dX) {
  const int Bv = cd.n * ho * wo;
  const int pix = blockIdx.x * 256 + threadIdx.x;
  if (pix >= cd.h * cd.w) return;
  const int ci = blockIdx.y, img = blockIdx.z;
  const int y = (int)div_by((uint32_t)pix, wdiv);
  const int x = pix - y * cd.w;
  const float* base = dcols + (int64_t)ci * cd.kh * cd.kw * Bv + (int64_t)img * ho * wo;
  float acc = 0.0f;
  for (int ky = 0; ky < cd.kh; ++ky) {
    const int ty = y + cd.pad - ky;
    if (ty < 0) break;                      // ty falls as ky grows
    int oy = ty;
    if (!S1) {
      oy = (int)div_by((uint32_t)ty, sdiv);
      if (oy * cd.stride != ty) continue;
    }
    if (oy >= ho) continue;
    for (int kx = 0; kx < cd.kw; ++kx) {
      const int tx = x + cd.pad - kx;
      if (tx < 0) break;
      int ox = tx;
      if (!S1) {
        ox = (int)div_by((uint32_t)tx, sdiv);
        if (ox * cd.stride != tx) continue;
      }
      if (ox >= wo) continue;
      acc += base[(int64_t)(ky * cd.kw + kx) * Bv + oy * wo + ox];
    }
  }
  const int64_t e = ((int64_t)img * cd.c_in + ci) * cd.h * cd.w + pix;
  const float xv = X[e];
  dX[e] = (xv >= 0.0f && xv <= x_max) ? acc : 0.0f;
}

// dW = sum of the split-K partial products, masked to |w| <= w_max.
__global__ __launch_bounds__(256) void k_bw_reduce_w(const float* __restrict__ part, int nparts,
                                                     int64_t n, const float* __restrict__ W,
                                                     float wmax_fixed, const float* d_wmax,
                                                     float* __restrict__ dW) {
  const float wmax = wmax_fixed > 0.0f ? wmax_fixed : *d_wmax;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    float acc = 0.0f;
    for (int s = 0; s < nparts; ++s) acc += part[(int64_t)s * n + e];
    dW[e] = fabsf(W[e]) <= wmax ? acc : 0.0f;
  }
}

unsigned grid_for(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (unsigned)(b < 16384 ? (b > 0 ? b : 1) : 16384);
}

std::mutex g_blas_mu;
std::map<int, rocblas_handle> g_blas;   // one handle per device

}  // namespace

// Row-major C_i (m x n) = op(A_i) (m x k) op(B_i) (k x n), i < batch, with
// row strides lda, ldb, ldc and element strides sA, sB, sC between the
// batch's matrices: the column-major product C^T = op(B)^T op(A)^T.
hipError_t bw_gemm_batched(int device, hipStream_t s, bool ta, bool tb, int m, int n, int k,
                           const float* A, int lda, int64_t sA, const float* B, int ldb,
                           int64_t sB, float* C, int ldc, int64_t sC, int batch) {
  std::lock_guard<std::mutex> g(g_blas_mu);
  rocblas_handle h;
  auto it = g_blas.find(device);
  if (it == g_blas.end()) {
    if (rocblas_create_handle(&h) != rocblas_status_success) return hipErrorUnknown;
    g_blas[device] = h;
  } else {
    h = it->second;
  }
  if (rocblas_set_stream(h, s) != rocblas_status_success) return hipErrorUnknown;
  const float one = 1.0f, zero = 0.0f;
  const rocblas_operation oa = ta ? rocblas_operation_transpose : rocblas_operation_none;
  const rocblas_operation ob = tb ? rocblas_operation_transpose : rocblas_operation_none;
  const rocblas_status st =
      batch == 1 ? rocblas_sgemm(h, ob, oa, n, m, k, &one, B, ldb, A, lda, &zero, C, ldc)
                 : rocblas_sgemm_strided_batched(h, ob, oa, n, m, k, &one, B, ldb, sB, A, lda, sA,
                                                 &zero, C, ldc, sC, batch);
  return st == rocblas_status_success ? hipGetLastError() : hipErrorUnknown;
}

hipError_t bw_gemm(int device, hipStream_t s, bool ta, bool tb, int m, int n, int k,
                   const float* A, int lda, const float* B, int ldb, float* C, int ldc) {
  return bw_gemm_batched(device, s, ta, tb, m, n, k, A, lda, 0, B, ldb, 0, C, ldc, 0, 1);
}

hipError_t launch_bw_clip(const float* X, int64_t n, float x_max, float* out, hipStream_t s) {
  hipLaunchKernelGGL(k_bw_clip, dim3(grid_for(n)), dim3(256), 0, s, X, n, x_max, out);
  return hipGetLastError();
}

hipError_t launch_bw_mask_x(float* dX, const float* X, int64_t n, float x_max, hipStream_t s) {
  hipLaunchKernelGGL(k_bw_mask_x, dim3(grid_for(n)), dim3(256), 0, s, dX, X, n, x_max);
  return hipGetLastError();
}

hipError_t launch_bw_mask_w(float* dW, const float* W, int64_t n, const MapScalars& ms,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_bw_mask_w, dim3(grid_for(n)), dim3(256), 0, s, dW, W, n, ms.wmax_fixed,
                     ms.d_wmax);
  return hipGetLastError();
}

hipError_t launch_bw_reduce_w(const float* part, int nparts, const float* W, int64_t n,
                              const MapScalars& ms, float* dW, hipStream_t s) {
  hipLaunchKernelGGL(k_bw_reduce_w, dim3(grid_for(n)), dim3(256), 0, s, part, nparts, n, W,
                     ms.wmax_fixed, ms.d_wmax, dW);
  return hipGetLastError();
}

hipError_t launch_bw_im2col(const float* X, const rxnn_conv_desc& cd, int ho, int wo,
                            float x_max, float* cols, hipStream_t s) {
  const int Bv = cd.n * ho * wo;
  const dim3 grid((unsigned)((Bv + 255) / 256), (unsigned)(cd.kh * cd.kw), (unsigned)cd.c_in);
  const PixDiv pd{fast_div((uint32_t)wo), fast_div((uint32_t)ho)};
  hipLaunchKernelGGL(k_bw_im2col, grid, dim3(256), 0, s, X, cd, pd, x_max, cols);
  return hipGetLastError();
}

hipError_t launch_bw_rows(const float* dY, int64_t Bv, int Q, int hw, float* rows, hipStream_t s) {
  const dim3 grid((unsigned)((Bv + 63) / 64), (unsigned)((Q + 63) / 64));
  hipLaunchKernelGGL(k_bw_rows, grid, dim3(256), 0, s, dY, (int)Bv, Q, fast_div((uint32_t)hw),
                     rows);
  return hipGetLastError();
}

hipError_t launch_bw_col2im(const float* dcols, const float* X, const rxnn_conv_desc& cd, int ho,
                            int wo, float x_max, float* dX, hipStream_t s) {
  const dim3 grid((unsigned)((cd.h * cd.w + 255) / 256), (unsigned)cd.c_in, (unsigned)cd.n);
  const FastDiv wdiv = fast_div((uint32_t)cd.w), sdiv = fast_div((uint32_t)cd.stride);
  if (cd.stride == 1)
    hipLaunchKernelGGL(k_bw_col2im<true>, grid, dim3(256), 0, s, dcols, X, cd, ho, wo, wdiv, sdiv,
                       x_max, dX);
  else
    hipLaunchKernelGGL(k_bw_col2im<false>, grid, dim3(256), 0, s, dcols, X, cd, ho, wo, wdiv,
                       sdiv, x_max, dX);
  return hipGetLastError();
}

}  // namespace rxnn
