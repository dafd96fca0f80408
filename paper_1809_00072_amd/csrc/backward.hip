// Backward pass of model-in-the-loop re-training (Sec. VI, re-training with RxNN):
// the forward pass runs on the crossbar model, the backward pass in floating
// point through the layer's ideal weights with straight-through DAC and ADC
// and the range constraints of the mapping:
//   dX = (dY W^T) * [0 <= x <= x_max]         (inputs the DAC clips: no gradient)
//   dW = clip(X, 0, x_max)^T dY * [|w| <= w_max]
// For a convolution X is its unrolled patch matrix (patch column
// k = (ci kh + ky) kw + kx, Sec. VI).  Both contractions are implicit GEMMs on
// the fp32 matrix cores: their operands are gathered from the NCHW tensors as
// the tiles are staged, so no patch matrix is ever written.
//   dW[k][q]   = sum over output pixels bv of clip(patch[bv][k]) dY[bv][q]
//                (M = P, N = Q, K = the n H_out W_out output pixels, split
//                over workgroups into partial sums that a reduction adds);
//   dX[pix][ci] = sum over taps (ky, kx) and outputs q of W[(ci, ky, kx)][q]
//                dY[img][q][oy][ox], where the tap reads input pixel (y, x)
//                from output pixel (oy, ox) = ((y + pad - ky) / s, (x + pad - kx) / s)
//                when both divisions are exact and in range
//                (M = the n H W input pixels, N = c_in, K = kh kw Q).
// A fully connected layer is the 1 x 1 convolution of 1 x 1 images
// (n = B, c_in = P, c_out = Q).  The generic kernels (k_bw_dw, k_bw_dx) gather
// every operand element by element; 3 x 3 convolutions whose widths are
// multiples of 4 use k_bw_dw3 / k_bw_dx3, which stage whole input or
// output-gradient rows of a pixel chunk in LDS once and read the nine taps
// from them.

#include <algorithm>

#include "common.h"

namespace rxnn {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BT = 64;         // output tile side
constexpr int KB = 32;         // reduction index per staged chunk
constexpr int LDA = BT + 4;    // LDS row stride (floats)
constexpr int NTH = 256;

// Shape of one backward call, prepared on the host.
struct BwGeom {
  int n, c_in, h, w, kh, kw, stride, pad, ho, wo;
  int P, Q, khw;
  int hw_in, hw_out;
  int Bv;                      // n ho wo output pixels
  int npix;                    // n h w input pixels
  FastDiv fd_wo, fd_ho, fd_w, fd_hwin, fd_kw, fd_khw, fd_Q, fd_s;
  float x_max;
};

// Workgroups are dispatched to the 8 XCDs in turn, each with its own L2: this
// renumbering gives every XCD a contiguous range of logical tiles.
__device__ __forceinline__ int xcd_tile(int i, int n) {
  const int q = n >> 3, r = n & 7, x = i & 7, j = i >> 3;
  return x * q + min(x, r) + j;
}

// One wave's 32 x 32 quarter of a 64 x 64 tile as 2 x 2 blocks of 16 x 16
// (v_mfma_f32_16x16x4f32): in a step over k .. k + 3, lane l supplies
// A[l % 16][k + l / 16] and B[k + l / 16][l % 16]; block (i, j) holds
// D[4 (l / 16) + v][l % 16] in element v of lane l.
struct Quarter {
  f32x4 acc[2][2];
  int wr, wc, lr, lc;
  __device__ __forceinline__ void init(int tid) {
    const int wv = tid >> 6, lane = tid & 63;
    wr = wv >> 1;
    wc = wv & 1;
    lr = lane >> 4;
    lc = lane & 15;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // one chunk: As[k][m], Bs[k][n] in LDS, k-major with row stride LDA
  __device__ __forceinline__ void step(const float* As, const float* Bs) {
#pragma unroll
    for (int k4 = 0; k4 < KB; k4 += 4) {
      float a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = As[(k4 + lr) * LDA + wr * 32 + i * 16 + lc];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = Bs[(k4 + lr) * LDA + wc * 32 + j * 16 + lc];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
  __device__ __forceinline__ int row(int i, int v) const { return wr * 32 + i * 16 + 4 * lr + v; }
  __device__ __forceinline__ int col(int j) const { return wc * 32 + j * 16 + lc; }
};

__device__ __forceinline__ float clip(float x, float x_max) { return fminf(fmaxf(x, 0.0f), x_max); }

// ---------------------------------------------------------------------------
// dW tile (k0 .. k0 + 63 patch columns) x (q0 .. q0 + 63 outputs) over the
// output pixels [bv_begin, bv_end) of split `split`.  A thread stages pixel
// tid % 32 of a chunk for 8 patch columns (and 8 outputs): k = k0 + tid / 32 +
// 8 i.  nsplit = 1: the masked gradient goes straight to dW; else the tile's
// partial sum goes to out + split P Q for k_bw_reduce_w.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTH) void k_bw_dw(BwGeom gm, const float* __restrict__ X,
                                               const float* __restrict__ dY,
                                               const float* __restrict__ W, float wmax_fixed,
                                               const float* d_wmax, int nsplit, int kc,
                                               float* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) float smem[2 * KB * LDA];
  float* As = smem;
  float* Bs = smem + KB * LDA;
  const int tid = threadIdx.x;
  const int nkb = (gm.P + BT - 1) / BT, nqb = (gm.Q + BT - 1) / BT;
  const int lin = xcd_tile((int)blockIdx.x, (int)gridDim.x);   // splits outermost
  const int split = lin / (nkb * nqb), tile = lin % (nkb * nqb);
  const int k0 = (tile / nqb) * BT, q0 = (tile % nqb) * BT;
  const int bv_begin = split * kc, bv_end = min(gm.Bv, bv_begin + kc);
  const int bl = tid & 31, grp = tid >> 5;
  // this thread's patch columns: channel plane offset and tap
  int xoff[8], ky[8], kx[8];
  bool kval[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int k = k0 + grp + 8 * i;
    kval[i] = k < gm.P;
    const int kk = kval[i] ? k : 0;
    const int ci = (int)div_by((uint32_t)kk, gm.fd_khw), tap = kk - ci * gm.khw;
    ky[i] = (int)div_by((uint32_t)tap, gm.fd_kw);
    kx[i] = tap - ky[i] * gm.kw;
    xoff[i] = ci * gm.hw_in;
  }
  float ra[8], rb[8];
  auto load = [&](int c0) {
    const int bv = c0 + bl;
    const bool ok = bv < bv_end;
    const int bvc = ok ? bv : bv_begin;
    const int t = (int)div_by((uint32_t)bvc, gm.fd_wo);
    const int ox = bvc - t * gm.wo;
    const int img = (int)div_by((uint32_t)t, gm.fd_ho);
    const int oy = t - img * gm.ho;
    const float* Xi = X + (int64_t)img * gm.c_in * gm.hw_in;
    const float* dYi = dY + (int64_t)img * gm.Q * gm.hw_out + oy * gm.wo + ox;
    const int y0 = oy * gm.stride - gm.pad, x0 = ox * gm.stride - gm.pad;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int y = y0 + ky[i], x = x0 + kx[i];
      const bool in = ok && kval[i] && y >= 0 && y < gm.h && x >= 0 && x < gm.w;
      ra[i] = in ? clip(Xi[xoff[i] + y * gm.w + x], gm.x_max) : 0.0f;
      const int q = q0 + grp + 8 * i;
      rb[i] = (ok && q < gm.Q) ? dYi[(int64_t)q * gm.hw_out] : 0.0f;
    }
  };
  Quarter qt;
  qt.init(tid);
  if (bv_begin < bv_end) load(bv_begin);
#pragma unroll 1
  for (int c0 = bv_begin; c0 < bv_end; c0 += KB) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      As[bl * LDA + grp + 8 * i] = ra[i];
      Bs[bl * LDA + grp + 8 * i] = rb[i];
    }
    __syncthreads();
    if (c0 + KB < bv_end) load(c0 + KB);   // in flight during this chunk's products
    qt.step(As, Bs);
    __syncthreads();
  }
  float wmax = 0.0f;
  if (nsplit == 1) wmax = wmax_fixed > 0.0f ? wmax_fixed : *d_wmax;
  float* dst = nsplit == 1 ? out : out + (int64_t)split * gm.P * gm.Q;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int k = k0 + qt.row(i, v), q = q0 + qt.col(j);
        if (k >= gm.P || q >= gm.Q) continue;
        const int64_t e = (int64_t)k * gm.Q + q;
        const float a = qt.acc[i][j][v];
        dst[e] = nsplit == 1 ? (fabsf(W[e]) <= wmax ? a : 0.0f) : a;
      }
}

// ---------------------------------------------------------------------------
// dX tile: input pixels p0 .. p0 + 63 x channels c0 .. c0 + 63, reduction over
// kk = tap Q + q.  A thread stages pixel (and channel) tid % 64 for 8 values
// of kk: kk0 + tid / 64 + 4 i.  The masked result leaves through LDS so that
// lanes write consecutive pixels of one channel.
// ---------------------------------------------------------------------------
template <bool S1>
__global__ __launch_bounds__(NTH) void k_bw_dx(BwGeom gm, const float* __restrict__ X,
                                               const float* __restrict__ dY,
                                               const float* __restrict__ W,
                                               float* __restrict__ dX) {
  __shared__ __attribute__((aligned(16))) float smem[2 * KB * LDA];
  float* As = smem;
  float* Bs = smem + KB * LDA;
  const int tid = threadIdx.x;
  const int ncb = (gm.c_in + BT - 1) / BT;
  const int lin = xcd_tile((int)blockIdx.x, (int)gridDim.x);
  const int p0 = (lin / ncb) * BT, c0 = (lin % ncb) * BT;
  const int K = gm.khw * gm.Q;
  const int pl = tid & 63, grp = tid >> 6;
  // this thread's pixel (rows of A) and channel (columns of B)
  const int pix = min(p0 + pl, gm.npix - 1);
  const bool pix_ok = p0 + pl < gm.npix;
  const int img = (int)div_by((uint32_t)pix, gm.fd_hwin);
  const int r = pix - img * gm.hw_in;
  const int y = (int)div_by((uint32_t)r, gm.fd_w), x = r - y * gm.w;
  const float* dYi = dY + (int64_t)img * gm.Q * gm.hw_out;
  const int ci = c0 + pl;
  const bool ci_ok = ci < gm.c_in;
  float ra[8], rb[8];
  auto load = [&](int kk0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int kk = kk0 + grp + 4 * i;
      const bool kok = kk < K;
      const int kc = kok ? kk : 0;
      const int tap = (int)div_by((uint32_t)kc, gm.fd_Q), q = kc - tap * gm.Q;
      const int ky = (int)div_by((uint32_t)tap, gm.fd_kw), kx = tap - ky * gm.kw;
      const int ty = y + gm.pad - ky, tx = x + gm.pad - kx;
      int oy = ty, ox = tx;
      bool ok = kok && pix_ok && ty >= 0 && tx >= 0;
      if (!S1) {
        oy = (int)div_by((uint32_t)max(ty, 0), gm.fd_s);
        ox = (int)div_by((uint32_t)max(tx, 0), gm.fd_s);
        ok = ok && oy * gm.stride == ty && ox * gm.stride == tx;
      }
      ok = ok && oy < gm.ho && ox < gm.wo;
      ra[i] = ok ? dYi[(int64_t)q * gm.hw_out + oy * gm.wo + ox] : 0.0f;
      rb[i] = (kok && ci_ok) ? W[((int64_t)ci * gm.khw + tap) * gm.Q + q] : 0.0f;
    }
  };
  Quarter qt;
  qt.init(tid);
  load(0);
#pragma unroll 1
  for (int kk0 = 0; kk0 < K; kk0 += KB) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      As[(grp + 4 * i) * LDA + pl] = ra[i];
      Bs[(grp + 4 * i) * LDA + pl] = rb[i];
    }
    __syncthreads();
    if (kk0 + KB < K) load(kk0 + KB);
    qt.step(As, Bs);
    __syncthreads();
  }
  // D[pixel][channel] -> LDS transposed [channel][pixel], then each wave
  // writes 16 channels, 64 consecutive pixels per instruction
  float* tb = smem;   // 64 x (64 + 1) floats fit the two staging buffers
  static_assert(BT * (BT + 1) <= 2 * KB * LDA, "the transposed tile fits");
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) tb[qt.col(j) * (BT + 1) + qt.row(i, v)] = qt.acc[i][j][v];
  __syncthreads();
  const int wv = tid >> 6;
  if (pix_ok) {
#pragma unroll 4
    for (int cc = wv; cc < BT; cc += 4) {
      const int ch = c0 + cc;
      if (ch >= gm.c_in) break;
      const int64_t e = ((int64_t)img * gm.c_in + ch) * gm.hw_in + r;
      const float xv = X[e];
      dX[e] = (xv >= 0.0f && xv <= gm.x_max) ? tb[cc * (BT + 1) + pl] : 0.0f;
    }
  }
}

// dW = sum of the split partial products, masked to |w| <= w_max.  A block
// takes 64 consecutive elements; wave g adds the splits g, g + 4, ... with
// eight loads in flight, and the four wave sums meet in LDS.
__global__ __launch_bounds__(256) void k_bw_reduce_w(const float* __restrict__ part, int nparts,
                                                     int64_t n, const float* __restrict__ W,
                                                     float wmax_fixed, const float* d_wmax,
                                                     float* __restrict__ dW) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int64_t e = (int64_t)blockIdx.x * 64 + lane;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (e < n) {
    int sp = g;
    for (; sp + 28 < nparts; sp += 32) {
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] += part[(int64_t)(sp + 4 * k) * n + e];
    }
    for (; sp < nparts; sp += 4) acc[0] += part[(int64_t)sp * n + e];
  }
  red[g][lane] = ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
  __syncthreads();
  if (g == 0 && e < n) {
    const float wmax = wmax_fixed > 0.0f ? wmax_fixed : *d_wmax;
    const float sum = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
    dW[e] = fabsf(W[e]) <= wmax ? sum : 0.0f;
  }
}

BwGeom bw_geom(const rxnn_conv_desc& cd, int P, int Q, float x_max) {
  BwGeom g;
  g.n = cd.n;
  g.c_in = cd.c_in;
  g.h = cd.h;
  g.w = cd.w;
  g.kh = cd.kh;
  g.kw = cd.kw;
  g.stride = cd.stride;
  g.pad = cd.pad;
  g.ho = (cd.h + 2 * cd.pad - cd.kh) / cd.stride + 1;
  g.wo = (cd.w + 2 * cd.pad - cd.kw) / cd.stride + 1;
  g.P = P;
  g.Q = Q;
  g.khw = cd.kh * cd.kw;
  g.hw_in = cd.h * cd.w;
  g.hw_out = g.ho * g.wo;
  g.Bv = cd.n * g.hw_out;
  g.npix = cd.n * g.hw_in;
  g.fd_wo = fast_div((uint32_t)g.wo);
  g.fd_ho = fast_div((uint32_t)g.ho);
  g.fd_w = fast_div((uint32_t)g.w);
  g.fd_hwin = fast_div((uint32_t)g.hw_in);
  g.fd_kw = fast_div((uint32_t)g.kw);
  g.fd_khw = fast_div((uint32_t)g.khw);
  g.fd_Q = fast_div((uint32_t)Q);
  g.fd_s = fast_div((uint32_t)cd.stride);
  g.x_max = x_max;
  return g;
}

// ---------------------------------------------------------------------------
// 3 x 3 kernels: the input (dW) or output gradient (dX) rows that a chunk of
// 64 consecutive pixels of one image touches are staged in LDS, and the nine
// taps read them at fixed offsets.  Image column x sits at LDS column x + 4 so
// that rows move as aligned 16-byte vectors; the border columns around them
// are zeroed once per workgroup and never written again.  The loads of the
// next chunk are in flight while the current one is multiplied.
// ---------------------------------------------------------------------------

// Zeros in device memory: what a masked lane of a staging load reads (a
// file-scope device array starts zeroed and is never written).
__device__ __attribute__((aligned(16))) float bw_zero[4];

// Halo geometry prepared on the host.
struct Halo {
  int HS;            // LDS row length (multiple of 4, >= w + pad + 4)
  int HR;            // halo rows per chunk
  int CS;            // LDS stride of one channel (dW) or output (dX) halo
  int n4;            // 16-byte vectors staged per chunk (dW: X halo; dX: dY halo)
  int upi;           // 64-pixel chunks per image
  int units;         // n upi
  int nsplit;        // dW: pixel splits
  int ncb, nqb;      // dW: blocks of 16 channels, of 64 outputs; dX: blocks of 64 channels
  FastDiv fd_upi;
  FastDiv fd_plane;  // vectors per staged plane: HR (row length) / 4
  FastDiv fd_row;    // vectors per staged row: (row length) / 4
};

constexpr int YS = 68;       // dW: LDS row of the output gradient (64 pixels + 4)
constexpr int DW_X4 = 6;     // dW: X halo vectors per thread (n4 <= 1536)
constexpr int QC = 8;        // dX: outputs per staged chunk
constexpr int WSTR = 12;     // dX: LDS row of W (QC + 4)
constexpr int WTAP = 64 * WSTR;
constexpr int DX_PIX = 128;  // dX: input pixels per workgroup
constexpr int DX_Y4 = 4;     // dX: dY halo vectors per thread (n4 <= 1024)
constexpr int DX_W4 = 9 * 64 * QC / 4 / NTH + 1;   // W vectors per thread (1152 in all)

__device__ __forceinline__ float4 clip4(float4 v, float x_max) {
  return make_float4(clip(v.x, x_max), clip(v.y, x_max), clip(v.z, x_max), clip(v.w, x_max));
}

// dW tile: 16 channels x 9 taps x 64 outputs, over the chunks
// [units split / nsplit, units (split + 1) / nsplit).  Wave v takes outputs
// 16 v .. 16 v + 15; lane (c, j) = (l % 16, l / 16) reads channel c of pixel
// 4 s + j in step s.  Without a split the masked gradient goes to `out` = dW,
// else the partial sum to out + split P Q.  Needs w and W_out divisible by 4.
__global__ __launch_bounds__(NTH) void k_bw_dw3(BwGeom gm, Halo hl, const float* __restrict__ X,
                                                const float* __restrict__ dY,
                                                const float* __restrict__ W, float wmax_fixed,
                                                const float* d_wmax, float* __restrict__ out) {
  extern __shared__ __attribute__((aligned(16))) float sm3[];
  float* Xs = sm3;                          // 16 channels x CS
  float* Ys = Xs + 16 * hl.CS;              // 64 outputs x YS
  int* pofs = (int*)(Ys + 64 * YS);         // pixel -> halo offset
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 15, j = lane >> 4;
  const int tiles = hl.ncb * hl.nqb;
  const int lin = xcd_tile((int)blockIdx.x, (int)gridDim.x);
  const int split = lin / tiles, tile = lin - split * tiles;
  const int ci0 = (tile / hl.nqb) * 16, q0 = (tile % hl.nqb) * 64;
  const int u0 = (int)((int64_t)split * hl.units / hl.nsplit);
  const int u1 = (int)((int64_t)(split + 1) * hl.units / hl.nsplit);
  const int s = gm.stride, HS = hl.HS;
  const int w4 = gm.w >> 2;
  for (int e = tid; e < 16 * hl.CS; e += NTH) Xs[e] = 0.0f;   // border columns
  // this thread's X vectors: (channel, row, column) of the flat index
  // tid + NTH i, and the output-gradient vectors (q, pixels) = (f / 16, f % 16)
  float4 rX[DW_X4], rY[4];
  auto fetch = [&](int u) {
    const int img = (int)div_by((uint32_t)u, hl.fd_upi);
    const int p0 = (u - img * hl.upi) * 64;
    const int len = min(64, gm.hw_out - p0);
    const float* ysrc = dY + ((int64_t)img * gm.Q + q0) * gm.hw_out + p0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int f = tid + NTH * i, q = f >> 4, p = 4 * (f & 15);
      const bool ok = q0 + q < gm.Q && p < len;
      rY[i] = *reinterpret_cast<const float4*>(ok ? ysrc + (int64_t)q * gm.hw_out + p : bw_zero);
    }
    const int y0 = (int)div_by((uint32_t)p0, gm.fd_wo) * s - gm.pad;
    const float* xsrc = X + ((int64_t)img * gm.c_in + ci0) * gm.hw_in;
#pragma unroll
    for (int i = 0; i < DW_X4; ++i) {
      const int f = tid + NTH * i;
      const int cl = (int)div_by((uint32_t)f, hl.fd_plane);
      const int r = f - cl * (int)hl.fd_plane.d;
      const int hr = (int)div_by((uint32_t)r, hl.fd_row);
      const int y = y0 + hr;
      const bool ok = f < hl.n4 && ci0 + cl < gm.c_in && y >= 0 && y < gm.h;
      const int64_t off = (int64_t)cl * gm.hw_in + (int64_t)y * gm.w + 4 * (r - hr * w4);
      rX[i] = *reinterpret_cast<const float4*>(ok ? xsrc + off : bw_zero);
    }
  };
  auto store = [&](int u) {
    if (tid < 64) {
      const int img = (int)div_by((uint32_t)u, hl.fd_upi);
      const int p0 = (u - img * hl.upi) * 64;
      const int len = min(64, gm.hw_out - p0);
      // pixels past the chunk read LDS columns 0 .. 2, which are never written
      // (image columns start at 4) and stay zero: their steps add exactly 0
      int po = gm.pad - 4;
      if (tid < len) {
        const int oy_first = (int)div_by((uint32_t)p0, gm.fd_wo);
        const int pix = p0 + tid;
        const int oy = (int)div_by((uint32_t)pix, gm.fd_wo);
        po = (oy - oy_first) * s * HS + (pix - oy * gm.wo) * s;
      }
      pofs[tid] = po;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int f = tid + NTH * i;
      *reinterpret_cast<float4*>(Ys + (f >> 4) * YS + 4 * (f & 15)) = rY[i];
    }
#pragma unroll
    for (int i = 0; i < DW_X4; ++i) {
      const int f = tid + NTH * i;
      if (f < hl.n4) {
        const int cl = (int)div_by((uint32_t)f, hl.fd_plane);
        const int r = f - cl * (int)hl.fd_plane.d;
        const int hr = (int)div_by((uint32_t)r, hl.fd_row);
        *reinterpret_cast<float4*>(Xs + cl * hl.CS + hr * HS + 4 + 4 * (r - hr * w4)) =
            clip4(rX[i], gm.x_max);
      }
    }
  };
  f32x4 acc[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int abase = c * hl.CS + 4 - gm.pad;
  const int bbase = (16 * wave + c) * YS + j;
  if (u0 < u1) fetch(u0);
#pragma unroll 1
  for (int u = u0; u < u1; ++u) {
    __syncthreads();   // the previous chunk's reads (and the border zeroing) are done
    store(u);
    __syncthreads();
    if (u + 1 < u1) fetch(u + 1);
    const int len = min(64, gm.hw_out - (u - (int)div_by((uint32_t)u, hl.fd_upi) * hl.upi) * 64);
    auto step = [&](int k4, int po) {
      const int a0 = abase + po;
      const float b = Ys[bbase + 4 * k4];
#pragma unroll
      for (int ky = 0; ky < 3; ++ky) {
        const int ar = a0 + ky * HS;
#pragma unroll
        for (int kx = 0; kx < 3; ++kx)
          acc[ky * 3 + kx] =
              __builtin_amdgcn_mfma_f32_16x16x4f32(Xs[ar + kx], b, acc[ky * 3 + kx], 0, 0, 0);
      }
    };
    // groups of four steps; pixels past the chunk contribute zeros
#pragma unroll 1
    for (int g = 0; g < len; g += 16) {
      int po[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) po[k] = pofs[g + 4 * k + j];
#pragma unroll
      for (int k = 0; k < 4; ++k) step((g >> 2) + k, po[k]);
    }
  }
  float wmax = 0.0f;
  if (hl.nsplit == 1) wmax = wmax_fixed > 0.0f ? wmax_fixed : *d_wmax;
  float* dst = hl.nsplit == 1 ? out : out + (int64_t)split * gm.P * gm.Q;
  const int q = q0 + 16 * wave + c;
  if (q < gm.Q) {
#pragma unroll
    for (int t = 0; t < 9; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int ci = ci0 + 4 * j + v;
        if (ci >= gm.c_in) continue;
        const int64_t e = ((int64_t)ci * 9 + t) * gm.Q + q;
        const float a = acc[t][v];
        dst[e] = hl.nsplit == 1 ? (fabsf(W[e]) <= wmax ? a : 0.0f) : a;
      }
  }
}

// dX tile of a stride-1 3 x 3 convolution: 128 input pixels of one image x 64
// channels, reduction over (tap, output q) with the output gradient staged QC
// outputs at a time.  Wave v takes pixels 32 v .. 32 v + 31 in two blocks of
// 16; lane (c, j) supplies pixel 32 v + 16 a + c of block a and output 4 s + j
// of step s, and channel 16 b + c of block b.  Needs w, W_out and Q divisible
// by 4.
__global__ __launch_bounds__(NTH) void k_bw_dx3(BwGeom gm, Halo hl, const float* __restrict__ X,
                                                const float* __restrict__ dY,
                                                const float* __restrict__ W,
                                                float* __restrict__ dX) {
  extern __shared__ __attribute__((aligned(16))) float sm3[];
  float* Ys = sm3;                  // QC outputs x CS: rows oy0 .., column ox at ox + 4
  float* Ws = Ys + QC * hl.CS;      // 9 taps x 64 channels x WSTR
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 15, j = lane >> 4;
  const int lin = xcd_tile((int)blockIdx.x, (int)gridDim.x);
  const int unit = lin / hl.ncb, ci0 = (lin - unit * hl.ncb) * 64;
  const int img = (int)div_by((uint32_t)unit, hl.fd_upi);
  const int p0 = (unit - img * hl.upi) * DX_PIX;
  const int len = min(DX_PIX, gm.hw_in - p0);
  const int y_first = (int)div_by((uint32_t)p0, gm.fd_w);
  const int HS = hl.HS;
  const int oy0 = y_first + gm.pad - 2;
  const int wo4 = gm.wo >> 2;
  for (int e = tid; e < QC * hl.CS; e += NTH) Ys[e] = 0.0f;   // border columns
  // this lane's two pixels (clamped into the chunk; rows past it are not stored)
  int abase[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int pp = p0 + min(32 * wave + 16 * a + c, len - 1);
    const int py = (int)div_by((uint32_t)pp, gm.fd_w);
    abase[a] = j * hl.CS + (py - y_first) * HS + (pp - py * gm.w) + gm.pad + 4;
  }
  const float* ysrc = dY + (int64_t)img * gm.Q * gm.hw_out;
  // W rows (channel, tap) r = f / 2 of the block's 9 x 64, outputs 4 (f % 2) ..
  const int wrows = 9 * min(64, gm.c_in - ci0);
  const float* wsrc = W + (int64_t)ci0 * 9 * gm.Q;
  float4 rY[DX_Y4], rW[DX_W4];
  auto fetch = [&](int qc0) {
#pragma unroll
    for (int i = 0; i < DX_Y4; ++i) {
      const int f = tid + NTH * i;
      const int ql = (int)div_by((uint32_t)f, hl.fd_plane);
      const int r = f - ql * (int)hl.fd_plane.d;
      const int hr = (int)div_by((uint32_t)r, hl.fd_row);
      const int oy = oy0 + hr, q = qc0 + ql;
      const bool ok = f < hl.n4 && q < gm.Q && oy >= 0 && oy < gm.ho;
      const int64_t off = (int64_t)q * gm.hw_out + (int64_t)oy * gm.wo + 4 * (r - hr * wo4);
      rY[i] = *reinterpret_cast<const float4*>(ok ? ysrc + off : bw_zero);
    }
#pragma unroll
    for (int i = 0; i < DX_W4; ++i) {
      const int f = tid + NTH * i, r = f >> 1, q = qc0 + 4 * (f & 1);
      const bool ok = r < wrows && q < gm.Q;
      rW[i] = *reinterpret_cast<const float4*>(ok ? wsrc + (int64_t)r * gm.Q + q : bw_zero);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < DX_Y4; ++i) {
      const int f = tid + NTH * i;
      if (f < hl.n4) {
        const int ql = (int)div_by((uint32_t)f, hl.fd_plane);
        const int r = f - ql * (int)hl.fd_plane.d;
        const int hr = (int)div_by((uint32_t)r, hl.fd_row);
        *reinterpret_cast<float4*>(Ys + ql * hl.CS + hr * HS + 4 + 4 * (r - hr * wo4)) = rY[i];
      }
    }
#pragma unroll
    for (int i = 0; i < DX_W4; ++i) {
      const int f = tid + NTH * i, r = f >> 1;
      if (r < 9 * 64) {
        const int cl = r / 9, tap = r - cl * 9;
        *reinterpret_cast<float4*>(Ws + tap * WTAP + cl * WSTR + 4 * (f & 1)) = rW[i];
      }
    }
  };
  f32x4 acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  fetch(0);
#pragma unroll 1
  for (int qc0 = 0; qc0 < gm.Q; qc0 += QC) {
    __syncthreads();   // the previous chunk's reads (and the border zeroing) are done
    store();
    __syncthreads();
    if (qc0 + QC < gm.Q) fetch(qc0 + QC);
#pragma unroll
    for (int ky = 0; ky < 3; ++ky)
#pragma unroll
      for (int kx = 0; kx < 3; ++kx) {
        const int toff = (2 - ky) * HS - kx;
        const float* wt = Ws + (ky * 3 + kx) * WTAP + c * WSTR + j;
#pragma unroll
        for (int k4 = 0; k4 < QC / 4; ++k4) {
          float av[2], bv[4];
#pragma unroll
          for (int a = 0; a < 2; ++a) av[a] = Ys[abase[a] + toff + 4 * k4 * hl.CS];
#pragma unroll
          for (int b = 0; b < 4; ++b) bv[b] = wt[16 * b * WSTR + 4 * k4];
#pragma unroll
          for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b)
              acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a], bv[b], acc[a][b], 0, 0, 0);
        }
      }
  }
  // element v of lane (c, j) in blocks (a, b): pixel 32 wave + 16 a + 4 j + v,
  // channel 16 b + c
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int pl = 32 * wave + 16 * a + 4 * j;
    if (pl >= len) continue;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int ci = ci0 + 16 * b + c;
      if (ci >= gm.c_in) continue;
      const int64_t e = ((int64_t)img * gm.c_in + ci) * gm.hw_in + p0 + pl;
      const float4 xv = *reinterpret_cast<const float4*>(X + e);
      float4 o;
      o.x = (xv.x >= 0.0f && xv.x <= gm.x_max) ? acc[a][b][0] : 0.0f;
      o.y = (xv.y >= 0.0f && xv.y <= gm.x_max) ? acc[a][b][1] : 0.0f;
      o.z = (xv.z >= 0.0f && xv.z <= gm.x_max) ? acc[a][b][2] : 0.0f;
      o.w = (xv.w >= 0.0f && xv.w <= gm.x_max) ? acc[a][b][3] : 0.0f;
      *reinterpret_cast<float4*>(dX + e) = o;
    }
  }
}

// 3 x 3 plans.  dW: a chunk of 64 output pixels spans `span` output rows and
// (span - 1) stride + 3 input rows; the channel stride is 4 mod 8 words so
// that the 16 channels of a read fall in distinct LDS banks.  dX (stride 1):
// 128 input pixels read span + 2 output-gradient rows; the per-output stride
// is 16 mod 64 words so that the 4 outputs of a read fall 16 banks apart.
// Rows move as 16-byte vectors: the widths (and dX's Q) must be multiples of
// 4.  lds = 0: the shape is served by the generic kernels.
struct HaloPlan {
  Halo h;
  size_t lds;
};

constexpr size_t kHaloLds = 64 * 1024;

int round4(int v) { return (v + 3) & ~3; }

HaloPlan dw3_plan(const rxnn_conv_desc& cd, int P, int Q) {
  HaloPlan r{};
  if (cd.kh != 3 || cd.kw != 3 || cd.pad > 4) return r;
  const BwGeom g = bw_geom(cd, P, Q, 0.0f);
  if (g.w % 4 || g.wo % 4) return r;
  const int span = std::min(g.ho, (63 + g.wo - 1) / g.wo + 1);
  r.h.HS = round4(g.w + g.pad + 4);
  r.h.HR = (span - 1) * g.stride + 3;
  int cs = r.h.HR * r.h.HS;
  while (cs % 8 != 4) ++cs;
  r.h.CS = cs;
  r.h.n4 = 16 * r.h.HR * (g.w / 4);
  if (r.h.n4 > DW_X4 * NTH) return r;
  const size_t lds = ((size_t)16 * cs + 64 * YS + 64) * sizeof(float);
  r.h.upi = (g.hw_out + 63) / 64;
  const int64_t units = (int64_t)g.n * r.h.upi;
  r.h.ncb = (g.c_in + 15) / 16;
  r.h.nqb = (Q + 63) / 64;
  const int64_t tiles = (int64_t)r.h.ncb * r.h.nqb;
  // about 512 workgroups (two per CU), each on whole chunks; the partial sums
  // within 2^24 floats
  int64_t sp = std::max<int64_t>(1, (512 + tiles - 1) / tiles);
  sp = std::min<int64_t>({sp, units, std::max<int64_t>(1, ((int64_t)1 << 24) / ((int64_t)P * Q))});
  if (lds > kHaloLds || units > INT32_MAX || tiles * sp >= ((int64_t)1 << 24)) return r;
  r.h.units = (int)units;
  r.h.nsplit = (int)sp;
  r.h.fd_upi = fast_div((uint32_t)r.h.upi);
  r.h.fd_plane = fast_div((uint32_t)(r.h.HR * (g.w / 4)));
  r.h.fd_row = fast_div((uint32_t)(g.w / 4));
  r.lds = lds;
  return r;
}

HaloPlan dx3_plan(const rxnn_conv_desc& cd, int P, int Q) {
  HaloPlan r{};
  if (cd.kh != 3 || cd.kw != 3 || cd.stride != 1) return r;
  const BwGeom g = bw_geom(cd, P, Q, 0.0f);
  if (g.w % 4 || g.wo % 4 || Q % 4) return r;
  const int span = std::min(g.h, (DX_PIX - 1 + g.w - 1) / g.w + 1);
  r.h.HS = round4(std::max(g.w + g.pad + 4, g.wo + 4));
  r.h.HR = span + 2;
  int cs = r.h.HR * r.h.HS;
  while (cs % 64 != 16) ++cs;
  r.h.CS = cs;
  r.h.n4 = QC * r.h.HR * (g.wo / 4);
  if (r.h.n4 > DX_Y4 * NTH) return r;
  const size_t lds = ((size_t)QC * cs + 9 * WTAP) * sizeof(float);
  r.h.upi = (g.hw_in + DX_PIX - 1) / DX_PIX;
  const int64_t units = (int64_t)g.n * r.h.upi;
  r.h.ncb = (g.c_in + 63) / 64;
  if (lds > kHaloLds || units * r.h.ncb >= ((int64_t)1 << 24)) return r;
  r.h.units = (int)units;
  r.h.nsplit = 1;
  r.h.nqb = 1;
  r.h.fd_upi = fast_div((uint32_t)r.h.upi);
  r.h.fd_plane = fast_div((uint32_t)(r.h.HR * (g.wo / 4)));
  r.h.fd_row = fast_div((uint32_t)(g.wo / 4));
  r.lds = lds;
  return r;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

BwPlan bw_plan(const rxnn_conv_desc& cd, int P, int Q, bool vec_ok) {
  BwPlan p;
  const HaloPlan h = vec_ok ? dw3_plan(cd, P, Q) : HaloPlan{};
  if (h.lds) {
    p.nsplit = h.h.nsplit;
    p.kc = 0;
    return p;
  }
  const int64_t ho = (cd.h + 2 * cd.pad - cd.kh) / cd.stride + 1;
  const int64_t wo = (cd.w + 2 * cd.pad - cd.kw) / cd.stride + 1;
  const int64_t Bv = cd.n * ho * wo;
  const int64_t tiles = (int64_t)((P + BT - 1) / BT) * ((Q + BT - 1) / BT);
  // split the pixels so that about 1024 workgroups run, each at least 256
  // pixels, the partials within 2^24 floats
  int64_t s = std::max<int64_t>(1, (1024 + tiles - 1) / tiles);
  s = std::min<int64_t>({s, 64, std::max<int64_t>(1, Bv / 256),
                         std::max<int64_t>(1, ((int64_t)1 << 24) / ((int64_t)P * Q))});
  const int64_t kc = ((Bv + s - 1) / s + KB - 1) / KB * KB;
  p.nsplit = (int)((Bv + kc - 1) / kc);
  p.kc = (int)kc;
  if (p.nsplit < 1) p.nsplit = 1;
  return p;
}

hipError_t launch_bw_dw(const rxnn_conv_desc& cd, int P, int Q, float x_max, const float* X,
                        const float* dY, const float* W, const MapScalars& ms, const BwPlan& plan,
                        float* out, hipStream_t s) {
  const BwGeom g = bw_geom(cd, P, Q, x_max);
  const HaloPlan h = plan.kc == 0 ? dw3_plan(cd, P, Q) : HaloPlan{};
  if (h.lds) {
    if (h.h.nsplit != plan.nsplit) return hipErrorInvalidValue;
    const int64_t grid = (int64_t)h.h.ncb * h.h.nqb * h.h.nsplit;
    hipLaunchKernelGGL(k_bw_dw3, dim3((unsigned)grid), dim3(NTH), h.lds, s, g, h.h, X, dY, W,
                       ms.wmax_fixed, ms.d_wmax, out);
    return hipGetLastError();
  }
  const int64_t tiles = (int64_t)((P + BT - 1) / BT) * ((Q + BT - 1) / BT);
  hipLaunchKernelGGL(k_bw_dw, dim3((unsigned)(tiles * plan.nsplit)), dim3(NTH), 0, s, g, X, dY, W,
                     ms.wmax_fixed, ms.d_wmax, plan.nsplit, plan.kc, out);
  return hipGetLastError();
}

hipError_t launch_bw_dx(const rxnn_conv_desc& cd, int P, int Q, float x_max, const float* X,
                        const float* dY, const float* W, float* dX, hipStream_t s) {
  const BwGeom g = bw_geom(cd, P, Q, x_max);
  const bool vec_ok = aligned16(X) && aligned16(dY) && aligned16(W) && aligned16(dX);
  const HaloPlan h = vec_ok ? dx3_plan(cd, P, Q) : HaloPlan{};
  if (h.lds) {
    const int64_t grid = (int64_t)h.h.units * h.h.ncb;
    hipLaunchKernelGGL(k_bw_dx3, dim3((unsigned)grid), dim3(NTH), h.lds, s, g, h.h, X, dY, W, dX);
    return hipGetLastError();
  }
  const int64_t tiles = (int64_t)((g.npix + BT - 1) / BT) * ((g.c_in + BT - 1) / BT);
  if (cd.stride == 1)
    hipLaunchKernelGGL(k_bw_dx<true>, dim3((unsigned)tiles), dim3(NTH), 0, s, g, X, dY, W, dX);
  else
    hipLaunchKernelGGL(k_bw_dx<false>, dim3((unsigned)tiles), dim3(NTH), 0, s, g, X, dY, W, dX);
  return hipGetLastError();
}

hipError_t launch_bw_reduce_w(const float* part, int nparts, const float* W, int64_t n,
                              const MapScalars& ms, float* dW, hipStream_t s) {
  if ((n + 63) / 64 > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_bw_reduce_w, dim3((unsigned)((n + 63) / 64)), dim3(256), 0, s, part,
                     nparts, n, W, ms.wmax_fixed, ms.d_wmax, dW);
  return hipGetLastError();
}

}  // namespace rxnn
