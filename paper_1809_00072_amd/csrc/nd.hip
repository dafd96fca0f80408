// Model generation by nested dissection: W -> G -> G' for every crossbar
// array of a layer (RxNN Sec. V-A generator steps 1-3; the network of
// Sec. V-B).  The paper reaches G' through one dense MN x MN inverse per tile
// (Eq. 12); the same exact matrix is obtained here with O(S^3) work per tile.
//
// The resistive network of one array is a two-layer grid: row-wire nodes
// a[i][j] (chained by r_row), column-wire nodes b[i][j] (chained by r_col),
// device G[i][j] between a[i][j] and b[i][j]; the driver of row i reaches
// a[i][0] through r_driver + r_row, and column j leaves b[M-1][j] through
// r_sense to the virtual ground.  The tile is embedded in a T x T grid
// (T a power of two, T >= 16) with extra rows above it and extra columns to
// its right holding no devices: such rows and columns carry no current, so the
// embedding is exact.
//
// A block of cells is described by its admittance matrix over its ports (the
// nodes it shares with neighbouring blocks), in the order
//   [left a-nodes | right a-nodes (if not at the right edge) |
//    top b-nodes (if not at the top edge) | bottom b-nodes]
// where a block owns the row-wire edge to the right of each of its cells and
// the column-wire edge below it (so the right / bottom ports are the first
// nodes of the neighbour), and the bottom ports of the last grid row are sink
// terminals behind the sense resistors.  Two blocks merge by adding their
// matrices on the shared nodes and eliminating those nodes (Schur complement).
// Cells merge pairwise, alternately top/bottom and left/right, until one block
// remains whose ports are the T row-input nodes and the T sink terminals.
// Attaching the drivers and eliminating the row-input nodes leaves the
// transfer admittance from the row sources to the sinks, i.e. G'.
//
// Levels up to 16 x 16 cells run in LDS, one workgroup per 16 x 16 block;
// every later merge and the final step is one workgroup that eliminates the
// shared nodes in blocks of 16 (Cholesky of the 16 x 16 pivot block,
// triangular solve of its rows, rank-16 update of the rest).  All arithmetic
// is fp64; wire conductances exceed device conductances by about four orders
// of magnitude, and the elimination of series wires loses about that many
// digits, leaving G' accurate to ~1e-12.  Every wire, driver and sense
// resistance must be positive (zero resistances take the row sweep instead).

#include "common.h"

namespace rxnn {

struct NdArgs {
  MapScalars ms;
  const float* W;
  float* gpt;
  int64_t arr0;          // first array of this chunk
  int T, row_off;        // grid side, first grid row of the tile (T - M)
  double g_r, g_c, g_s, g_d;
  double* buf_in;        // level buffers and scratch (per array strides below)
  double* buf_out;
  double* scratch;
  int64_t in_stride, out_stride, scr_stride;  // doubles per array
  int h, w, vert;        // children size and merge direction (merge kernel)
};

namespace {

constexpr int SB = 16;          // side of the blocks reduced in LDS
constexpr int NTH = 256;
constexpr int LBUF = 6400;      // doubles per LDS level buffer
constexpr int KB = 16;          // pivots per elimination block

__device__ __forceinline__ void ports(int i0, int j0, int h, int w, int T, int& nL, int& nR,
                                      int& nT, int& nB) {
  nL = h;
  nR = (j0 + w < T) ? h : 0;
  nT = (i0 > 0) ? w : 0;
  nB = w;
}

// Where port p of child `ch` (0: top/left, 1: bottom/right) of a merge of two
// h x w blocks at (i0, j0) goes: >= 0 an external port of the merged block,
// < 0 the shared (cut) node -1 - k.
__device__ __forceinline__ int merge_dest(int ch, int p, int i0, int j0, int h, int w, bool vert,
                                          int T) {
  const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
  const bool Rn = j0 + nw < T, Tn = i0 > 0;
  const int oR = nh, oT = nh + (Rn ? nh : 0), oB = oT + (Tn ? nw : 0);
  const int ci = (vert && ch) ? i0 + h : i0, cj = (!vert && ch) ? j0 + w : j0;
  const bool Rc = cj + w < T, Tc = ci > 0;
  int seg, idx = p;  // 0 L, 1 R, 2 T, 3 B
  if (idx < h) seg = 0;
  else {
    idx -= h;
    if (Rc && idx < h) seg = 1;
    else {
      if (Rc) idx -= h;
      if (Tc && idx < w) seg = 2;
      else {
        if (Tc) idx -= w;
        seg = 3;
      }
    }
  }
  if (vert) {
    if (ch == 0) {
      if (seg == 0) return idx;
      if (seg == 1) return oR + idx;
      if (seg == 2) return oT + idx;
      return -1 - idx;
    }
    if (seg == 0) return h + idx;
    if (seg == 1) return oR + h + idx;
    if (seg == 2) return -1 - idx;
    return oB + idx;
  }
  if (ch == 0) {
    if (seg == 0) return idx;
    if (seg == 1) return -1 - idx;
    if (seg == 2) return oT + idx;
    return oB + idx;
  }
  if (seg == 0) return -1 - idx;
  if (seg == 1) return oR + idx;
  if (seg == 2) return oT + w + idx;
  return oB + w + idx;
}

__device__ __forceinline__ int nports(int i0, int j0, int h, int w, int T) {
  int a, b, c, d;
  ports(i0, j0, h, w, T, a, b, c, d);
  return a + b + c + d;
}

// W -> G of the device at grid cell (gi, gj) of array `arr` (0 outside the tile).
__device__ __forceinline__ double cell_conductance(const MapScalars& ms, const float* W,
                                                   double wmax, int64_t arr, int gi, int gj,
                                                   int row_off) {
  const int i = gi - row_off, j = gj;
  if (i < 0 || j >= ms.N) return 0.0;
  const int a = (int)(arr % ms.A);
  const int64_t rc = arr / ms.A;
  const int r = (int)(rc % ms.R), c = (int)(rc / ms.R);
  const int64_t p = (int64_t)r * ms.M + i, q = (int64_t)c * ms.N + j;
  const float wf = (p < ms.P && q < ms.Q) ? W[p * ms.Q + q] : 0.0f;
  const double wv = (double)wf;
  const int side = a & 1, s = a >> 1;
  if (ms.slice_bits == 0) {
    if (!(wmax > 0.0)) return ms.g_min;
    const double s_w = (ms.g_max - ms.g_min) / wmax;
    const double mag = side ? fmax(-wv, 0.0) : fmax(wv, 0.0);
    return ms.g_min + s_w * mag;
  }
  const double lw = (double)((1 << ms.weight_bits) - 1);
  double qv = 0.0;
  if (wmax > 0.0) qv = fmin(lw, rint(fabs(wv) * (lw / wmax)));
  const int64_t qi = (int64_t)qv;
  const int64_t d = (qi >> (ms.slice_bits * s)) & ((1 << ms.slice_bits) - 1);
  const double dG = (ms.g_max - ms.g_min) / (double)((1 << ms.slice_bits) - 1);
  const bool on = side ? (wf < 0.0f) : (wf > 0.0f);
  return on ? ms.g_min + (double)d * dG : ms.g_min;
}

// ---------------------------------------------------------------------------
// Levels 1 x 1 .. 16 x 16 of one 16 x 16 block, in LDS.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTH) void k_nd_block16(NdArgs na) {
  __shared__ double bufA[LBUF];
  __shared__ double bufB[LBUF];
  const int tid = threadIdx.x;
  const int T = na.T;
  const int nsb = T / SB;
  const int64_t la = blockIdx.x / (nsb * nsb);
  const int sb = (int)(blockIdx.x % (nsb * nsb));
  const int I0 = (sb / nsb) * SB, J0 = (sb % nsb) * SB;
  const int64_t arr = na.arr0 + la;
  const MapScalars& ms = na.ms;
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;

  // leaves: one cell per thread, 4 x 4 slots
  {
    const int li = tid / SB, lj = tid % SB;
    const int gi = I0 + li, gj = J0 + lj;
    const double G = cell_conductance(ms, na.W, wmax, arr, gi, gj, na.row_off);
    const bool hasR = gj + 1 < T, hasT = gi > 0;
    const double gv = (gi + 1 < T) ? na.g_c : na.g_s;
    double* Y = bufA + tid * 16;
#pragma unroll
    for (int e = 0; e < 16; ++e) Y[e] = 0.0;
    const int L = 0, R = 1, Tp = hasR ? 2 : 1, B = (hasR ? 2 : 1) + (hasT ? 1 : 0);
    auto st = [&](int p, int q, double g) {
      Y[p * 4 + p] += g;
      Y[q * 4 + q] += g;
      Y[p * 4 + q] -= g;
      Y[q * 4 + p] -= g;
    };
    if (hasR) st(L, R, na.g_r);
    if (hasT) {
      st(L, Tp, G);
      st(Tp, B, gv);
    } else {
      const double ge = G > 0.0 ? (G * gv) / (G + gv) : 0.0;
      st(L, B, ge);
    }
  }
  __syncthreads();

  double* in = bufA;
  double* out = bufB;
  int h = 1, w = 1, ld_in = 4;
  bool vert = true;
  while (h < SB || w < SB) {
    const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
    const int E = 2 * (nh + nw), c = vert ? w : h, ld = E + c, slot = ld * ld;
    const int cols = SB / nw;                    // merged blocks per row of the 16 x 16 block
    const int nmerge = (SB / nh) * cols;
    const int ccols = SB / w;                    // child blocks per row
    for (int e = tid; e < nmerge * slot; e += NTH) out[e] = 0.0;
    __syncthreads();
    for (int ch = 0; ch < 2; ++ch) {
      const int n_child = (ld_in) * (ld_in);
      for (int e = tid; e < nmerge * n_child; e += NTH) {
        const int m = e / n_child, rem = e % n_child;
        const int p = rem / ld_in, q = rem % ld_in;
        const int mi = m / cols, mj = m % cols;
        const int i0 = I0 + mi * nh, j0 = J0 + mj * nw;
        const int np = nports((vert && ch) ? i0 + h : i0, (!vert && ch) ? j0 + w : j0, h, w, T);
        if (p >= np || q >= np) continue;
        const int cm = (vert ? (mi * 2 + ch) * ccols + mj : mi * ccols + mj * 2 + ch);
        const double v = in[cm * ld_in * ld_in + p * ld_in + q];
        int dp = merge_dest(ch, p, i0, j0, h, w, vert, T);
        int dq = merge_dest(ch, q, i0, j0, h, w, vert, T);
        dp = dp >= 0 ? dp : E + (-1 - dp);
        dq = dq >= 0 ? dq : E + (-1 - dq);
        out[m * slot + dp * ld + dq] += v;
      }
      __syncthreads();
    }
    // eliminate the c shared nodes (pivot rows / columns E .. E + c - 1)
    for (int k = 0; k < c; ++k) {
      const int pv = E + k;
      // pivot row / pivot, then the rank-1 update of every other entry
      for (int e = tid; e < nmerge * ld; e += NTH) {
        const int m = e / ld, y = e % ld;
        double* A = out + m * slot;
        if (y != pv) A[pv * ld + y] /= A[pv * ld + pv];
      }
      __syncthreads();
      for (int e = tid; e < nmerge * ld * ld; e += NTH) {
        const int m = e / (ld * ld), rem = e % (ld * ld);
        const int x = rem / ld, y = rem % ld;
        if (x == pv || y == pv) continue;
        double* A = out + m * slot;
        const double f = A[x * ld + pv];
        if (f != 0.0) A[x * ld + y] -= f * A[pv * ld + y];
      }
      __syncthreads();
    }
    double* t = in;
    in = out;
    out = t;
    ld_in = ld;
    h = nh;
    w = nw;
    vert = !vert;
  }
  // the 16 x 16 block's matrix -> global (ld 64)
  double* dst = na.buf_out + la * na.out_stride + (int64_t)sb * 64 * 64;
  for (int e = tid; e < 64 * 64; e += NTH) {
    const int p = e / 64, q = e % 64;
    dst[e] = (p < ld_in && q < ld_in) ? in[p * ld_in + q] : 0.0;
  }
}

// ---------------------------------------------------------------------------
// Blocked elimination of the c cut nodes of one merge.
//   cut:  c rows (row stride ldc): c cut columns, then E external columns
//   ext:  E x E (row stride ld_e), the external block, updated in place into
//         the Schur complement.
// ---------------------------------------------------------------------------
__device__ void eliminate(double* cut, int c, int E, int ldc, double* ext, int ld_e,
                          double* lds) {
  const int tid = threadIdx.x;
  double* D = lds;              // KB x KB pivot block, then its Cholesky factor
  double* Zx = lds + KB * KB;   // KB x 64 panel slices for the rank-KB update
  double* Zy = Zx + KB * 64;
  for (int kb = 0; kb < c; kb += KB) {
    const int nk = min(KB, c - kb);
    for (int e = tid; e < KB * KB; e += NTH) {
      const int i = e / KB, j = e % KB;
      D[e] = (i < nk && j < nk) ? cut[(int64_t)(kb + i) * ldc + kb + j] : (i == j ? 1.0 : 0.0);
    }
    __syncthreads();
    // Cholesky of the pivot block (lower factor in place)
    for (int k = 0; k < KB; ++k) {
      if (tid == 0) D[k * KB + k] = sqrt(D[k * KB + k]);
      __syncthreads();
      if (tid > k && tid < KB) D[tid * KB + k] /= D[k * KB + k];
      __syncthreads();
      for (int e = tid; e < KB * KB; e += NTH) {
        const int i = e / KB, j = e % KB;
        if (i > k && j > k && j <= i) D[i * KB + j] -= D[i * KB + k] * D[j * KB + k];
      }
      __syncthreads();
    }
    // panel: rows kb .. kb + nk of the remaining columns <- L^-1 rows
    const int col0 = kb + nk;
    const int ncol = c + E - col0;
    for (int jc = tid; jc < ncol; jc += NTH) {
      double z[KB];
#pragma unroll
      for (int i = 0; i < KB; ++i) {
        double v = i < nk ? cut[(int64_t)(kb + i) * ldc + col0 + jc] : 0.0;
#pragma unroll
        for (int j = 0; j < i; ++j) v -= D[i * KB + j] * z[j];
        z[i] = v / D[i * KB + i];
      }
#pragma unroll
      for (int i = 0; i < KB; ++i)
        if (i < nk) cut[(int64_t)(kb + i) * ldc + col0 + jc] = z[i];
    }
    __syncthreads();
    // rank-nk update of the trailing part: virtual index v < nrem is cut row
    // col0 + v, v >= nrem is external v - nrem.
    const int nrem = c - col0;
    const int nv = nrem + E;
    for (int tx0 = 0; tx0 < nv; tx0 += 64) {
      for (int ty0 = 0; ty0 < nv; ty0 += 64) {
        if (tx0 >= nrem && ty0 + 64 <= nrem) continue;  // external rows x cut columns: mirror
        for (int e = tid; e < KB * 64; e += NTH) {
          const int k = e / 64, v = e % 64;
          double zx = 0.0, zy = 0.0;
          if (k < nk) {
            const int vx = tx0 + v, vy = ty0 + v;
            if (vx < nv) zx = cut[(int64_t)(kb + k) * ldc + (vx < nrem ? col0 + vx : c + vx - nrem)];
            if (vy < nv) zy = cut[(int64_t)(kb + k) * ldc + (vy < nrem ? col0 + vy : c + vy - nrem)];
          }
          Zx[k * 64 + v] = zx;
          Zy[k * 64 + v] = zy;
        }
        __syncthreads();
        const int rx = (tid / 16) * 4, ry = (tid % 16) * 4;
        double acc[4][4];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = 0.0;
        for (int k = 0; k < nk; ++k) {
          double xa[4], yb[4];
#pragma unroll
          for (int a = 0; a < 4; ++a) xa[a] = Zx[k * 64 + rx + a];
#pragma unroll
          for (int b = 0; b < 4; ++b) yb[b] = Zy[k * 64 + ry + b];
#pragma unroll
          for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) acc[a][b] = fma(xa[a], yb[b], acc[a][b]);
        }
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int vx = tx0 + rx + a;
          if (vx >= nv) continue;
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int vy = ty0 + ry + b;
            if (vy >= nv) continue;
            if (vx >= nrem && vy < nrem) continue;
            double* dst;
            if (vx < nrem) dst = cut + (int64_t)(col0 + vx) * ldc + (vy < nrem ? col0 + vy : c + vy - nrem);
            else dst = ext + (int64_t)(vx - nrem) * ld_e + (vy - nrem);
            *dst -= acc[a][b];
          }
        }
        __syncthreads();
      }
    }
  }
}

// One merge of two h x w blocks (children in buf_in, result to buf_out).
__global__ __launch_bounds__(NTH) void k_nd_merge(NdArgs na) {
  __shared__ double lds[KB * KB + 2 * KB * 64];
  const int tid = threadIdx.x;
  const int T = na.T, h = na.h, w = na.w;
  const bool vert = na.vert != 0;
  const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
  const int cols = T / nw, nmerge = (T / nh) * cols;
  const int64_t la = blockIdx.x / nmerge;
  const int m = (int)(blockIdx.x % nmerge);
  const int mi = m / cols, mj = m % cols;
  const int i0 = mi * nh, j0 = mj * nw;
  const int Emax = 2 * (nh + nw), c = vert ? w : h;
  const int Ein = 2 * (h + w);
  const int ccols = T / w;
  const int ldc = c + Emax;
  double* ext = na.buf_out + la * na.out_stride + (int64_t)m * Emax * Emax;
  double* cut = na.scratch + la * na.scr_stride + (int64_t)m * c * ldc;
  for (int e = tid; e < Emax * Emax; e += NTH) ext[e] = 0.0;
  for (int e = tid; e < c * ldc; e += NTH) cut[e] = 0.0;
  __syncthreads();
  for (int ch = 0; ch < 2; ++ch) {
    const int ci = (vert && ch) ? i0 + h : i0, cj = (!vert && ch) ? j0 + w : j0;
    const int np = nports(ci, cj, h, w, T);
    const int cm = vert ? (mi * 2 + ch) * ccols + mj : mi * ccols + mj * 2 + ch;
    const double* Yc = na.buf_in + la * na.in_stride + (int64_t)cm * Ein * Ein;
    for (int e = tid; e < np * np; e += NTH) {
      const int p = e / np, q = e % np;
      const double v = Yc[p * Ein + q];
      const int dp = merge_dest(ch, p, i0, j0, h, w, vert, T);
      const int dq = merge_dest(ch, q, i0, j0, h, w, vert, T);
      if (dp >= 0 && dq >= 0) ext[dp * Emax + dq] += v;
      else if (dp < 0) cut[(-1 - dp) * ldc + (dq < 0 ? (-1 - dq) : c + dq)] += v;
    }
    __syncthreads();
  }
  eliminate(cut, c, nports(i0, j0, nh, nw, T), ldc, ext, Emax, lds);
}

// Drivers and sinks: G'^T = -(Y_sL (Y_LL + g_d I)^-1 g_d E), written as fp32.
__global__ __launch_bounds__(NTH) void k_nd_final(NdArgs na) {
  __shared__ double lds[KB * KB + 2 * KB * 64];
  const int tid = threadIdx.x;
  const int T = na.T, M = na.ms.M, N = na.ms.N;
  const int64_t la = blockIdx.x;
  const int Ein = 4 * T;                 // ld of the last level's matrix (2 (T + T))
  const double* Y = na.buf_in + la * na.in_stride;
  const int E = M + T, c = T, ldc = c + E;
  double* ext = na.scratch + la * na.scr_stride;
  double* cut = ext + (int64_t)E * E;
  // ports of the whole grid: L (T) then B (T); externals: sources t (M), sinks s (T)
  for (int e = tid; e < E * E; e += NTH) {
    const int x = e / E, y = e % E;
    double v = 0.0;
    if (x < M && y < M) v = (x == y) ? na.g_d : 0.0;
    else if (x >= M && y >= M) v = Y[(T + x - M) * Ein + (T + y - M)];
    ext[e] = v;
  }
  for (int e = tid; e < c * ldc; e += NTH) {
    const int i = e / ldc, y = e % ldc;
    double v;
    if (y < c) v = Y[i * Ein + y] + (i == y ? na.g_d : 0.0);
    else if (y < c + M) v = (i == na.row_off + (y - c)) ? -na.g_d : 0.0;
    else v = Y[i * Ein + T + (y - c - M)];
    cut[e] = v;
  }
  __syncthreads();
  eliminate(cut, c, E, ldc, ext, E, lds);
  const int64_t arr = na.arr0 + la;
  float* out = na.gpt + arr * (int64_t)na.ms.Np * na.ms.Mp;
  for (int e = tid; e < na.ms.Np * na.ms.Mp; e += NTH) {
    const int j = e / na.ms.Mp, k = e % na.ms.Mp;
    out[e] = (j < N && k < M) ? (float)(-ext[(int64_t)(M + j) * E + k]) : 0.0f;
  }
}

}  // namespace

// Doubles of workspace one array needs (level buffers in, out, scratch).
void nd_sizes(int T, int M, int64_t* in_stride, int64_t* out_stride, int64_t* scr_stride) {
  int64_t lvl = (int64_t)(T / SB) * (T / SB) * 64 * 64;
  int64_t scr = 0;
  int h = SB, w = SB;
  bool vert = true;
  while (h < T || w < T) {
    const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
    const int64_t nmerge = (int64_t)(T / nh) * (T / nw);
    const int Emax = 2 * (nh + nw), c = vert ? w : h;
    lvl = lvl > nmerge * Emax * Emax ? lvl : nmerge * Emax * Emax;
    const int64_t s = nmerge * c * (int64_t)(c + Emax);
    scr = scr > s ? scr : s;
    h = nh;
    w = nw;
    vert = !vert;
  }
  const int64_t fin = (int64_t)(M + T) * (M + T) + (int64_t)T * (T + M + T);
  scr = scr > fin ? scr : fin;
  *in_stride = lvl;
  *out_stride = lvl;
  *scr_stride = scr;
}

int nd_side(int M, int N) {
  int T = SB;
  while (T < M || T < N) T *= 2;
  return T;
}

// Builds G' of arrays [arr0, arr0 + n) with the workspace ws (ping-pong
// level buffers and scratch, sized by nd_sizes for one array, times n).
hipError_t launch_nd_build(const MapScalars& ms, const float* W, float* gpt, int64_t arr0,
                           int64_t n, double* ws, hipStream_t s) {
  NdArgs na;
  na.ms = ms;
  na.W = W;
  na.gpt = gpt;
  na.arr0 = arr0;
  na.T = nd_side(ms.M, ms.N);
  na.row_off = na.T - ms.M;
  na.g_r = 1.0 / ms.r_row;
  na.g_c = 1.0 / ms.r_col;
  na.g_s = 1.0 / ms.r_sense;
  na.g_d = 1.0 / (ms.r_driver + ms.r_row);
  int64_t si, so, sc;
  nd_sizes(na.T, ms.M, &si, &so, &sc);
  double* bufA = ws;
  double* bufB = ws + n * si;
  na.scratch = ws + n * (si + so);
  na.in_stride = si;
  na.out_stride = so;
  na.scr_stride = sc;
  const int nsb = na.T / SB;
  na.buf_in = nullptr;
  na.buf_out = bufA;
  hipLaunchKernelGGL(k_nd_block16, dim3((unsigned)(n * nsb * nsb)), dim3(NTH), 0, s, na);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  double* cur = bufA;
  double* nxt = bufB;
  int h = SB, w = SB;
  bool vert = true;
  while (h < na.T || w < na.T) {
    const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
    const int64_t nmerge = (int64_t)(na.T / nh) * (na.T / nw);
    na.buf_in = cur;
    na.buf_out = nxt;
    na.h = h;
    na.w = w;
    na.vert = vert ? 1 : 0;
    hipLaunchKernelGGL(k_nd_merge, dim3((unsigned)(n * nmerge)), dim3(NTH), 0, s, na);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    double* t = cur;
    cur = nxt;
    nxt = t;
    h = nh;
    w = nw;
    vert = !vert;
  }
  na.buf_in = cur;
  hipLaunchKernelGGL(k_nd_final, dim3((unsigned)n), dim3(NTH), 0, s, na);
  return hipGetLastError();
}

}  // namespace rxnn
