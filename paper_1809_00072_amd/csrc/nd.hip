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
  int e_layout;          // largest external port count of a merge at this level
};

namespace {

constexpr int SBMIN = 8;        // smallest side of the blocks reduced in LDS
constexpr int NTH = 256;        // threads of the kernels on the blocked global path
constexpr int NTB = 1024;       // threads of the LDS-resident kernels (four waves per SIMD)
// doubles per LDS level buffer of a bs x bs block reduction
__host__ __device__ constexpr int lbuf(int bs) { return bs == 16 ? 6400 : 1600; }
constexpr int KB = 16;          // pivots per elimination block
constexpr int ULDS = 16384;     // doubles of cut rows a merge may keep in LDS

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

__device__ __forceinline__ int lg2ceil(int v) {
  int l = 0;
  while ((1 << l) < v) ++l;
  return l;
}

// 1 / a to within an ulp or two: hardware reciprocal and two Newton steps.
__device__ __forceinline__ double recip(double a) {
  double r = __builtin_amdgcn_rcp(a);
  r = fma(r, fma(-a, r, 1.0), r);
  r = fma(r, fma(-a, r, 1.0), r);
  return r;
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
// Levels 1 x 1 .. SB x SB of one SB x SB block, in LDS.
// ---------------------------------------------------------------------------
template <int SB, int NB>
__global__ __launch_bounds__(NB) void k_nd_block(NdArgs na) {
  __shared__ double bufA[lbuf(SB)];
  __shared__ double bufB[lbuf(SB)];
  __shared__ short tab[1024];
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
  if (tid < SB * SB) {
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
    const int cols = SB / nw;                    // merged blocks per row of the block
    const int nmerge = (SB / nh) * cols;
    const int ccols = SB / w;                    // child blocks per row
    const int npc = ld_in;                       // child slot side
    // destination of every child port in its merge's combined matrix
    for (int t = tid; t < nmerge * 2 * npc; t += NB) {
      const int m = t / (2 * npc), r2 = t - m * 2 * npc, ch = r2 >= npc ? 1 : 0;
      const int p = r2 - ch * npc;
      const int mi = m / cols, mj = m - mi * cols;
      const int i0 = I0 + mi * nh, j0 = J0 + mj * nw;
      const int np = nports((vert && ch) ? i0 + h : i0, (!vert && ch) ? j0 + w : j0, h, w, T);
      int d = -1;
      if (p < np) {
        d = merge_dest(ch, p, i0, j0, h, w, vert, T);
        d = d >= 0 ? d : E + (-1 - d);
      }
      tab[t] = (short)d;
    }
    for (int e = tid; e < nmerge * slot; e += NB) out[e] = 0.0;
    __syncthreads();
    // child entries: consecutive threads take consecutive columns q; task
    // spaces are padded to powers of two so that indices come from shifts
    const int lgq = lg2ceil(npc), lgc = lg2ceil(cols), lgcc = lg2ceil(ccols);
    for (int ch = 0; ch < 2; ++ch) {
      for (int t = tid; t < nmerge << (2 * lgq); t += NB) {
        const int q = t & ((1 << lgq) - 1), p = (t >> lgq) & ((1 << lgq) - 1);
        const int m = t >> (2 * lgq);
        if (p >= npc || q >= npc) continue;
        const short* dt = tab + (m * 2 + ch) * npc;
        const int dp = dt[p], dq = dt[q];
        if (dp < 0 || dq < 0) continue;
        const int mi = m >> lgc, mj = m & (cols - 1);
        const int cm = vert ? (((mi * 2 + ch) << lgcc) + mj) : ((mi << lgcc) + mj * 2 + ch);
        out[m * slot + dp * ld + dq] += in[cm * npc * npc + p * npc + q];
      }
      __syncthreads();
    }
    // eliminate the c shared nodes (pivot rows / columns E .. E + c - 1):
    // a task is one column y of one merge over a chunk of 8 rows
    const int lgy = lg2ceil(ld), lgx = lg2ceil((ld + 7) / 8);
    for (int k = 0; k < c; ++k) {
      const int pv = E + k;
      for (int t = tid; t < nmerge << (lgy + lgx); t += NB) {
        const int y = t & ((1 << lgy) - 1);
        const int x0 = ((t >> lgy) & ((1 << lgx) - 1)) * 8;
        const int m = t >> (lgy + lgx);
        if (y >= ld || y == pv || x0 >= ld) continue;
        double* A = out + m * slot;
        const double g = A[pv * ld + y] * recip(A[pv * ld + pv]);
        if (g == 0.0) continue;
        double axp[8], axy[8];
#pragma unroll
        for (int xx = 0; xx < 8; ++xx) {
          const int x = min(x0 + xx, ld - 1);
          axp[xx] = A[x * ld + pv];
          axy[xx] = A[x * ld + y];
        }
#pragma unroll
        for (int xx = 0; xx < 8; ++xx) {
          const int x = x0 + xx;
          if (x < ld && x != pv) A[x * ld + y] = axy[xx] - axp[xx] * g;
        }
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
  constexpr int EO = 4 * SB;   // ports of an interior SB x SB block
  double* dst = na.buf_out + la * na.out_stride + (int64_t)sb * EO * EO;
  for (int e = tid; e < EO * EO; e += NB) {
    const int p = e / EO, q = e % EO;
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

// Pivot-by-pivot elimination of the c cut rows U (row stride ldu, c cut
// columns then E external columns) held in LDS, followed by Z = D^-1/2 U_ext:
// afterwards the Schur complement of the externals is ext - Z^T Z.
// Pivot-by-pivot elimination of the c cut rows U (row stride ldu, c cut
// columns then E external columns) held in LDS, followed by Z = D^-1/2 U_ext:
// afterwards the Schur complement of the externals is ext - Z^T Z.  A task is
// one column over a chunk of 8 rows, its loads issued before its stores.
template <int NT>
__device__ void eliminate_lds(double* U, int c, int E, int ldu, double* isq) {
  const int tid = threadIdx.x;
  const int lgy = lg2ceil(c + E);
  for (int k = 0; k < c; ++k) {
    const double inv = recip(U[k * ldu + k]);
    const int nxc = (c - k - 1 + 7) / 8;
    for (int t = tid; t < nxc << lgy; t += NT) {
      const int y = t & ((1 << lgy) - 1);
      if (y <= k || y >= c + E) continue;
      const int x0 = k + 1 + (t >> lgy) * 8;
      const double uky = U[k * ldu + y] * inv;
      double uxk[8], uxy[8];
#pragma unroll
      for (int xx = 0; xx < 8; ++xx) {
        const int x = min(x0 + xx, c - 1);
        uxk[xx] = U[x * ldu + k];
        uxy[xx] = U[x * ldu + y];
      }
#pragma unroll
      for (int xx = 0; xx < 8; ++xx)
        if (x0 + xx < c) U[(x0 + xx) * ldu + y] = uxy[xx] - uxk[xx] * uky;
    }
    __syncthreads();
  }
  for (int t = tid; t < c; t += NT) isq[t] = 1.0 / sqrt(U[t * ldu + t]);
  __syncthreads();
  const int lge = lg2ceil(E);
  for (int t = tid; t < c << lge; t += NT) {
    const int k = t >> lge, y = t & ((1 << lge) - 1);
    if (y < E) U[k * ldu + c + y] *= isq[k];
  }
  __syncthreads();
}

// The same elimination in blocks of PB pivots: the pivot rows of a block are
// eliminated among themselves, every later row then gets its PB multipliers
// from its own entries in the block's columns, and one pass applies the
// rank-PB update to the trailing rows.  The trailing matrix is read and
// written once per block instead of once per pivot (the rank-1 form is bound
// by that LDS traffic).  aux: LDS scratch of 4 (c + 1) doubles.
template <int NT>
__device__ void eliminate_lds_blocked(double* U, int c, int E, int ldu, double* isq,
                                      double* aux) {
  constexpr int PB = 4;
  const int tid = threadIdx.x;
  const int ncol = c + E;
  const int lgy = lg2ceil(ncol);
  double* lm = aux;               // multipliers, PB per row
  double* inv = aux + PB * c;     // pivot reciprocals of the block
  for (int k0 = 0; k0 < c; k0 += PB) {
    const int kb = min(PB, c - k0);
    // pivot rows of the block, among themselves
    for (int i = 0; i < kb; ++i) {
      const int k = k0 + i;
      const double ik = recip(U[k * ldu + k]);
      if (tid == 0) inv[i] = ik;
      const int nr = kb - 1 - i;   // later rows of the block
      for (int t = tid; t < nr << lgy; t += NT) {
        const int y = t & ((1 << lgy) - 1);
        if (y <= k || y >= ncol) continue;
        const int x = k + 1 + (t >> lgy);
        U[x * ldu + y] -= U[x * ldu + k] * ik * U[k * ldu + y];
      }
      __syncthreads();
    }
    const int r0 = k0 + kb;
    // multipliers of the trailing rows
    for (int x = r0 + tid; x < c; x += NT) {
      double l[PB];
#pragma unroll
      for (int i = 0; i < PB; ++i) {
        if (i >= kb) break;
        double t = U[x * ldu + k0 + i];
        for (int j = 0; j < i; ++j) t -= l[j] * U[(k0 + j) * ldu + k0 + i];
        l[i] = t * inv[i];
        lm[x * PB + i] = l[i];
      }
    }
    __syncthreads();
    // rank-kb update of the trailing rows, 8-row chunks per task
    const int nxc = (c - r0 + 7) / 8;
    for (int t = tid; t < nxc << lgy; t += NT) {
      const int y = t & ((1 << lgy) - 1);
      if (y < r0 || y >= ncol) continue;
      const int x0 = r0 + (t >> lgy) * 8;
      double p[PB];
#pragma unroll
      for (int i = 0; i < PB; ++i) p[i] = i < kb ? U[(k0 + i) * ldu + y] : 0.0;
      double u[8];
#pragma unroll
      for (int xx = 0; xx < 8; ++xx) u[xx] = U[min(x0 + xx, c - 1) * ldu + y];
#pragma unroll
      for (int xx = 0; xx < 8; ++xx) {
        const int x = x0 + xx;
        if (x >= c) continue;
        double v = u[xx];
#pragma unroll
        for (int i = 0; i < PB; ++i)
          if (i < kb) v -= lm[x * PB + i] * p[i];
        U[x * ldu + y] = v;
      }
    }
    __syncthreads();
  }
  for (int t = tid; t < c; t += NT) isq[t] = 1.0 / sqrt(U[t * ldu + t]);
  __syncthreads();
  const int lge = lg2ceil(E);
  for (int t = tid; t < c << lge; t += NT) {
    const int k = t >> lge, y = t & ((1 << lge) - 1);
    if (y < E) U[k * ldu + c + y] *= isq[k];
  }
  __syncthreads();
}

// One merge of two h x w blocks (children in buf_in, result to buf_out).
template <bool LDSP, int NT>
__global__ __launch_bounds__(NT) void k_nd_merge(NdArgs na) {
  extern __shared__ double lds[];   // cut rows (LDS path) or the blocked path's panels
  __shared__ short tab[2 * 1024];   // children of a 256 x 256 grid have up to 768 ports
  __shared__ double isq[256];
  __shared__ double aux[4 * 257];
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
  const int E = nports(i0, j0, nh, nw, T);
  const int Ein = 2 * (h + w);
  const int ccols = T / w;
  double* ext = na.buf_out + la * na.out_stride + (int64_t)m * Emax * Emax;
  const int ldc = LDSP ? c + na.e_layout : c + Emax;
  double* cut = LDSP ? lds : na.scratch + la * na.scr_stride + (int64_t)m * c * ldc;
  for (int t = tid; t < 2 * Ein; t += NT) {
    const int ch = t / Ein, p = t - ch * Ein;
    const int ci = (vert && ch) ? i0 + h : i0, cj = (!vert && ch) ? j0 + w : j0;
    tab[t] = (short)(p < nports(ci, cj, h, w, T) ? merge_dest(ch, p, i0, j0, h, w, vert, T)
                                                 : -1000);
  }
  {
    const int lge = lg2ceil(E);
    for (int e = tid; e < E << lge; e += NT) {
      const int y = e & ((1 << lge) - 1);
      if (y < E) ext[(e >> lge) * Emax + y] = 0.0;
    }
  }
  for (int e = tid; e < c * ldc; e += NT) cut[e] = 0.0;
  __syncthreads();
  for (int ch = 0; ch < 2; ++ch) {
    const int cm = vert ? (mi * 2 + ch) * ccols + mj : mi * ccols + mj * 2 + ch;
    const double* Yc = na.buf_in + la * na.in_stride + (int64_t)cm * Ein * Ein;
    const short* dt = tab + ch * Ein;
    const int lgi = lg2ceil(Ein);
    for (int t0 = tid; t0 < Ein << lgi; t0 += 8 * NT) {
      double v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = min(t0 + u * NT, (Ein << lgi) - 1);
        const int p = t >> lgi, q = min(t & ((1 << lgi) - 1), Ein - 1);
        v[u] = Yc[p * Ein + q];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = t0 + u * NT;
        if (t >= Ein << lgi) continue;
        const int p = t >> lgi, q = t & ((1 << lgi) - 1);
        if (q >= Ein) continue;
        const int dp = dt[p], dq = dt[q];
        if (dp == -1000 || dq == -1000) continue;
        if (dp >= 0) {
          if (dq >= 0) ext[dp * Emax + dq] = v[u];
        } else {
          cut[(-1 - dp) * ldc + (dq < 0 ? (-1 - dq) : c + dq)] += v[u];
        }
      }
    }
    __syncthreads();
  }
  if (!LDSP) {
    eliminate(cut, c, E, ldc, ext, Emax, lds);
    return;
  }
  eliminate_lds_blocked<NT>(cut, c, E, ldc, isq, aux);
  // ext -= Z^T Z, square tiles of TS x TS entries, 4 x 4 per thread
  constexpr int TS = NT == 1024 ? 128 : 64;
  const int rx = (tid / (TS / 4)) * 4, ry = (tid % (TS / 4)) * 4;
  for (int tx0 = 0; tx0 < E; tx0 += TS)
    for (int ty0 = 0; ty0 < E; ty0 += TS) {
      double acc[4][4];
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = 0.0;
      for (int k = 0; k < c; ++k) {
        const double* z = cut + k * ldc + c;
        double xa[4], yb[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) xa[a] = z[min(tx0 + rx + a, E - 1)];
#pragma unroll
        for (int b = 0; b < 4; ++b) yb[b] = z[min(ty0 + ry + b, E - 1)];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = fma(xa[a], yb[b], acc[a][b]);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int x = tx0 + rx + a;
        if (x >= E) continue;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int y = ty0 + ry + b;
          if (y < E) ext[x * Emax + y] -= acc[a][b];
        }
      }
    }
}

// Drivers and sinks: G'^T = -(Y_sL (Y_LL + g_d I)^-1 g_d E), written as fp32.
// Externals: the M source terminals t, then the T sink terminals s; cut: the
// T row-input nodes.  Only the (s, t) block of the result is needed.
template <bool LDSP>
__global__ __launch_bounds__(LDSP ? NTB : NTH) void k_nd_final(NdArgs na) {
  constexpr int NT = LDSP ? NTB : NTH;
  extern __shared__ double lds[];
  __shared__ double isq[256];
  __shared__ double aux[4 * 257];
  const int tid = threadIdx.x;
  const int T = na.T, M = na.ms.M, N = na.ms.N;
  const int64_t la = blockIdx.x;
  const int Ein = 4 * T;                 // ld of the last level's matrix (2 (T + T))
  const double* Y = na.buf_in + la * na.in_stride;
  const int E = M + T, c = T, ldc = c + E;
  double* ext = na.scratch + la * na.scr_stride;
  double* cut = LDSP ? lds : ext + (int64_t)E * E;
  if (!LDSP) {
    for (int e = tid; e < E * E; e += NT) {
      const int x = e / E, y = e % E;
      double v = 0.0;
      if (x < M && y < M) v = (x == y) ? na.g_d : 0.0;
      else if (x >= M && y >= M) v = Y[(T + x - M) * Ein + (T + y - M)];
      ext[e] = v;
    }
  }
  const int lgl = lg2ceil(ldc);
  for (int e = tid; e < c << lgl; e += NT) {
    const int i = e >> lgl, y = e & ((1 << lgl) - 1);
    if (y >= ldc) continue;
    double v;
    if (y < c) v = Y[i * Ein + y] + (i == y ? na.g_d : 0.0);
    else if (y < c + M) v = (i == na.row_off + (y - c)) ? -na.g_d : 0.0;
    else v = Y[i * Ein + T + (y - c - M)];
    cut[i * ldc + y] = v;
  }
  __syncthreads();
  const int64_t arr = na.arr0 + la;
  float* out = na.gpt + arr * (int64_t)na.ms.Np * na.ms.Mp;
  if (!LDSP) {
    eliminate(cut, c, E, ldc, ext, E, lds);
    for (int e = tid; e < na.ms.Np * na.ms.Mp; e += NT) {
      const int j = e / na.ms.Mp, k = e % na.ms.Mp;
      out[e] = (j < N && k < M) ? (float)(-ext[(int64_t)(M + j) * E + k]) : 0.0f;
    }
    return;
  }
  eliminate_lds_blocked<NT>(cut, c, E, ldc, isq, aux);
  const int lgm = lg2ceil(na.ms.Mp);
  for (int e = tid; e < na.ms.Np << lgm; e += NT) {
    const int j = e >> lgm, k = e & ((1 << lgm) - 1);
    if (k >= na.ms.Mp) continue;
    double v = 0.0;
    if (j < N && k < M)
      for (int l = 0; l < c; ++l) v = fma(cut[l * ldc + c + M + j], cut[l * ldc + c + k], v);
    out[j * na.ms.Mp + k] = (float)v;
  }
}

}  // namespace

// Side of the blocks reduced in LDS: 8 x 8 blocks give more, smaller
// workgroups (several per CU) when the arrays of a chunk alone would not fill
// the device; 16 x 16 blocks need fewer merge passes.
int nd_block_side(int T, int64_t n_arrays) {
  return (n_arrays * (T / 16) * (T / 16) < 1024) ? 8 : 16;
}

// Doubles of workspace one array needs (level buffers in, out, scratch).
void nd_sizes(int T, int M, int bs, int64_t* in_stride, int64_t* out_stride,
              int64_t* scr_stride) {
  int64_t lvl = (int64_t)(T / bs) * (T / bs) * (4 * bs) * (4 * bs);
  int64_t scr = 0;
  int h = bs, w = bs;
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
  int T = 16;
  while (T < M || T < N) T *= 2;
  return T;
}

static bool g_nd_attr = false;

// Builds G' of arrays [arr0, arr0 + n) with the workspace ws (ping-pong
// level buffers and scratch, sized by nd_sizes for one array, times n).
hipError_t launch_nd_build(const MapScalars& ms, const float* W, float* gpt, int64_t arr0,
                           int64_t n, int bs, double* ws, hipStream_t s) {
  if (!g_nd_attr) {
    const int mx = ULDS * (int)sizeof(double);
    hipError_t e0 = hipFuncSetAttribute((const void*)k_nd_merge<true, NTB>,
                                        hipFuncAttributeMaxDynamicSharedMemorySize, mx);
    if (e0 == hipSuccess)
      e0 = hipFuncSetAttribute((const void*)k_nd_merge<true, NTH>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, mx);
    if (e0 == hipSuccess)
      e0 = hipFuncSetAttribute((const void*)k_nd_final<true>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, mx);
    if (e0 != hipSuccess) return e0;
    g_nd_attr = true;
  }
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
  nd_sizes(na.T, ms.M, bs, &si, &so, &sc);
  double* bufA = ws;
  double* bufB = ws + n * si;
  na.scratch = ws + n * (si + so);
  na.in_stride = si;
  na.out_stride = so;
  na.scr_stride = sc;
  const int nsb = na.T / bs;
  na.buf_in = nullptr;
  na.buf_out = bufA;
  {
    ProfScope prof("nd_block", s);
    const dim3 grid((unsigned)(n * nsb * nsb));
    if (bs == 8)
      hipLaunchKernelGGL((k_nd_block<8, NTH>), grid, dim3(NTH), 0, s, na);
    else
      hipLaunchKernelGGL((k_nd_block<16, NTB>), grid, dim3(NTB), 0, s, na);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  double* cur = bufA;
  double* nxt = bufB;
  int h = bs, w = bs;
  bool vert = true;
  while (h < na.T || w < na.T) {
    const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
    const int64_t nmerge = (int64_t)(na.T / nh) * (na.T / nw);
    na.buf_in = cur;
    na.buf_out = nxt;
    na.h = h;
    na.w = w;
    na.vert = vert ? 1 : 0;
    int e_layout = 0;
    for (int bi = 0; bi < na.T / nh; ++bi)
      for (int bj = 0; bj < na.T / nw; ++bj) {
        const int e_b = nh + ((bj + 1) * nw < na.T ? nh : 0) + (bi > 0 ? nw : 0) + nw;
        e_layout = e_layout > e_b ? e_layout : e_b;
      }
    na.e_layout = e_layout;
    const int c = vert ? w : h;
    const int64_t u = (int64_t)c * (c + e_layout);
    const dim3 grid((unsigned)(n * nmerge));
    {
      ProfScope prof("nd_merge", s);
      if (u <= ULDS && c <= 16)
        hipLaunchKernelGGL((k_nd_merge<true, NTH>), grid, dim3(NTH),
                           (unsigned)(u * sizeof(double)), s, na);
      else if (u <= ULDS)
        hipLaunchKernelGGL((k_nd_merge<true, NTB>), grid, dim3(NTB),
                           (unsigned)(u * sizeof(double)), s, na);
      else
        hipLaunchKernelGGL((k_nd_merge<false, NTH>), grid, dim3(NTH),
                           (unsigned)((KB * KB + 2 * KB * 64) * sizeof(double)), s, na);
    }
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
  {
    ProfScope prof("nd_final", s);
    const int64_t uf = (int64_t)na.T * (na.T + ms.M + na.T);
    if (uf <= ULDS)
      hipLaunchKernelGGL(k_nd_final<true>, dim3((unsigned)n), dim3(NTB),
                         (unsigned)(uf * sizeof(double)), s, na);
    else
      hipLaunchKernelGGL(k_nd_final<false>, dim3((unsigned)n), dim3(NTH),
                         (unsigned)((KB * KB + 2 * KB * 64) * sizeof(double)), s, na);
  }
  return hipGetLastError();
}

}  // namespace rxnn
