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
// Levels up to 16 x 16 cells: one workgroup per 16 x 16 region (k_nd_block):
// each wave builds an 8 x 8 block (its 2 x 2 blocks in registers, each larger
// merge by the whole wave: the cut rows eliminated by lane reads, the Schur
// update on fp64 MFMA tiles), then the workgroup merges the four into the
// region's block.  Merges with 8 to 64 shared nodes: one workgroup per
// merge eliminates them with the shared rows in registers (k_nd_cut; each
// lane reads one multiplier per 16 rows from LDS, the FMAs take them by DPP
// row broadcast), and the Schur update of the external block runs on 64 x 64
// fp64 MFMA tiles of its lower triangle, in the same workgroup for small
// merges, else in k_nd_schur; the final step with at most 64 row inputs
// likewise.  Merges with 128 shared nodes: k_nd_cut2 (panels of 256 external
// columns), then k_nd_schur.  The merge of the two halves of a large grid
// and its final step: the combined matrix is built dense (k_nd_dense0) and
// eliminated in stages of 64 pivots (k_nd_cut<64, 2>, k_nd_dschur).  Other
// sizes run on one workgroup with the shared rows in global memory,
// eliminated in blocks of 16 (Cholesky of the 16 x 16 pivot block,
// triangular solve of its rows, rank-16 update of the rest).  All
// arithmetic is fp64; wire conductances exceed device conductances by about
// four orders of magnitude, and the elimination of series wires loses about
// that many digits, leaving G' accurate to ~1e-12.  Every wire, driver and
// sense resistance must be positive (zero resistances take the row sweep
// instead).

#include <algorithm>
#include <utility>

#include "common.h"
#include "device_map.h"

namespace rxnn {

struct NdArgs {
  MapScalars ms;
  const float* W;
  float* gpt;
  int64_t arr0;          // first array of this chunk
  int64_t n_arrays;      // arrays in this chunk
  int T, row_off;        // grid side, first grid row of the tile (T - M)
  double g_r, g_c, g_s, g_d;
  double* buf_in;        // level buffers and scratch (per array strides below)
  double* buf_out;
  double* scratch;
  int64_t in_stride, out_stride, scr_stride;  // doubles per array
  int h, w, vert;        // children size and merge direction (merge kernel)
  int e_layout;          // largest external port count of a merge at this level
  // staged elimination of a dense combined matrix (more than 128 cut nodes)
  const double* dA;      // stage input, dn x dn (row stride dld) per array (stride in_stride)
  double* dB;            // stage output (row stride dldo) per array
  int dn, dld, dldo;
  int dpanel;            // external columns per workgroup of the cut kernel
  int npan;              // workgroups (column panels of dpanel) per merge of the
                         // cut kernel's merge mode (0 or 1: one, all columns)
  int dead[4];           // staged path: index ranges [dead[0], dead[1]) and
                         // [dead[2], dead[3]) of the combined matrix whose
                         // mutual entries nothing reads (sinks x sinks,
                         // sources x sources): neither written nor updated
  int fuse;              // k_nd_cut finishes the Schur update itself (its kFuse
                         // path; the host's schur_fused decides)
  // several layers at once (null tables: the one layer of ms / W / gpt)
  NdBatch batch;
};

namespace {

constexpr int NTH = 256;        // threads of the kernels on the blocked global path
constexpr int KB = 16;          // pivots per elimination block

__host__ __device__ constexpr void ports(int i0, int j0, int h, int w, int T, int& nL, int& nR,
                                      int& nT, int& nB) {
  nL = h;
  nR = (j0 + w < T) ? h : 0;
  nT = (i0 > 0) ? w : 0;
  nB = w;
}

// Where port p of child `ch` (0: top/left, 1: bottom/right) of a merge of two
// h x w blocks at (i0, j0) goes: >= 0 an external port of the merged block,
// < 0 the shared (cut) node -1 - k.
__host__ __device__ constexpr int merge_dest(int ch, int p, int i0, int j0, int h, int w, bool vert,
                                          int T) {
  const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
  const bool Rn = j0 + nw < T, Tn = i0 > 0;
  const int oR = nh, oT = nh + (Rn ? nh : 0), oB = oT + (Tn ? nw : 0);
  const int ci = (vert && ch) ? i0 + h : i0, cj = (!vert && ch) ? j0 + w : j0;
  const bool Rc = cj + w < T, Tc = ci > 0;
  int seg = 0, idx = p;  // 0 L, 1 R, 2 T, 3 B
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

// 1 / sqrt(a) for a > 0: the hardware estimate and two Newton steps
// (r <- r + r (1 - a r^2) / 2), each squaring the relative error: from any
// estimate good to 14 bits or more that reaches fp64 accuracy; nine
// instructions instead of a correctly rounded square root and division.
__device__ __forceinline__ double rsqrt_nr(double a) {
  double r = __builtin_amdgcn_rsq(a);
#pragma unroll
  for (int i = 0; i < 2; ++i) r = fma(0.5 * r, fma(-a * r, r, 1.0), r);
  return r;
}

// A level's merged blocks are symmetric, and the Schur kernels store only
// their 64 x 64 tiles on and below the diagonal: entry (r, c) of a block
// with row stride ld is read from its mirror when it lies in a tile above.
__host__ __device__ __forceinline__ int sym_at(int r, int c, int ld) {
  return (r >> 6) >= (c >> 6) ? r * ld + c : c * ld + r;
}

__host__ __device__ constexpr int nports(int i0, int j0, int h, int w, int T) {
  int a = 0, b = 0, c = 0, d = 0;
  ports(i0, j0, h, w, T, a, b, c, d);
  return a + b + c + d;
}

// W -> G of the device at grid cell (gi, gj) of array `arr` (0 outside the tile).
__device__ __forceinline__ double cell_conductance(const MapScalars& ms, const float* W,
                                                   double wmax, int64_t arr, int gi, int gj,
                                                   int row_off) {
  const int i = gi - row_off, j = gj;
  if (i < 0 || j >= ms.N) return 0.0;
  return device_g(ms, W, wmax, arr, i, j);
}

// Array `la` of the launch: its layer's scalars and weights, its index in
// that layer, and where its G' goes.  Every layer of a batch shares M, N (so
// Mp, Np) with na.ms.
struct ArrRef {
  const MapScalars* ms;
  const float* W;
  int64_t arr;
  float* out;
};

__device__ __forceinline__ ArrRef nd_ref(const NdArgs& na, int64_t la) {
  const int64_t tile = (int64_t)na.ms.Np * na.ms.Mp;
  if (na.batch.ent) {
    const int2 e = na.batch.ent[na.arr0 + la];
    const NdBatchLayer* bl = na.batch.layers + e.x;
    return ArrRef{&bl->ms, bl->W, (int64_t)e.y, bl->gpt + (int64_t)e.y * tile};
  }
  const int64_t arr = na.arr0 + la;
  return ArrRef{&na.ms, na.W, arr, na.gpt + arr * tile};
}

// ---------------------------------------------------------------------------
// Levels 1 x 1 .. 16 x 16: one workgroup per 16 x 16 region, wave w building
// the 8 x 8 block (w / 2, w % 2) of it in its own LDS buffers (no workgroup
// barrier), then the workgroup merging the four.
// ---------------------------------------------------------------------------
constexpr int BS = 8;                 // side of the blocks one wave builds
constexpr int BWAVES = 4;             // waves per workgroup of the block kernel
constexpr int BLEVELS = 7;  // 1x1 -> 2x1 -> 2x2 -> 4x2 -> 4x4 -> 8x4 -> 8x8 -> 16x8
// In LDS every merged block's matrix takes its side squared plus one double:
// consecutive matrices then start in different banks.
__host__ __device__ constexpr int lds_mat(int side) { return side * side + 1; }
// doubles per wave: the odd levels' results (16 x 65 for the 2 x 2 blocks,
// 4 x 257, then the 8 x 8 block) and the even levels' (8 x 145, 2 x 577)
constexpr int BUFA = 16 * 65, BUFB = 8 * 145;

// Child port landing on each combined slot (cut nodes 0 .. c-1, then the
// externals), per level and per boundary variant (bit 1: the merged block
// has ports on its right, bit 0: on its top) - the only geometry on which
// the port maps of a merge depend.
struct alignas(16) BlkTab {
  short s[BLEVELS][4][2][64];
};

constexpr BlkTab make_blk_tab() {
  BlkTab t{};
  for (int l = 0; l < BLEVELS; ++l)
    for (int v = 0; v < 4; ++v)
      for (int ch = 0; ch < 2; ++ch)
        for (int k = 0; k < 64; ++k) t.s[l][v][ch][k] = -1;
  const int hs[BLEVELS] = {1, 2, 2, 4, 4, 8, 8}, ws[BLEVELS] = {1, 1, 2, 2, 4, 4, 8};
  const int Tr = 1024;   // any grid larger than the merged block
  for (int l = 0; l < BLEVELS; ++l) {
    const bool vert = (l % 2) == 0;
    const int h = hs[l], w = ws[l];
    const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
    const int c = vert ? w : h;
    for (int v = 0; v < 4; ++v) {
      const int i0 = (v & 1) ? nh : 0, j0 = (v & 2) ? 0 : Tr - nw;
      for (int ch = 0; ch < 2; ++ch) {
        const int ci = (vert && ch) ? i0 + h : i0, cj = (!vert && ch) ? j0 + w : j0;
        const int np = nports(ci, cj, h, w, Tr);
        for (int p = 0; p < np; ++p) {
          const int d = merge_dest(ch, p, i0, j0, h, w, vert, Tr);
          t.s[l][v][ch][d >= 0 ? c + d : -1 - d] = (short)p;
        }
      }
    }
  }
  return t;
}

__constant__ BlkTab kBlkTab = make_blk_tab();

typedef __attribute__((address_space(3))) double lds_f64;
typedef __attribute__((address_space(3))) short lds_i16;

// An LDS pointer the compiler cannot see through: element reads at fixed
// indices then use the instruction's offset field instead of a register
// holding each address.
template <typename P>
__device__ __forceinline__ P* opaque_lds(const void* p) {
  unsigned a = (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
  asm volatile("" : "+v"(a));
  return (P*)(uintptr_t)a;
}

__device__ __forceinline__ double readlane_d(double v, int l) {
  const unsigned long long b = __builtin_bit_cast(unsigned long long, v);
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)b, l);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(b >> 32), l);
  return __builtin_bit_cast(double, ((unsigned long long)hi << 32) | lo);
}

// LDS written by some lanes of a wave, then read by others of the same wave.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Lane k of every row of 16 lanes, to the whole row (DPP row broadcast).
template <int K>
__device__ __forceinline__ double rowbcast_d(double v) {
  // every source lane of a row broadcast exists: bound_ctrl only spares the
  // move that would set the unused old value
  return __builtin_amdgcn_update_dpp(0.0, v, 0x150 + K, 0xf, 0xf, true);
}

__device__ __forceinline__ double rowbcast_d(double v, int k) {
  switch (k & 15) {
    case 0: return rowbcast_d<0>(v);
    case 1: return rowbcast_d<1>(v);
    case 2: return rowbcast_d<2>(v);
    case 3: return rowbcast_d<3>(v);
    case 4: return rowbcast_d<4>(v);
    case 5: return rowbcast_d<5>(v);
    case 6: return rowbcast_d<6>(v);
    case 7: return rowbcast_d<7>(v);
    case 8: return rowbcast_d<8>(v);
    case 9: return rowbcast_d<9>(v);
    case 10: return rowbcast_d<10>(v);
    case 11: return rowbcast_d<11>(v);
    case 12: return rowbcast_d<12>(v);
    case 13: return rowbcast_d<13>(v);
    case 14: return rowbcast_d<14>(v);
    default: return rowbcast_d<15>(v);
  }
}

// The region kernel's LDS matrices (row stride ein, lds_mat(ein) apart)
// hold a zero in the slot after their last entry, index ein * ein.  A
// column's key: its port, or a large negative number when the port is
// absent (computed once per column).
__device__ __forceinline__ int col_key(int s) { return s < 0 ? -(1 << 20) : s; }
// Entry (r, column key sk) of such a matrix: an absent row port (r < 0) or
// column port makes the index negative, and the unsigned minimum turns it
// into the zero slot, so neither case needs a select of the value.
__device__ __forceinline__ double pick(const double* c, int r, int sk, int ein) {
  return c[min((unsigned)(r * ein + sk), (unsigned)(ein * ein))];
}

// The eight 2 x 2 -> 4 x 2 merges of a wave's 8 x 8 block (children
// lds_mat(8) apart in `in`, results lds_mat(12) apart in `out`), in two
// passes of four, a group of 16 lanes per merge: lane y holds column y of
// its merge's combined matrix [2 cut nodes | 12 external ports], every row
// in registers, and the multiplier of row x at pivot k (lane k's register x,
// the matrix being symmetric) comes by a DPP row broadcast; eliminating the
// cut rows leaves the merged block in the external rows.
__device__ __forceinline__ void level2_dpp(int T, int I0, int J0, const short* tab,
                                           const double* in, double* out, int lane) {
  constexpr int L = 2, NH = 4, NW = 2, C = 2, EM = 12, EIN = 8, LD = C + EM, GS = 16;
  const int g = lane / GS, yl = lane % GS;
#pragma unroll 1
  for (int pass = 0; pass < 2; ++pass) {
    const int m = pass * (64 / GS) + g;
    const int mi = m >> 2, mj = m & 3;
    const int i0 = I0 + mi * NH, j0 = J0 + mj * NW;
    const bool rn = j0 + NW < T, tn = i0 > 0;
    const int ld = C + NH + (rn ? NH : 0) + (tn ? NW : 0) + NW;
    const int cm0 = mi * 8 + mj, cm1 = cm0 + 4;
    const short* t0 = tab + (((L * 4) + (rn ? 2 : 0) + (tn ? 1 : 0)) * 2) * 64;
    const short* t1 = t0 + 64;
    const double* c0 = in + cm0 * lds_mat(EIN);
    const double* c1 = in + cm1 * lds_mat(EIN);
    const int k0 = col_key(t0[yl]), k1 = col_key(t1[yl]);
    double U[LD];
#pragma unroll
    for (int x = 0; x < LD; ++x) U[x] = pick(c0, t0[x], k0, EIN) + pick(c1, t1[x], k1, EIN);
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const double t = U[k] * recip(rowbcast_d(U[k], k));
#pragma unroll
      for (int x = k + 1; x < LD; ++x) U[x] = fma(-rowbcast_d(U[x], k), t, U[x]);
    }
    if (yl >= C && yl < ld) {
#pragma unroll
      for (int x = C; x < LD; ++x)
        if (x < ld) out[m * lds_mat(EM) + (x - C) * EM + (yl - C)] = U[x];
    }
    if (yl == 0) out[m * lds_mat(EM) + EM * EM] = 0.0;   // the zero slot
  }
  wave_sync();
}

// Conductance g between nodes p and q of a small symmetric matrix held in
// registers (lower triangle used).
template <int N>
__device__ __forceinline__ void stamp(double (&X)[N][N], int p, int q, double g) {
  X[p][p] += g;
  X[q][q] += g;
  if (p > q) X[p][q] -= g;
  else X[q][p] -= g;
}

// Eliminates nodes 0 .. NC - 1 of the symmetric N x N matrix X (lower
// triangle): X[i][j] -= X[i][k] X[j][k] / X[k][k] for i >= j > k.
template <int N, int NC>
__device__ __forceinline__ void eliminate_lead(double (&X)[N][N]) {
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const double r = recip(X[k][k]);
#pragma unroll
    for (int i = k + 1; i < N; ++i) {
      const double f = X[i][k] * r;
#pragma unroll
      for (int j = k + 1; j <= i; ++j) X[i][j] = fma(-f, X[j][k], X[i][j]);
    }
  }
}

// Levels 1 x 1 and 2 x 1 -> 2 x 2 of the 2 x 2 block whose top-left cell is
// (gi0, gj0), in one lane's registers: each cell's ports in the padded order
// [L | R | T | B] (an absent R or T port is a zero row: no row-wire edge at
// the right edge of the grid; at the top the cell's b-node is eliminated in
// series), the cells of each column merged (their shared b-node eliminated),
// then the two 2 x 1 halves (their two shared a-nodes); Gc[r][c] is the
// conductance of cell (gi0 + r, gj0 + c).  Returns the 8 x 8 matrix over
// [L0 L1 | R0 R1 | T0 T1 | B0 B1] in rows 2 .. 9 of X.
__device__ __forceinline__ void block2x2(const double (&Gc)[2][2], int gi0, int gj0, int T,
                                         double g_r, double g_c, double g_s, double (&X)[10][10]) {
#pragma unroll
  for (int i = 0; i < 10; ++i)
#pragma unroll
    for (int j = 0; j <= i; ++j) X[i][j] = 0.0;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    // the column's two cells over [s | L0 L1 | R0 R1 | T | B], s the b-node
    // between them
    double Y[7][7];
#pragma unroll
    for (int i = 0; i < 7; ++i)
#pragma unroll
      for (int j = 0; j <= i; ++j) Y[i][j] = 0.0;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int gi = gi0 + r, gj = gj0 + c;
      const double G = Gc[r][c];
      const bool hasT = gi > 0;
      const double gv = (gi + 1 < T) ? g_c : g_s;
      const int iL = 1 + r, iR = 3 + r, iT = r == 0 ? 5 : 0, iB = r == 0 ? 0 : 6;
      stamp(Y, iL, iR, gj + 1 < T ? g_r : 0.0);
      stamp(Y, iL, iT, hasT ? G : 0.0);
      stamp(Y, iT, iB, hasT ? gv : 0.0);
      stamp(Y, iL, iB, (!hasT && G > 0.0) ? (G * gv) / (G + gv) : 0.0);
    }
    eliminate_lead<7, 1>(Y);
    // the half's ports [L0 L1 R0 R1 T B] in the 2 x 2 merge's order
    // [s0 s1 | L0 L1 | R0 R1 | T0 T1 | B0 B1] (s: the shared a-nodes)
    constexpr int kMap[2][6] = {{2, 3, 0, 1, 6, 8}, {0, 1, 4, 5, 7, 9}};
#pragma unroll
    for (int p = 0; p < 6; ++p)
#pragma unroll
      for (int q = 0; q <= p; ++q) {
        const int a = kMap[c][p], b = kMap[c][q];
        if (a >= b) X[a][b] += Y[1 + p][1 + q];
        else X[b][a] += Y[1 + p][1 + q];
      }
  }
  eliminate_lead<10, 2>(X);
}

__device__ void region_merge16(int T, int RI, int RJ, const double* ch, double* dst,
                               double* scr);
template <int L, int H, int W, bool VERT, int NB, bool SPLIT = false>
__device__ __forceinline__ void merge_mfma(int T, int i0, int j0, const short* tab,
                                           const double* c0, const double* c1, double* out,
                                           int lane, int part = 0);

// One 16 x 16 region per workgroup (every build, whatever its size, so that
// an array's arithmetic never depends on how many arrays are built with it):
// wave w builds its 8 x 8 block (row w / 2, column w % 2 of the region)
// alone, without workgroup barriers, in its LDS buffers A and B: the 2 x 2
// blocks in registers, the merges 2 x 2 -> 4 x 2 in 16-lane groups
// (level2_dpp), then 4 x 2 -> 4 x 4 -> 8 x 4 -> 8 x 8, each by the whole
// wave (merge_mfma).  Waves m and 2 + m then merge
// column m's pair into a 16 x 8 block (in LDS), and the workgroup merges
// those into the region's 16 x 16 block, which goes to the level buffer.
// LDS (78 KB) allows two workgroups per CU.
__global__ __launch_bounds__(64 * BWAVES) void k_nd_block(NdArgs na) {
  __shared__ __attribute__((aligned(16))) short tab[BLEVELS * 4 * 2 * 64];
  __shared__ double bufA[BWAVES][BUFA];
  __shared__ double bufB[BWAVES][BUFB];
  {
    // the port tables to LDS, 16 bytes per thread and load
    constexpr int NV = BLEVELS * 4 * 2 * 64 * (int)sizeof(short) / 16;
    static_assert(BLEVELS * 4 * 2 * 64 * sizeof(short) % 16 == 0, "whole 16-byte pieces");
    const uint4* ct = reinterpret_cast<const uint4*>(&kBlkTab.s[0][0][0][0]);
    uint4* lt = reinterpret_cast<uint4*>(&tab[0]);
    for (int e = threadIdx.x; e < NV; e += 64 * BWAVES) lt[e] = ct[e];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int T = na.T;
  const int nr = T / (2 * BS);   // regions per side
  const int64_t rg = blockIdx.x;
  if (rg >= na.n_arrays * nr * nr) return;   // whole workgroups
  const int64_t la = rg / (nr * nr);
  const int sr = (int)(rg % (nr * nr));      // region
  const int RI = (sr / nr) * 2 * BS, RJ = (sr % nr) * 2 * BS;
  const int I0 = RI + (wv >> 1) * BS, J0 = RJ + (wv & 1) * BS;
  const ArrRef ref = nd_ref(na, la);
  const MapScalars& ms = *ref.ms;
  const int64_t arr = ref.arr;
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;
  double* A = bufA[wv];
  double* B = bufB[wv];
  // levels 1 x 1 .. 2 x 2 in registers, lane q < 16 taking 2 x 2 block q,
  // written to A with ports [L | R (not at the right edge) | T (not at the
  // top) | B], row stride 8, lds_mat(8) apart
  {
    // the 64 cells' conductances, one per lane (lane q + 16 r + 32 c: row r,
    // column c of 2 x 2 block q), through B to the lanes of their blocks
    const int q = lane & 15, r = (lane >> 4) & 1, c = lane >> 5;
    B[lane] = cell_conductance(ms, ref.W, wmax, arr, I0 + 2 * (q >> 2) + r, J0 + 2 * (q & 3) + c,
                               na.row_off);
  }
  wave_sync();
  if (lane < 16) {
    const int qi = lane >> 2, qj = lane & 3;
    const int gi0 = I0 + 2 * qi, gj0 = J0 + 2 * qj;
    double Gc[2][2];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int c = 0; c < 2; ++c) Gc[r][c] = B[lane + 16 * r + 32 * c];
    double X[10][10];
    block2x2(Gc, gi0, gj0, T, na.g_r, na.g_c, na.g_s, X);
    const bool rn = gj0 + 2 < T, tn = gi0 > 0;
    const int oT = rn ? 4 : 2, oB = oT + (tn ? 2 : 0);
    // padded port -> stored port (-1: absent)
    int pos[8];
    pos[0] = 0;
    pos[1] = 1;
    pos[2] = rn ? 2 : -1;
    pos[3] = rn ? 3 : -1;
    pos[4] = tn ? oT : -1;
    pos[5] = tn ? oT + 1 : -1;
    pos[6] = oB;
    pos[7] = oB + 1;
    double* o = A + lane * lds_mat(8);
#pragma unroll
    for (int p = 0; p < 8; ++p)
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const double v = p >= q ? X[2 + p][2 + q] : X[2 + q][2 + p];
        if (pos[p] >= 0 && pos[q] >= 0) o[pos[p] * 8 + pos[q]] = v;
      }
    o[64] = 0.0;   // the zero slot
  }
  wave_sync();
  level2_dpp(T, I0, J0, tab, A, B, lane);
  // the four 4 x 2 -> 4 x 4 merges (children lds_mat(12) apart in B,
  // results lds_mat(16) apart in A)
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int cm0 = (m >> 1) * 4 + (m & 1) * 2;
    merge_mfma<3, 4, 2, false, 1>(T, I0 + (m >> 1) * 4, J0 + (m & 1) * 4, tab,
                                  B + cm0 * lds_mat(12), B + (cm0 + 1) * lds_mat(12),
                                  A + m * lds_mat(16), lane);
  }
  // the two 4 x 4 -> 8 x 4 merges (children lds_mat(16) apart in A, results
  // lds_mat(24) apart in B)
#pragma unroll
  for (int m = 0; m < 2; ++m)
    merge_mfma<4, 4, 4, true, 2>(T, I0, J0 + m * 4, tab, A + m * lds_mat(16),
                                 A + (2 + m) * lds_mat(16), B + m * lds_mat(24), lane);
  // the 8 x 8 block to A (row stride 32); the region's two 16 x 8 merges
  // (children BUFA apart: the waves' A buffers) to the B buffers (row stride
  // 48); their 16 x 16 merge (the A buffers as scratch) to merged block
  // (region row, region column) of the 16 x 16 level
  merge_mfma<5, 8, 4, false, 2>(T, I0, J0, tab, B, B + lds_mat(24), A, lane);
  __syncthreads();
  {   // waves m and 2 + m: the pair of column m (children: the A buffers of
      // waves m, 2 + m), each wave half of its tiles
    const double* ca = &bufA[0][0];
    const int m = wv & 1;
    merge_mfma<6, 8, 8, true, 3, true>(T, RI, RJ + m * BS, tab, ca + m * BUFA, ca + (2 + m) * BUFA,
                                       &bufB[0][0] + m * lds_mat(48), lane, wv >> 1);
  }
  __syncthreads();
  constexpr int E16 = 8 * BS;   // ports of an interior 16 x 16 block
  double* dst = na.buf_out + la * na.out_stride +
                ((int64_t)(RI / (2 * BS)) * (T / (2 * BS)) + RJ / (2 * BS)) * E16 * E16;
  region_merge16(T, RI, RJ, &bufB[0][0], dst, &bufA[0][0]);
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

// One merge of two h x w blocks (children in buf_in, result to buf_out) with
// the cut rows in global memory: merges with more than 64 cut nodes.
__global__ __launch_bounds__(NTH) void k_nd_merge(NdArgs na) {
  constexpr int NT = NTH;
  extern __shared__ double lds[];   // the blocked elimination's panels
  __shared__ short tab[2 * 1024];   // children of a 256 x 256 grid have up to 768 ports
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
  const int ldc = c + Emax;
  double* cut = na.scratch + la * na.scr_stride + (int64_t)m * c * ldc;
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
        v[u] = Yc[sym_at(p, q, Ein)];
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
  eliminate(cut, c, E, ldc, ext, Emax, lds);
}

// Drivers and sinks: G'^T = -(Y_sL (Y_LL + g_d I)^-1 g_d E), written as fp32.
// Externals: the M source terminals t, then the T sink terminals s; cut: the
// T row-input nodes.  Only the (s, t) block of the result is needed.
__global__ __launch_bounds__(NTH) void k_nd_final(NdArgs na) {
  constexpr int NT = NTH;
  extern __shared__ double lds[];
  const int tid = threadIdx.x;
  const int T = na.T, M = na.ms.M, N = na.ms.N;
  const int64_t la = blockIdx.x;
  const int Ein = 4 * T;                 // ld of the last level's matrix (2 (T + T))
  const double* Y = na.buf_in + la * na.in_stride;
  const int E = M + T, c = T, ldc = c + E;
  double* ext = na.scratch + la * na.scr_stride;
  double* cut = ext + (int64_t)E * E;
  for (int e = tid; e < E * E; e += NT) {
    const int x = e / E, y = e % E;
    double v = 0.0;
    if (x < M && y < M) v = (x == y) ? na.g_d : 0.0;
    else if (x >= M && y >= M) v = Y[sym_at(T + x - M, T + y - M, Ein)];
    ext[e] = v;
  }
  const int lgl = lg2ceil(ldc);
  for (int e = tid; e < c << lgl; e += NT) {
    const int i = e >> lgl, y = e & ((1 << lgl) - 1);
    if (y >= ldc) continue;
    double v;
    if (y < c) v = Y[sym_at(i, y, Ein)] + (i == y ? na.g_d : 0.0);
    else if (y < c + M) v = (i == na.row_off + (y - c)) ? -na.g_d : 0.0;
    else v = Y[sym_at(i, T + (y - c - M), Ein)];
    cut[i * ldc + y] = v;
  }
  __syncthreads();
  float* out = nd_ref(na, la).out;
  eliminate(cut, c, E, ldc, ext, E, lds);
  for (int e = tid; e < na.ms.Np * na.ms.Mp; e += NT) {
    const int j = e / na.ms.Mp, k = e % na.ms.Mp;
    out[e] = (j < N && k < M) ? (float)(-ext[(int64_t)(M + j) * E + k]) : 0.0f;
  }
}

// ---------------------------------------------------------------------------
// Merges and the final step with at most 64 cut nodes: one workgroup of
// ceil(ncol / 64) waves per merge.  Lane y holds column y of the combined
// matrix (the C cut columns first, then the E externals) with all C cut rows
// in registers.  The cut block is symmetric, so row k is also column k: at
// pivot k the cut-column lanes publish row k in LDS and every lane updates
// its rows x > k with t = U[k][y] / U[k][k]:  U[x][y] -= U[k][x] t.  One
// barrier per pivot, one FMA per row and pivot.  The eliminated rows, scaled
// by D^-1/2, leave as Z (C x E, row stride Emax) for the Schur update
// ext - Z^T Z, which k_nd_schur computes on 64 x 64 tiles over many
// workgroups.
// ---------------------------------------------------------------------------
constexpr int MAXSLOT = 512;    // cut + external slots of a merge with c <= 64


// Empty asm that takes rows x0 .. x0 + 7 of U (those below N) as operands:
// their updates must be complete here and cannot be deferred past it.
template <int N>
__device__ __forceinline__ void pin8(double (&U)[N], int x0) {
  double* u = U + x0;
  if (x0 + 8 <= N) {
    asm volatile("" : "+v"(u[0]), "+v"(u[1]), "+v"(u[2]), "+v"(u[3]), "+v"(u[4]), "+v"(u[5]),
                 "+v"(u[6]), "+v"(u[7]));
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (x0 + i < N) asm volatile("" : "+v"(u[i]));
  }
}

// u += m(lane K of this row of 16 lanes) * tn: one FMA whose first operand
// comes through a DPP row broadcast (64-bit DPP takes row_newbcast only).
// The compiler does not look into inline assembly for DPP hazards: the
// s_nop gives the two wait states a DPP instruction needs after a write of
// any VGPR it reads, and the callers branch only on scalar conditions, so
// that no VALU write of EXEC comes before it.
template <int K>
__device__ __forceinline__ void fmac_bcast(double& u, double m, double tn) {
  asm("s_nop 1\n\tv_fmac_f64_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf bound_ctrl:1"
      : "+v"(u)
      : "v"(m), "v"(tn), "i"(K));
}

// The same for eight rows u[i] with the multipliers of lanes B + i, after
// one s_nop (the eight FMAs write no register that another of them reads).
template <int B>
__device__ __forceinline__ void fmac8_bcast(double* u, double m, double tn) {
#define RXNN_FMAC_DPP(d, k) \
  "v_fmac_f64_dpp %" #d ", %8, %9 row_newbcast:%" #k " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
  asm("s_nop 1\n\t" RXNN_FMAC_DPP(0, 10) RXNN_FMAC_DPP(1, 11) RXNN_FMAC_DPP(2, 12)
          RXNN_FMAC_DPP(3, 13) RXNN_FMAC_DPP(4, 14) RXNN_FMAC_DPP(5, 15) RXNN_FMAC_DPP(6, 16)
              RXNN_FMAC_DPP(7, 17)
      : "+v"(u[0]), "+v"(u[1]), "+v"(u[2]), "+v"(u[3]), "+v"(u[4]), "+v"(u[5]), "+v"(u[6]),
        "+v"(u[7])
      : "v"(m), "v"(tn), "i"(B), "i"(B + 1), "i"(B + 2), "i"(B + 3), "i"(B + 4), "i"(B + 5),
        "i"(B + 6), "i"(B + 7));
#undef RXNN_FMAC_DPP
}

// U[x0 + i] -= m(lane B + i of this row of 16 lanes) * t for the rows x0 + i
// of a chunk of 8 with x0 + i >= lo, given tn = -t (the same rounded result
// as negating the multiplier)
template <int B, int N, int... I>
__device__ __forceinline__ void fma8_bcast_seq(double (&U)[N], int x0, int lo, double m, double tn,
                                               std::integer_sequence<int, I...>) {
  ((x0 + I >= lo && x0 + I < N ? fmac_bcast<B + I>(U[x0 + I], m, tn) : (void)0), ...);
}
template <int B, int N>
__device__ __forceinline__ void fma8_bcast(double (&U)[N], int x0, int lo, double m, double tn) {
  if (x0 >= lo && x0 + 8 <= N) fmac8_bcast<B>(U + x0, m, tn);
  else fma8_bcast_seq<B>(U, x0, lo, m, tn, std::make_integer_sequence<int, 8>{});
}

// Buffer descriptor over [p, p + bytes) with a wave-uniform base and size:
// loads through it take a per-lane 32-bit offset and a scalar offset, so a
// gather of many rows holds no 64-bit address per load.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t nd_rsrc(const void* p, unsigned bytes) {
  const uint64_t a = (uint64_t)p;
  const uint64_t au = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(a >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((int)a);
  return __builtin_amdgcn_make_buffer_rsrc((void*)au, (short)0,
                                           __builtin_amdgcn_readfirstlane((int)bytes), 0x00020000);
}

// A per-lane buffer offset beyond every level buffer's range: the load returns
// 0 and touches no memory (the range check covers the VGPR offset).
constexpr unsigned kNdOob = 0x80000000u;


__device__ __forceinline__ double nd_load(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
  return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}


// Geometry of merge `m` of the level described by na (children h x w).
struct MergeGeom {
  int64_t la;
  int m, mi, mj, i0, j0, c, E, Emax, Ein, cm0, cm1;
};

__device__ __forceinline__ MergeGeom merge_geom(const NdArgs& na, int64_t blk) {
  MergeGeom g;
  const int T = na.T, h = na.h, w = na.w;
  const bool vert = na.vert != 0;
  const int nh = vert ? 2 * h : h, nw = vert ? w : 2 * w;
  const int cols = T / nw, nmerge = (T / nh) * cols;
  g.la = blk / nmerge;
  g.m = (int)(blk % nmerge);
  g.mi = g.m / cols;
  g.mj = g.m % cols;
  g.i0 = g.mi * nh;
  g.j0 = g.mj * nw;
  g.Emax = 2 * (nh + nw);
  g.c = vert ? w : h;
  g.E = nports(g.i0, g.j0, nh, nw, T);
  g.Ein = 2 * (h + w);
  const int ccols = T / w;
  g.cm0 = vert ? (g.mi * 2) * ccols + g.mj : g.mi * ccols + g.mj * 2;
  g.cm1 = vert ? (g.mi * 2 + 1) * ccols + g.mj : g.mi * ccols + g.mj * 2 + 1;
  return g;
}

// invt[ch][slot]: the port of child ch that lands on merged slot `slot`
// (cut node k -> slot k, external port d -> slot c + d), or -1.
template <int NS>
__device__ void inverse_tables(const NdArgs& na, const MergeGeom& g, short (*invt)[NS], int NT) {
  const int tid = threadIdx.x;
  const bool vert = na.vert != 0;
  // every slot -1 (no port), 16 bytes per store
  static_assert(2 * NS * sizeof(short) % 16 == 0, "whole 16-byte pieces");
  uint4* iv = reinterpret_cast<uint4*>(&invt[0][0]);
  for (int t = tid; t < 2 * NS * (int)sizeof(short) / 16; t += NT)
    iv[t] = make_uint4(~0u, ~0u, ~0u, ~0u);
  __syncthreads();
  for (int t = tid; t < 2 * g.Ein; t += NT) {
    const int ch = t / g.Ein, p = t - ch * g.Ein;
    const int ci = (vert && ch) ? g.i0 + na.h : g.i0, cj = (!vert && ch) ? g.j0 + na.w : g.j0;
    if (p < nports(ci, cj, na.h, na.w, na.T)) {
      const int d = merge_dest(ch, p, g.i0, g.j0, na.h, na.w, vert, na.T);
      invt[ch][d >= 0 ? g.c + d : -1 - d] = (short)p;
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// 64 x 64 tiles of acc[x][y] = sum_k Za[k][x] Zb[k][y] on the fp64 matrix
// cores (v_mfma_f64_16x16x4f64).  The workgroup's 4 waves each own a 32 x 32
// quarter (wave w: rows 32 (w / 2), columns 32 (w % 2)) as 2 x 2 blocks of
// 16 x 16.  Operands: lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16]
// of a 16 x 4 by 4 x 16 step; the result block holds D[l / 16 + 4 v][l % 16]
// in element v of lane l.  The k-chunks pass through LDS rows of KLD doubles:
// 16 lanes read 128 contiguous bytes, and the 640-byte row stride puts the
// four row groups of a read in different bank halves.
// ---------------------------------------------------------------------------
typedef double f64x4 __attribute__((ext_vector_type(4)));
constexpr int KC64 = 16;      // k per LDS chunk
constexpr int KLD = 80;       // LDS row stride (doubles)

struct MfmaTile {
  f64x4 acc[2][2];
  int wr, wc, lr, lc;         // wave quarter, lane row group, lane column
  __device__ __forceinline__ void init(int tid) {
    const int wv = tid >> 6, lane = tid & 63;
    wr = wv >> 1;
    wc = wv & 1;
    lr = lane >> 4;
    lc = lane & 15;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
  }
  // one chunk of KC64 k from LDS (za, zb: [KC64][KLD], k-major)
  __device__ __forceinline__ void step(const double* za, const double* zb) {
#pragma unroll
    for (int k4 = 0; k4 < KC64; k4 += 4) {
      double a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = za[(k4 + lr) * KLD + wr * 32 + i * 16 + lc];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = zb[(k4 + lr) * KLD + wc * 32 + j * 16 + lc];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
  // kn k (a multiple of 4) from k-major LDS rows of ld doubles; columns at or
  // beyond `lim` of either operand read as 0
  __device__ __forceinline__ void step_ld(const double* za, const double* zb, int ld, int kn,
                                          int xlim, int ylim) {
    for (int k4 = 0; k4 < kn; k4 += 4) {
      double a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int x = wr * 32 + i * 16 + lc;
        a[i] = x < xlim ? za[(k4 + lr) * ld + x] : 0.0;
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int y = wc * 32 + j * 16 + lc;
        b[j] = y < ylim ? zb[(k4 + lr) * ld + y] : 0.0;
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
  // tile-local coordinates of this lane's element v of block (i, j)
  __device__ __forceinline__ int row(int i, int v) const { return wr * 32 + i * 16 + lr + 4 * v; }
  __device__ __forceinline__ int col(int j) const { return wc * 32 + j * 16 + lc; }
};

// Workgroups are dispatched to the 8 XCDs in turn, each with its own L2: this
// renumbering gives every XCD a contiguous range of logical workgroups, so the
// tiles of one merge (which all read its Z) share one L2.
__device__ __forceinline__ int64_t nd_xcd(int64_t i, int64_t n) {
  const int64_t q = n >> 3, r = n & 7, x = i & 7, j = i >> 3;
  return x * q + (x < r ? x : r) + j;
}

// Tile (tx, ty), tx >= ty, of the lower triangle of an nt x nt tile grid from
// its index tt in row-major order of that triangle.
__device__ __forceinline__ void tri_tile(int tt, int* tx, int* ty) {
  int x = (int)((sqrtf(8.0f * (float)tt + 1.0f) - 1.0f) * 0.5f);
  while ((x + 1) * (x + 2) / 2 <= tt) ++x;
  while (x * (x + 1) / 2 > tt) --x;
  *tx = x;
  *ty = tt - x * (x + 1) / 2;
}

// One merge of the region kernel by one wave, with its Schur update on the
// fp64 matrix cores: level L, children H x W (VERT: stacked), the merged
// block at (i0, j0), children c0 and c1 (matrices of EIN ports, row stride
// EIN), result to `out` (row stride EM = the merged block's largest port
// count).  Lane y holds column y of the merge's C cut rows only and
// eliminates them (pivot k's column by lane reads from lane k); Z (the
// eliminated rows scaled by D^-1/2, zero past the block's ports and in the
// rows that pad C to a multiple of 4) goes to `out` as scratch, under the
// last tile row, and the merged block V - Z^T Z is NB x NB tiles of 16 x 16
// (lane l: rows 16 bi + l / 16 + 4 v, column 16 bj + l % 16), each written
// at once except the last tile row's, which waits until Z is read.  SPLIT:
// two waves share the merge (every wave of the workgroup calls it, so the
// waits are workgroup barriers): both eliminate, part 0 writes Z and takes
// the first half of the tiles in row-major order, part 1 the rest.
template <int L, int H, int W, bool VERT, int NB, bool SPLIT>
__device__ __forceinline__ void merge_mfma(int T, int i0, int j0, const short* tab,
                                           const double* c0, const double* c1, double* out,
                                           int lane, int part) {
  constexpr int NH = VERT ? 2 * H : H, NW = VERT ? W : 2 * W;
  constexpr int C = VERT ? W : H;
  constexpr int EM = 2 * (NH + NW), EIN = 2 * (H + W), ZS = 16 * NB, CK = (C + 3) & ~3;
  static_assert(C <= 16 && EM <= 16 * NB && EM > 16 * (NB - 1) && C + 16 * NB <= 64,
                "one wave per merge");
  static_assert(CK * ZS <= (EM - 16 * (NB - 1)) * EM, "Z only under the last tile row");
  const bool rn = j0 + NW < T, tn = i0 > 0;
  const int E = NH + (rn ? NH : 0) + (tn ? NW : 0) + NW;   // ports of the merged block
  const short* t0 = tab + (((L * 4) + (rn ? 2 : 0) + (tn ? 1 : 0)) * 2) * 64;
  const short* t1 = t0 + 64;
  const int k0 = col_key(t0[lane]), k1 = col_key(t1[lane]);
  double U[C];
#pragma unroll
  for (int x = 0; x < C; ++x) U[x] = pick(c0, t0[x], k0, EIN) + pick(c1, t1[x], k1, EIN);
  double sq[C];
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const double piv = readlane_d(U[k], k);
    sq[k] = rsqrt_nr(piv);
    const double t = U[k] * recip(piv);
#pragma unroll
    for (int x = k + 1; x < C; ++x) U[x] = fma(-readlane_d(U[x], k), t, U[x]);
  }
  double* z = out + 16 * (NB - 1) * EM;
  if (lane >= C && lane < C + 16 * NB && (!SPLIT || part == 0)) {
    const int e = lane - C;
#pragma unroll
    for (int k = 0; k < CK; ++k) z[k * ZS + e] = (k < C && e < E) ? U[k] * sq[k] : 0.0;
  }
  if constexpr (SPLIT) __syncthreads();
  else wave_sync();
  const int lr = lane >> 4, lc = lane & 15;
  // tile by tile (few registers live): its product and V entries; the
  // last tile row waits in registers until every tile has read Z
  double res[NB][4];
#pragma unroll
  for (int bi = 0; bi < NB; ++bi)
#pragma unroll
    for (int bj = 0; bj < NB; ++bj) {
      if (SPLIT && (bi * NB + bj < (NB * NB + 1) / 2) != (part == 0)) continue;
      const int yy = 16 * bj + lc;
      const int kb0 = col_key(t0[C + yy]), kb1 = col_key(t1[C + yy]);
      f64x4 acc = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int k4 = 0; k4 < CK; k4 += 4) {
        const double a = z[(k4 + lr) * ZS + 16 * bi + lc];
        const double b = z[(k4 + lr) * ZS + 16 * bj + lc];
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int xx = 16 * bi + lr + 4 * v;
        const double r =
            pick(c0, t0[C + xx], kb0, EIN) + pick(c1, t1[C + xx], kb1, EIN) - acc[v];
        if (bi + 1 < NB) {
          if (xx < E && yy < E) out[xx * EM + yy] = r;
        } else {
          res[bj][v] = r;
        }
      }
    }
  // Z read before the last tile row overwrites it
  if constexpr (SPLIT) __syncthreads();
  else wave_sync();
#pragma unroll
  for (int bj = 0; bj < NB; ++bj) {
    if (SPLIT && ((NB - 1) * NB + bj < (NB * NB + 1) / 2) != (part == 0)) continue;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int xx = 16 * (NB - 1) + lr + 4 * v, yy = 16 * bj + lc;
      if (xx < E && yy < E) out[xx * EM + yy] = res[bj][v];
    }
  }
  if (lane == 0 && (!SPLIT || part == 0)) out[EM * EM] = 0.0;   // the zero slot
  wave_sync();
}

// The 16 x 16 merge of a region's two 16 x 8 halves (left, right) at (RI, RJ):
// ch holds them in LDS (row stride 48, lds_mat(48) apart), the merged block
// (E <= 64 ports, row stride 64) goes to dst, scr is LDS scratch of at least
// 1400 doubles.  Waves 0 and 1 each hold, lane by lane, columns of the
// combined matrix's 16 cut rows (the shared a-nodes): lanes 0 .. 15 the cut
// columns (both waves), the other lanes externals 0 .. 47 (wave 0) and
// 48 .. 63 (wave 1).  Each wave eliminates the cut rows by itself, taking
// pivot k's column from lane k by lane reads (no barriers); Z (the
// eliminated rows scaled by D^-1/2) goes to LDS, and the external block
// V - Z^T Z is one 64 x 64 tile on the fp64 matrix cores (all four waves).
__device__ void region_merge16(int T, int RI, int RJ, const double* ch, double* dst,
                               double* scr) {
  constexpr int C = 16, EIN = 48, CH1 = EIN * EIN + 1, ZL = 68;
  const int tid = threadIdx.x;
  short* invt = reinterpret_cast<short*>(scr);   // [2][80]
  double* zl = scr + 48;                         // [16][ZL]
  const int E = nports(RI, RJ, C, C, T);
  for (int t = tid; t < 160; t += 256) invt[t] = -1;
  __syncthreads();
  if (tid < 2 * EIN) {
    const int c = tid / EIN, p = tid - c * EIN;
    if (p < nports(RI, RJ + c * (C / 2), C, C / 2, T)) {
      const int d = merge_dest(c, p, RI, RJ, C, C / 2, false, T);
      invt[c * 80 + (d >= 0 ? C + d : -1 - d)] = (short)p;
    }
  }
  __syncthreads();
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  if (wv < 2) {
    const int y = lane < C ? lane : C + 48 * wv + (lane - C);   // combined column
    const int kb0 = col_key(y < C + E ? invt[y] : -1), kb1 = col_key(y < C + E ? invt[80 + y] : -1);
    double U[C];
#pragma unroll
    for (int x = 0; x < C; ++x)
      U[x] = pick(ch, invt[x], kb0, EIN) + pick(ch + CH1, invt[80 + x], kb1, EIN);
    double sq[C];
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const double piv = readlane_d(U[k], k);
      sq[k] = rsqrt_nr(piv);
      const double t = U[k] * recip(piv);
#pragma unroll
      for (int x = k + 1; x < C; ++x) U[x] = fma(-readlane_d(U[x], k), t, U[x]);
    }
    if (lane >= C && y < C + E) {
#pragma unroll
      for (int x = 0; x < C; ++x) zl[x * ZL + (y - C)] = U[x] * sq[x];
    }
  }
  __syncthreads();
  MfmaTile mt;
  mt.init(tid);
  double vv[2][2][4];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int yy = min(mt.col(j), E - 1);
    const int kb0 = col_key(invt[C + yy]), kb1 = col_key(invt[80 + C + yy]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int x = min(mt.row(i, v), E - 1);
        vv[i][j][v] = pick(ch, invt[C + x], kb0, EIN) + pick(ch + CH1, invt[80 + C + x], kb1, EIN);
      }
  }
  mt.step_ld(zl, zl, ZL, C, E, E);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int x = mt.row(i, v), yy = mt.col(j);
        if (x < E && yy < E) dst[x * 64 + yy] = vv[i][j][v] - mt.acc[i][j][v];
      }
}

// MODE 0: a merge (children through the port tables); 1: the final step;
// 2: a stage of a dense combined matrix (its first C rows are the pivots,
// the rest of its columns are handled in panels of na.dpanel).
template <int C, int MODE>
__global__ __launch_bounds__(512) void k_nd_cut(NdArgs na) {
  static_assert(C <= 64, "at most 64 cut rows");
  constexpr bool FINAL = MODE == 1;
  __shared__ __attribute__((aligned(16))) short invt[2][MAXSLOT];
  __shared__ double rowb[2][64];
  __shared__ double isq[64];
  // final step: the eliminated rows' sink and source columns for G'
  __shared__ double zs[FINAL ? C : 1][FINAL ? 64 + 2 : 1];
  __shared__ double zq[FINAL ? C : 1][FINAL ? 64 + 2 : 1];
  // small merges (C <= 32 cut nodes, at most 192 ports): Z stays in LDS and
  // this workgroup also computes the Schur update on fp64 MFMA tiles
  constexpr bool kFuse = MODE == 0 && C <= 32;
  constexpr int ZLD = C <= 8 ? 52 : (C <= 16 ? 100 : 196);   // Z row stride in LDS
  __shared__ __attribute__((aligned(16))) double zl[kFuse ? C * ZLD : 1];
  // merges and dense stages with 64 cut rows: a wave's batch of 8 rows of
  // the gather on its way to the lanes of their columns
  constexpr bool kTGather = (MODE == 0 || MODE == 2) && C == 64;
  constexpr int TBL = 65;
  __shared__ double tb[kTGather ? 8 : 1][kTGather ? 8 * TBL : 1];
  const int y = threadIdx.x;
  const int T = na.T;
  int E, ncol, Emax = 0;
  int zld = 0, ebase = 0;   // Z row stride, first external column of this workgroup
  int64_t la;
  double* z = nullptr;
  double U[C];
  MergeGeom g{};
  const double* Y0 = nullptr;
  const double* Y1 = nullptr;
  if constexpr (MODE == 2) {
    const int npan = (na.dn - C + na.dpanel - 1) / na.dpanel;
    la = blockIdx.x / npan;
    const int pn = (int)(blockIdx.x % npan);
    E = na.dn - C;
    zld = E;
    ebase = pn * na.dpanel;
    ncol = C + min(na.dpanel, E - ebase);
    z = na.scratch + la * na.scr_stride;
    const double* A = na.dA + la * na.in_stride;
    const int col = y < C ? y : (y < ncol ? C + ebase + (y - C) : 0);
    // the pivot rows' entries A[x][col] are read as A[col][x] (A is
    // symmetric, and a stage writes only its lower tiles)
    const __amdgpu_buffer_rsrc_t ra = nd_rsrc(A, (unsigned)(na.dn * na.dld * 8));
    if constexpr (kTGather) {
      // batches of 8 rows in 8 x 8 blocks through LDS, as for the merges:
      // lane l loads entry x0 + l % 8 of column c0 + 8 s + l / 8, eight lanes
      // 64 contiguous bytes of one row of A
      const int lane = y & 63, xq = lane & 7, yq = lane >> 3;
      const int c0 = y - lane;   // the wave's first column
      double* tw = &tb[y >> 6][0];
      unsigned ro[8];            // byte offsets of the columns' rows of A (out of range: none)
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int ys = c0 + 8 * s + yq;
        const int cs = ys < C ? ys : (ys < ncol ? C + ebase + (ys - C) : -1);
        ro[s] = cs >= 0 ? 8u * (unsigned)(cs * na.dld) : kNdOob;
      }
#pragma unroll
      for (int b = 0; b < C / 8; ++b) {
        double v[8];
#pragma unroll
        for (int s = 0; s < 8; ++s)
          v[s] = nd_load(ra, ro[s] == kNdOob ? kNdOob : ro[s] + 8u * (unsigned)(8 * b + xq), 0);
#pragma unroll
        for (int s = 0; s < 8; ++s) tw[xq * TBL + 8 * s + yq] = v[s];
        wave_sync();
#pragma unroll
        for (int i = 0; i < 8; ++i) U[8 * b + i] = tw[i * TBL + lane];
        pin8(U, 8 * b);
        wave_sync();   // read before the next batch is written
      }
    } else {
#pragma unroll
      for (int x = 0; x < C; ++x) {
        const double v = nd_load(ra, 8u * (unsigned)(col * na.dld), 8u * (unsigned)x);
        U[x] = y < ncol ? v : 0.0;
        if ((x & 15) == 15) {
          pin8(U, x - 15);
          pin8(U, x - 7);
        }
      }
    }
  } else if constexpr (FINAL) {
    la = blockIdx.x;
    E = na.ms.M + T;
    ncol = C + E;
    const int Ein = 4 * T, M = na.ms.M;
    const double* Y = na.buf_in + la * na.in_stride;
    // column of this lane in the last level's matrix (clamped: always valid);
    // branch-free, so that the loads of a chunk stay in flight together
    const bool useY = y < C || (y >= C + M && y < ncol);
    const int yc = y < C ? y : (useY ? T + (y - C - M) : 0);
    const int srow = (y >= C && y < C + M) ? na.row_off + (y - C) : -1;   // driver of row
    const __amdgpu_buffer_rsrc_t ry = nd_rsrc(Y, (unsigned)(2 * T * Ein * 8));
#pragma unroll
    for (int x = 0; x < C; ++x) {
      const double yv = nd_load(ry, 8u * (unsigned)sym_at(x, yc, Ein), 0);
      const double v = (useY ? yv : 0.0) + (x == y ? na.g_d : 0.0) - (x == srow ? na.g_d : 0.0);
      U[x] = v;
      if ((x & 31) == 31) {   // 32 loads in flight per round trip
        pin8(U, x - 31);
        pin8(U, x - 23);
        pin8(U, x - 15);
        pin8(U, x - 7);
      }
    }
  } else {
    // with several panels per merge, workgroup pn takes the cut columns and
    // externals [pn dpanel, (pn + 1) dpanel)
    const int npan = max(na.npan, 1), pn = (int)(blockIdx.x % npan);
    g = merge_geom(na, blockIdx.x / npan);
    inverse_tables<MAXSLOT>(na, g, invt, blockDim.x);
    la = g.la;
    E = g.E;
    Emax = g.Emax;
    zld = Emax;
    ebase = npan > 1 ? pn * na.dpanel : 0;
    ncol = C + (npan > 1 ? max(0, min(na.dpanel, E - ebase)) : E);
    z = na.scratch + la * na.scr_stride + (int64_t)g.m * g.Emax * C;
    Y0 = na.buf_in + la * na.in_stride + (int64_t)g.cm0 * g.Ein * g.Ein;
    Y1 = na.buf_in + la * na.in_stride + (int64_t)g.cm1 * g.Ein * g.Ein;
    const int slot = y < C ? y : (y < ncol ? C + ebase + (y - C) : -1);
    const int pb0 = slot >= 0 ? invt[0][slot] : -1, pb1 = slot >= 0 ? invt[1][slot] : -1;
    const unsigned cb = (unsigned)(g.Ein * g.Ein * 8);
    const __amdgpu_buffer_rsrc_t r0 = nd_rsrc(Y0, cb), r1 = nd_rsrc(Y1, cb);
    const lds_i16* iv = opaque_lds<lds_i16>(&invt[0][0]);
    if constexpr (kTGather) {
      // batches of 8 rows: lane l loads the entry of row x0 + l % 8 and
      // column c0 + 8 s + l / 8 (s = 0 .. 7), so that eight lanes read 64
      // contiguous bytes whichever mirror position of the entry the child
      // stores (lower tiles only); the batch passes through LDS to the lanes
      // of its columns
      const int lane = y & 63, xq = lane & 7, yq = lane >> 3;
      const int c0 = y - lane;   // the wave's first column
      double* tw = &tb[y >> 6][0];
      int qb[8];   // the ports of column c0 + 8 s + l / 8 in the children, 16 bits each
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int ys = c0 + 8 * s + yq;
        const int sl = ys < C ? ys : (ys < ncol ? C + ebase + (ys - C) : -1);
        const int q0 = sl >= 0 ? invt[0][sl] : -1, q1 = sl >= 0 ? invt[1][sl] : -1;
        qb[s] = (q0 & 0xffff) | (q1 << 16);
      }
#pragma unroll
      for (int b = 0; b < C / 8; ++b) {
        const int pa0 = iv[8 * b + xq], pa1 = iv[MAXSLOT + 8 * b + xq];
        double v[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const int q0 = (int)(short)(qb[s] & 0xffff), q1 = qb[s] >> 16;
          const double v0 = nd_load(r0, (pa0 >= 0 && q0 >= 0) ? 8u * (unsigned)sym_at(pa0, q0, g.Ein)
                                                              : kNdOob, 0);
          const double v1 = nd_load(r1, (pa1 >= 0 && q1 >= 0) ? 8u * (unsigned)sym_at(pa1, q1, g.Ein)
                                                              : kNdOob, 0);
          v[s] = v0 + v1;
        }
#pragma unroll
        for (int s = 0; s < 8; ++s) tw[xq * TBL + 8 * s + yq] = v[s];
        wave_sync();
#pragma unroll
        for (int i = 0; i < 8; ++i) U[8 * b + i] = tw[i * TBL + lane];
        pin8(U, 8 * b);
        wave_sync();   // read before the next batch is written
      }
    } else {
      // the row's port is uniform, the column's fixed per lane; an entry
      // without a port takes the out-of-range offset, so it reads 0 without a
      // memory access, and every load of a chunk stays in flight together
#pragma unroll
      for (int x = 0; x < C; ++x) {
        const int pa0 = __builtin_amdgcn_readfirstlane(iv[x]);
        const int pa1 = __builtin_amdgcn_readfirstlane(iv[MAXSLOT + x]);
        const double v0 = nd_load(r0, (pa0 >= 0 && pb0 >= 0) ? 8u * (unsigned)sym_at(pa0, pb0, g.Ein)
                                                             : kNdOob, 0);
        const double v1 = nd_load(r1, (pa1 >= 0 && pb1 >= 0) ? 8u * (unsigned)sym_at(pa1, pb1, g.Ein)
                                                             : kNdOob, 0);
        U[x] = v0 + v1;
        // 16 rows (32 loads) in flight per round trip
        if ((x & 15) == 15) {
          pin8(U, x - 15);
          pin8(U, x - 7);
        }
      }
    }
  }
  if (y < C) rowb[0][y] = U[0];
  const lds_f64* rbase = opaque_lds<lds_f64>(&rowb[0][0]);
  constexpr int G = C < 16 ? C : 16;   // rows per multiplier read
  const int lg = y & (G - 1);
#pragma clang loop unroll(full)
  for (int k = 0; k < C; ++k) {
    __syncthreads();
    const lds_f64* rb = rbase + (k & 1) * 64;
    const double piv = rb[k];
    if (y == 0) isq[k] = piv;
    const double t = U[k] * recip(piv);
    // row k + 1 first, so that it is published early; every row is updated
    // here (the empty asm keeps the compiler from deferring an update to the
    // row's own pivot, which would hold every pivot row's values live)
    if (k + 1 < C) {
      U[k + 1] = fma(-rb[k + 1], t, U[k + 1]);
      if (y < C) rowb[(k + 1) & 1][y] = U[k + 1];
    }
    // rows k + 2 .. in groups of G: lane l of every row of 16 lanes reads
    // the multiplier of row g0 + l % G (one LDS read per group, where each
    // lane reading every multiplier would make the loop bound by LDS
    // bandwidth), and the FMA of row g0 + i takes it from lane i of its
    // row of lanes (DPP row broadcast); t is negated instead of the
    // multiplier, which gives the same rounded result
    const double tn = -t;
    double m[C / G];
#pragma clang loop unroll(full)
    for (int g0 = 0; g0 < C; g0 += G)
      if (g0 + G > k + 2) m[g0 / G] = rb[g0 + lg];
#pragma clang loop unroll(full)
    for (int g0 = 0; g0 < C; g0 += G) {
      if (g0 + G <= k + 2) continue;
#pragma clang loop unroll(full)
      for (int x0 = g0; x0 < g0 + G; x0 += 8) {
        if (x0 + 8 <= k + 2) continue;
        if (x0 % G == 0) fma8_bcast<0>(U, x0, k + 2, m[g0 / G], tn);
        else fma8_bcast<8>(U, x0, k + 2, m[g0 / G], tn);
        pin8(U, x0);
      }
    }
  }
  __syncthreads();
  if (y < C) isq[y] = 1.0 / sqrt(isq[y]);
  __syncthreads();
  const lds_f64* is = opaque_lds<lds_f64>(&isq[0]);
  if constexpr (kFuse) {
    if (na.fuse && Emax <= ZLD - 4) {   // schur_fused(C, Emax): launched with 256 threads
      if (y >= C && y < ncol) {
#pragma unroll
        for (int x = 0; x < C; ++x) zl[x * ZLD + (y - C)] = U[x] * is[x];
      }
      __syncthreads();
      double* ext = na.buf_out + la * na.out_stride + (int64_t)g.m * Emax * Emax;
      // an entry of V is one child's (an external port is a port of one
      // child only): one load per entry over both children's blocks
      const int cml = min(g.cm0, g.cm1);
      const unsigned e2 = (unsigned)(g.Ein * g.Ein);
      const unsigned o0 = (unsigned)(g.cm0 - cml) * e2, o1 = (unsigned)(g.cm1 - cml) * e2;
      const __amdgpu_buffer_rsrc_t ry =
          nd_rsrc(na.buf_in + la * na.in_stride + (int64_t)cml * e2,
                  (unsigned)(abs(g.cm1 - g.cm0) + 1) * e2 * 8u);
      const int nt = (E + 63) / 64;
      // ext = V - Z^T Z on the 64 x 64 tiles of its lower triangle (ext is
      // symmetric; readers take the mirror of an entry above); the children's
      // entries of a tile are loaded before its product, so that they arrive
      // during it
      // at the bottom of the grid, tiles wholly among the B ports (sinks)
      const int bsink = g.i0 + (na.vert ? 2 * na.h : na.h) == T ? E - (na.vert ? na.w : 2 * na.w)
                                                              : E;
#pragma unroll 1
      for (int tt = 0; tt < nt * (nt + 1) / 2; ++tt) {
        int tx, ty;
        tri_tile(tt, &tx, &ty);
        const int x0 = tx * 64, y0 = ty * 64;
        if (x0 >= bsink && y0 >= bsink) continue;
        MfmaTile mt;
        mt.init(threadIdx.x);
        double vv[2][2][4];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int yy = min(y0 + mt.col(j), E - 1);
          const int pb0 = invt[0][C + yy], pb1 = invt[1][C + yy];
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int x = min(x0 + mt.row(i, v), E - 1);
              const int pa0 = invt[0][C + x], pa1 = invt[1][C + x];
              const unsigned off =
                  (pa0 >= 0 && pb0 >= 0)   ? 8u * (o0 + (unsigned)sym_at(pa0, pb0, g.Ein))
                  : (pa1 >= 0 && pb1 >= 0) ? 8u * (o1 + (unsigned)sym_at(pa1, pb1, g.Ein))
                                           : kNdOob;
              vv[i][j][v] = nd_load(ry, off, 0);
            }
        }
        mt.step_ld(zl + x0, zl + y0, ZLD, C, E - x0, E - y0);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int x = x0 + mt.row(i, v), yy = y0 + mt.col(j);
              if (x < E && yy < E) {
                ext[x * Emax + yy] = vv[i][j][v] - mt.acc[i][j][v];
              }
            }
      }
      return;
    }
  }
  if (!FINAL) {
    // Z[x][ebase + y - C] = U[x][y] / sqrt(D_x) for the external columns
    if (y >= C && y < ncol) {
      double* zc = z + (unsigned)(ebase + y - C);
#pragma unroll
      for (int x = 0; x < C; ++x) {
        zc[(unsigned)(x * zld)] = U[x] * is[x];
        if ((x & 15) == 15) __builtin_amdgcn_sched_barrier(0);
      }
    }
    return;
  }
  // G'[j][k] = sum_x Z[x][sink j] Z[x][source k]
  const int M = na.ms.M, N = na.ms.N;
  if (y >= C && y < C + M && y - C < 64) {
#pragma unroll
    for (int x = 0; x < C; ++x) zq[x][y - C] = U[x] * is[x];
  } else if (y >= C + M && y < ncol && y - C - M < 64) {
#pragma unroll
    for (int x = 0; x < C; ++x) zs[x][y - C - M] = U[x] * is[x];
  }
  __syncthreads();
  float* out = nd_ref(na, la).out;
  const int Np = na.ms.Np, Mp = na.ms.Mp;
  for (int it = threadIdx.x; it < 256; it += blockDim.x) {
    const int tx = it >> 4, ty = it & 15;
    if (4 * tx >= Np || 4 * ty >= Mp) continue;
    double acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = 0.0;
#pragma unroll 4
    for (int x = 0; x < C; ++x) {
      double sa[4], qb[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) sa[a] = zs[x][4 * tx + a];
#pragma unroll
      for (int b = 0; b < 4; ++b) qb[b] = zq[x][4 * ty + b];
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = fma(sa[a], qb[b], acc[a][b]);
    }
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int j = 4 * tx + a;
      if (j >= Np) continue;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int k = 4 * ty + b;
        if (k < Mp) out[j * Mp + k] = (j < N && k < M) ? (float)acc[a][b] : 0.0f;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Merges and the final step with 128 cut nodes: two row groups of 64 (lane y
// of row group rg holds rows 64 rg .. 64 rg + 63 of column y in registers),
// columns = the 128 cut columns plus a panel of up to 256 external columns
// per workgroup (the cut block is eliminated again in every panel's
// workgroup, so the panels need no exchange).  Pivot k: the row group
// holding row k publishes it in LDS with the entries at and left of the
// pivot column set to zero, so that every lane applies the pivot to all its
// rows with one FMA each and no row test (a zero multiplier leaves a row
// unchanged); chunks of 8 rows wholly at or above the pivot are skipped.
// Every lane reads one multiplier per 16 rows from LDS and the FMAs take them
// by DPP row broadcast (the LDS traffic of every lane reading every
// multiplier would bound the loop).  The pivots go in pairs, one barrier per
// pair (below); the loop runs over blocks of 8 pivots unrolled, which keeps
// the code small.  The gather takes 8 x 8 blocks through LDS (below).  Z
// (the eliminated rows scaled by D^-1/2, over this panel's externals) goes
// to scratch for k_nd_schur or, for the final step, for k_nd_gprod.
// ---------------------------------------------------------------------------
constexpr int C2 = 128;              // cut nodes
constexpr int P2 = 256;              // external columns per panel
constexpr int CP2 = C2 + P2;         // columns per workgroup
constexpr int MAXSLOT2 = 1024;       // slots of a merge with 128 cut nodes (<= 7 c)

template <bool FINAL>
__global__ __launch_bounds__(2 * CP2) void k_nd_cut2(NdArgs na) {
  __shared__ __attribute__((aligned(16))) short invt[2][FINAL ? 1 : MAXSLOT2];
  __shared__ double rowb[2][2][CP2];   // [pair parity][row of the pair][column]
  __shared__ double pivs[2][3];
  __shared__ double dg[C2];
  // a wave's batch of 8 rows on its way to the lanes of their columns
  constexpr int TBL = 65;
  __shared__ double tb[FINAL ? 1 : 2 * CP2 / 64][FINAL ? 1 : 8 * TBL];
  // rg: uniform per wave (CP2 is a multiple of 64), kept in a scalar register
  const int yl = threadIdx.x % CP2, rg = __builtin_amdgcn_readfirstlane(threadIdx.x / CP2);
  const int T = na.T;
  int64_t la;
  int E, zld, pn;
  double* z;
  double U[64];
  if constexpr (FINAL) {
    la = blockIdx.x;
    pn = 0;
    E = na.ms.M + T;
    zld = E;
    z = na.scratch + la * na.scr_stride;
    const int Ein = 4 * T, M = na.ms.M;
    const double* Y = na.buf_in + la * na.in_stride;
    const int e = yl - C2;
    const bool useY = yl < C2 || (e >= M && e < E);
    const int yc = yl < C2 ? yl : (useY ? T + (e - M) : 0);
    const int srow = (e >= 0 && e < M) ? na.row_off + e : -1;
    const __amdgpu_buffer_rsrc_t ry = nd_rsrc(Y, (unsigned)(2 * T * Ein * 8));
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      const int x = 64 * rg + i;
      const double yv = nd_load(ry, 8u * (unsigned)sym_at(x, yc, Ein), 0);
      U[i] = (useY ? yv : 0.0) + (x == yl ? na.g_d : 0.0) - (x == srow ? na.g_d : 0.0);
      if ((i & 7) == 7) pin8(U, i - 7);
    }
  } else {
    const int nh = na.vert ? 2 * na.h : na.h, nw = na.vert ? na.w : 2 * na.w;
    const int npan = (2 * (nh + nw) + P2 - 1) / P2;
    pn = (int)(blockIdx.x % npan);
    const MergeGeom g = merge_geom(na, blockIdx.x / npan);
    inverse_tables<MAXSLOT2>(na, g, invt, 2 * CP2);
    la = g.la;
    E = g.E;
    zld = g.Emax;
    z = na.scratch + la * na.scr_stride + (int64_t)g.m * g.Emax * C2;
    const double* Y0 = na.buf_in + la * na.in_stride + (int64_t)g.cm0 * g.Ein * g.Ein;
    const double* Y1 = na.buf_in + la * na.in_stride + (int64_t)g.cm1 * g.Ein * g.Ein;
    const unsigned cb = (unsigned)(g.Ein * g.Ein * 8);
    const __amdgpu_buffer_rsrc_t r0 = nd_rsrc(Y0, cb), r1 = nd_rsrc(Y1, cb);
    // batches of 8 rows: lane l loads the entry of row x0 + l % 8 and column
    // c0 + 8 s + l / 8 (s = 0 .. 7), so that eight lanes read 64 contiguous
    // bytes whichever mirror position of the entry the child stores (lower
    // tiles only); the batch passes through LDS to the lanes of its columns
    const int lane = threadIdx.x & 63, xq = lane & 7, yq = lane >> 3;
    const int c0 = yl - lane;   // the wave's first column
    double* tw = &tb[threadIdx.x >> 6][0];
    int qb[8];   // the ports of column c0 + 8 s + l / 8 in the children, 16 bits each
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int ys = c0 + 8 * s + yq, es = pn * P2 + (ys - C2);
      const int slot = ys < C2 ? ys : (es < E ? C2 + es : -1);
      const int q0 = slot >= 0 ? invt[0][slot] : -1, q1 = slot >= 0 ? invt[1][slot] : -1;
      qb[s] = (q0 & 0xffff) | (q1 << 16);
    }
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const int x = 64 * rg + 8 * b + xq;
      const int pa0 = invt[0][x], pa1 = invt[1][x];
      double v[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int pb0 = (int)(short)(qb[s] & 0xffff), pb1 = qb[s] >> 16;
        const double v0 = nd_load(r0, (pa0 >= 0 && pb0 >= 0) ? 8u * (unsigned)sym_at(pa0, pb0, g.Ein)
                                                             : kNdOob, 0);
        const double v1 = nd_load(r1, (pa1 >= 0 && pb1 >= 0) ? 8u * (unsigned)sym_at(pa1, pb1, g.Ein)
                                                             : kNdOob, 0);
        v[s] = v0 + v1;
      }
#pragma unroll
      for (int s = 0; s < 8; ++s) tw[xq * TBL + 8 * s + yq] = v[s];
      wave_sync();
#pragma unroll
      for (int i = 0; i < 8; ++i) U[8 * b + i] = tw[i * TBL + lane];
      pin8(U, 8 * b);
      wave_sync();   // read before the next batch is written
    }
  }
  // pivots in pairs (k, k + 1), one barrier per pair: rows k and k + 1 as
  // they stand before pivot k are published with the entries at and left of
  // column k + 1 set to zero, with S[k][k], S[k][k + 1], S[k + 1][k + 1]
  // apart; every lane derives row k + 1 after pivot k (in its own column and,
  // for the multipliers, in the columns of its row of 16 lanes), which gives
  // the same rounded values as eliminating one pivot per barrier
  if (rg == 0) {
    rowb[0][0][yl] = yl > 1 ? U[0] : 0.0;
    rowb[0][1][yl] = yl > 1 ? U[1] : 0.0;
    if (yl == 0) pivs[0][0] = U[0];
    if (yl == 1) {
      pivs[0][1] = U[0];
      pivs[0][2] = U[1];
    }
  }
  const int l16 = threadIdx.x & 15;
  const lds_f64* rbase = opaque_lds<lds_f64>(&rowb[0][0][0]);
#pragma unroll 1
  for (int q = 0; q < C2 / 8; ++q) {
#pragma clang loop unroll(full)
    for (int p = 0; p < 4; ++p) {
      const int k = 8 * q + 2 * p, par = p & 1;
      __syncthreads();
      const lds_f64* r0 = rbase + 2 * par * CP2;
      const lds_f64* r1 = r0 + CP2;
      const double d0 = pivs[par][0], s01 = pivs[par][1], e11 = pivs[par][2];
      const double rd0 = recip(d0);
      // S[k + 1][k + 1] after pivot k
      const double d1 = fma(s01, -(s01 * rd0), e11);
      if (threadIdx.x == 0) {
        dg[k] = d0;
        dg[k + 1] = d1;
      }
      // negated t of both pivots for this lane's column (the same rounded
      // result as negating the multipliers); row k + 1 after pivot k
      const double t0n = -(r0[yl] * rd0);
      const double t1n = -(fma(s01, t0n, r1[yl]) * recip(d1));
      // lane l of every row of 16 lanes takes the multipliers of row
      // xb + l % 16 (xb = 64 rg + 16 j) for both pivots; row xb + i takes
      // them from lane i (DPP row broadcast)
#pragma clang loop unroll(full)
      for (int j = 0; j < 4; ++j) {
        const int xb = 64 * rg + 16 * j;
        if (xb + 15 > k + 1) {
          const double m0 = r0[xb + l16];
          const double m1 = fma(s01, -(m0 * rd0), r1[xb + l16]);
#pragma clang loop unroll(full)
          for (int h = 0; h < 2; ++h) {
            if (xb + 8 * h + 7 > k + 1) {
              if (h == 0) {
                fma8_bcast<0>(U, 16 * j, 0, m0, t0n);
                fma8_bcast<0>(U, 16 * j, 0, m1, t1n);
              } else {
                fma8_bcast<8>(U, 16 * j + 8, 0, m0, t0n);
                fma8_bcast<8>(U, 16 * j + 8, 0, m1, t1n);
              }
              pin8(U, 16 * j + 8 * h);
            }
          }
        }
      }
      // row k + 1 in its row group: its value after pivot k (its published
      // entries at the pair's columns were zero, so the loop left it as is)
      if (rg == (k >> 6)) {
        const int jj = (k & 63) >> 3;
#pragma clang loop unroll(full)
        for (int j = 0; j < 8; ++j)
          if (j == jj) U[8 * j + 2 * p + 1] = fma(s01, t0n, U[8 * j + 2 * p + 1]);
      }
      // publish rows k + 2 and k + 3 from their row group
      const int k2 = k + 2;
      if (k2 < C2 && rg == (k2 >> 6)) {
        const int jj = (k2 & 63) >> 3, np = par ^ 1;
        double v2 = 0.0, v3 = 0.0;
#pragma clang loop unroll(full)
        for (int j = 0; j < 8; ++j)
          if (j == jj) {
            v2 = U[8 * j + ((2 * p + 2) & 7)];
            v3 = U[8 * j + ((2 * p + 3) & 7)];
          }
        rowb[np][0][yl] = yl > k2 + 1 ? v2 : 0.0;
        rowb[np][1][yl] = yl > k2 + 1 ? v3 : 0.0;
        if (yl == k2) pivs[np][0] = v2;
        if (yl == k2 + 1) {
          pivs[np][1] = v2;
          pivs[np][2] = v3;
        }
      }
    }
  }
  __syncthreads();
  if (threadIdx.x < C2) dg[threadIdx.x] = 1.0 / sqrt(dg[threadIdx.x]);
  __syncthreads();
  // Z[x][e] = U[x][e] / sqrt(D_x) for this panel's externals
  const int e = pn * P2 + (yl - C2);
  if (yl >= C2 && e < E) {
    const lds_f64* is = opaque_lds<lds_f64>(&dg[0]);
    double* zc = z + (unsigned)e;
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      zc[(unsigned)((64 * rg + i) * zld)] = U[i] * is[64 * rg + i];
      if ((i & 15) == 15) __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// G' of the final step with more than 64 row inputs: G'[j][k] = sum_x
// Z[x][M + j] Z[x][k] (Z: T x (M + T) in scratch) on 64 x 64 tiles.
__global__ __launch_bounds__(256) void k_nd_gprod(NdArgs na) {
  __shared__ __attribute__((aligned(16))) double za[KC64 * KLD];
  __shared__ __attribute__((aligned(16))) double zb[KC64 * KLD];
  const int tid = threadIdx.x;
  const int M = na.ms.M, N = na.ms.N, T = na.T, Np = na.ms.Np, Mp = na.ms.Mp;
  const int ntx = (Np + 63) / 64, nty = (Mp + 63) / 64;
  const int64_t lin = nd_xcd(blockIdx.x, gridDim.x);   // an array's tiles share one L2
  const int64_t la = lin / (ntx * nty);
  const int tt = (int)(lin % (ntx * nty));
  const int j0 = (tt / nty) * 64, k0 = (tt % nty) * 64;
  const int zld = M + T;
  const double* z = na.scratch + la * na.scr_stride;
  MfmaTile mt;
  mt.init(tid);
  for (int x0 = 0; x0 < T; x0 += KC64) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int e = tid + 256 * rr, xx = e & 63, kk = e >> 6;
      const int x = x0 + kk;
      const int j = j0 + xx, k = k0 + xx;
      za[kk * KLD + xx] = (x < T && j < N) ? z[(int64_t)x * zld + M + j] : 0.0;
      zb[kk * KLD + xx] = (x < T && k < M) ? z[(int64_t)x * zld + k] : 0.0;
    }
    __syncthreads();
    mt.step(za, zb);
    __syncthreads();
  }
  float* out = nd_ref(na, la).out;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jb = 0; jb < 2; ++jb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int j = j0 + mt.row(i, v), k = k0 + mt.col(jb);
        if (j < Np && k < Mp) out[j * Mp + k] = (j < N && k < M) ? (float)mt.acc[i][jb][v] : 0.0f;
      }
}

// ---------------------------------------------------------------------------
// More than 128 cut nodes (the top merge and the final step of 256 x 256
// grids): the combined matrix [cut | externals] is written out dense
// (k_nd_dense0) and eliminated in stages of 64 pivots, each a k_nd_cut<64>
// (mode 2) over column panels followed by the Schur update of the rest
// (k_nd_dschur).  The last stage writes the merged block (or G').
// ---------------------------------------------------------------------------
// Entry (x, y) of a staged combined matrix lies in one of its dead ranges.
__device__ __forceinline__ bool dead_pair(const NdArgs& na, int x, int y) {
  return (x >= na.dead[0] && x < na.dead[1] && y >= na.dead[0] && y < na.dead[1]) ||
         (x >= na.dead[2] && x < na.dead[3] && y >= na.dead[2] && y < na.dead[3]);
}

// The whole 64 x 64 tile at (x, y) lies in one dead range (the ranges need
// not be tile-aligned: M is any row count).
__device__ __forceinline__ bool dead_tile(const NdArgs& na, int x, int y) {
  return dead_pair(na, x, y) && dead_pair(na, x + 63, y + 63) && dead_pair(na, x, y + 63);
}

// Dense combined matrix of one merge (rows in blocks of 16 per workgroup) or
// of the final step: [row inputs (T) | sources (M) | sinks (T)].  Only the
// 64 x 64 tiles on and below the diagonal are written: the stages read no
// others (the cut kernel reads the pivot columns as rows, k_nd_dschur the
// lower tiles).
template <bool FINAL>
__global__ __launch_bounds__(256) void k_nd_dense0(NdArgs na) {
  __shared__ __attribute__((aligned(16))) short invt[2][MAXSLOT2];
  const int n = na.dn, ld = na.dldo;
  const int nrb = (n + 15) / 16;
  const int64_t la = blockIdx.x / nrb;
  const int x0 = (int)(blockIdx.x % nrb) * 16;
  double* B = na.dB + la * na.out_stride;
  // the 16 rows share their lower tiles' column range [0, ylim); for a merge
  // 64 threads take an 8 x 8 block (lane l: row l % 8, column l / 8), so
  // that eight lanes read 64 contiguous bytes whichever mirror position of
  // the entry the child stores, and write 64 contiguous bytes of a row
  const int ylim = min(n, (x0 / 64 + 1) * 64), nyb = (ylim + 7) / 8;
  if constexpr (FINAL) {
    const int T = na.T, M = na.ms.M, Ein = 4 * T;
    const double* Y = na.buf_in + la * na.in_stride;
    // index -> port of the last level (-1: a source terminal)
    auto port = [&](int i) { return i < T ? i : (i < T + M ? -1 : T + (i - T - M)); };
    for (int x = x0; x < min(x0 + 16, n); ++x) {
      const int px = port(x);
      for (int y = threadIdx.x; y < ylim; y += 256) {
        if (dead_pair(na, x, y)) continue;
        const int py = port(y);
        double v = (px >= 0 && py >= 0) ? Y[sym_at(px, py, Ein)] : 0.0;
        if (x == y && (x < T || px < 0)) v += na.g_d;   // driver at the row input / source
        if (x < T && py < 0 && x == na.row_off + (y - T)) v -= na.g_d;
        if (y < T && px < 0 && y == na.row_off + (x - T)) v -= na.g_d;
        B[(int64_t)x * ld + y] = v;
      }
    }
  } else {
    const MergeGeom g = merge_geom(na, la);   // one merge per array at this level
    inverse_tables<MAXSLOT2>(na, g, invt, 256);
    const double* Y0 = na.buf_in + la * na.in_stride + (int64_t)g.cm0 * g.Ein * g.Ein;
    const double* Y1 = na.buf_in + la * na.in_stride + (int64_t)g.cm1 * g.Ein * g.Ein;
    for (int e = threadIdx.x; e < 2 * nyb * 64; e += 256) {
      const int x = x0 + 8 * (e / (nyb * 64)) + (e & 7), y = 8 * ((e >> 6) % nyb) + ((e >> 3) & 7);
      if (x >= n || y >= ylim || dead_pair(na, x, y)) continue;
      const int pa0 = invt[0][x], pa1 = invt[1][x];
      const int pb0 = invt[0][y], pb1 = invt[1][y];
      double v = 0.0;
      if (pa0 >= 0 && pb0 >= 0) v += Y0[sym_at(pa0, pb0, g.Ein)];
      if (pa1 >= 0 && pb1 >= 0) v += Y1[sym_at(pa1, pb1, g.Ein)];
      B[(int64_t)x * ld + y] = v;
    }
  }
}

// One stage's Schur update on a 64 x 64 tile: with Z (64 x E, E = dn - 64)
// of the stage's pivots, OUT 0 writes A[64 + x][64 + y] - (Z^T Z)[x][y] for
// x, y < E to dB (row stride dldo); OUT 1 writes G' = (Z^T Z - A) over the
// sink x source block (A: [sources (M) | sinks (T)] after the pivots).
// OUT 0 is symmetric: a workgroup computes and writes one tile of the lower
// triangle (tx >= ty); the tiles above are never read.
template <int OUT>
__global__ __launch_bounds__(256) void k_nd_dschur(NdArgs na) {
  __shared__ __attribute__((aligned(16))) double zab[2 * KC64 * KLD];
  double* za = zab;
  double* zb = zab + KC64 * KLD;
  const int tid = threadIdx.x;
  const int E = na.dn - 64;
  const int M = na.ms.M;
  const int nrx = OUT == 0 ? E : na.ms.Np, nry = OUT == 0 ? E : na.ms.Mp;
  const int ntx = (nrx + 63) / 64, nty = (nry + 63) / 64;
  const int ntiles = OUT == 0 ? ntx * (ntx + 1) / 2 : ntx * nty;
  const int64_t lin = nd_xcd(blockIdx.x, gridDim.x);   // an array's tiles share one L2
  const int64_t la = lin / ntiles;
  const int tt = (int)(lin % ntiles);
  int tx, ty;
  if (OUT == 0) {
    tri_tile(tt, &tx, &ty);
  } else {
    tx = tt / nty;
    ty = tt % nty;
  }
  const int x0 = tx * 64, y0 = ty * 64;
  // a tile wholly in a dead range (combined index = stage index + dld - dn
  // + 64) is neither read nor written
  if (OUT == 0 && dead_tile(na, na.dld - na.dn + 64 + x0, na.dld - na.dn + 64 + y0)) return;
  // rows of Z and of A behind this tile's x and y
  const int zx0 = OUT == 0 ? x0 : M + x0, zy0 = y0;
  const int lx = OUT == 0 ? E : min(na.ms.N, na.T), ly = OUT == 0 ? E : M;   // valid x, y
  const double* z = na.scratch + la * na.scr_stride;
  const double* A = na.dA + la * na.in_stride;
  MfmaTile mt;
  mt.init(tid);
  // this lane's entries of A behind the tile, loaded first so that they
  // arrive during the product (an entry outside the tile reads 0 without a
  // memory access)
  const __amdgpu_buffer_rsrc_t ra = nd_rsrc(A, (unsigned)(na.dn * na.dld * 8));
  const int N = na.ms.N;
  double av[2][2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int x = x0 + mt.row(i, v), y = y0 + mt.col(j);
        const bool in = OUT == 0 ? (x < E && y < E) : (x < N && y < M);
        const int row = OUT == 0 ? 64 + x : 64 + M + x;
        av[i][j][v] = nd_load(ra, in ? 8u * (unsigned)(row * na.dld + 64 + y) : kNdOob, 0);
      }
  // Z chunk by chunk (KC64 rows), software pipelined: the next chunk's loads
  // are in flight while this chunk is multiplied
  const __amdgpu_buffer_rsrc_t rz = nd_rsrc(z, (unsigned)(64 * E * 8));
  const int xl = tid & 63;
  const unsigned ox = x0 + xl < lx ? 8u * (unsigned)(zx0 + xl) : kNdOob;
  const unsigned oy = y0 + xl < ly ? 8u * (unsigned)(zy0 + xl) : kNdOob;
  auto load_chunk = [&](int k0, double (&pa)[4], double (&pb)[4]) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int kk = (tid >> 6) + 4 * r;   // uniform per wave
      const unsigned ko = (unsigned)__builtin_amdgcn_readfirstlane((k0 + kk) * E * 8);
      pa[r] = nd_load(rz, ox, ko);
      pb[r] = nd_load(rz, oy, ko);
    }
  };
  double pza[4], pzb[4];
  load_chunk(0, pza, pzb);
#pragma unroll 1
  for (int k0 = 0; k0 < 64; k0 += KC64) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int kk = (tid >> 6) + 4 * r;
      za[kk * KLD + xl] = pza[r];
      zb[kk * KLD + xl] = pzb[r];
    }
    __syncthreads();
    if (k0 + KC64 < 64) load_chunk(k0 + KC64, pza, pzb);
    mt.step(za, zb);
    __syncthreads();
  }
  if constexpr (OUT == 0) {
    double* B = na.dB + la * na.out_stride;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int x = x0 + mt.row(i, v), y = y0 + mt.col(j);
          if (x < E && y < E) B[(int64_t)x * na.dldo + y] = av[i][j][v] - mt.acc[i][j][v];
        }

  } else {
    const int Np = na.ms.Np, Mp = na.ms.Mp;
    float* out = nd_ref(na, la).out;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int jb = 0; jb < 2; ++jb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int j = x0 + mt.row(i, v), k = y0 + mt.col(jb);
          if (j >= Np || k >= Mp) continue;
          out[j * Mp + k] = (j < N && k < M) ? (float)(mt.acc[i][jb][v] - av[i][jb][v]) : 0.0f;
        }
  }
}

// ext = V - Z^T Z of one merge (V: the children's external-external
// entries).  ext is symmetric, so a workgroup computes and writes one 64 x 64
// tile of the lower triangle (tx >= ty); readers take the mirror of an entry
// above.
// Five waves per SIMD (96 VGPRs): its gathers need many waves in flight.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(5))) void k_nd_schur(NdArgs na) {
  __shared__ __attribute__((aligned(16))) short invt[2][MAXSLOT2];
  __shared__ __attribute__((aligned(16))) double zab[2 * KC64 * KLD];
  double* za = zab;
  double* zb = zab + KC64 * KLD;
  const int tid = threadIdx.x;
  const int nh = na.vert ? 2 * na.h : na.h, nw = na.vert ? na.w : 2 * na.w;
  const int Emax = 2 * (nh + nw);
  const int nt = (Emax + 63) / 64;
  const int ntri = nt * (nt + 1) / 2;
  const int64_t lin = nd_xcd(blockIdx.x, gridDim.x);
  const int64_t blk = lin / ntri;
  const MergeGeom g = merge_geom(na, blk);
  const int c = g.c, E = g.E;
  int tx, ty;
  tri_tile((int)(lin % ntri), &tx, &ty);
  const int x0 = tx * 64, y0 = ty * 64;
  const int nrx = min(64, E - x0), nry = min(64, E - y0);
  if (nrx <= 0 || nry <= 0) return;
  // at the bottom of the grid the B ports (the last nw) are sinks: entries
  // between two sinks are never read (sinks are never pivots, and G' is the
  // sink x source block), so tiles wholly among them are skipped
  if (g.i0 + nh == na.T && x0 >= E - nw && y0 >= E - nw) return;
  inverse_tables<MAXSLOT2>(na, g, invt, 256);
  const double* z = na.scratch + g.la * na.scr_stride + (int64_t)g.m * Emax * c;
  MfmaTile mt;
  mt.init(tid);
  // Z chunk by chunk (KC64 rows), software pipelined: the next chunk's loads
  // are in flight while this chunk is multiplied
  const __amdgpu_buffer_rsrc_t rz = nd_rsrc(z, (unsigned)(c * Emax * 8));
  const unsigned ox = 8u * (unsigned)(x0 + min(tid & 63, nrx - 1));
  const unsigned oy = 8u * (unsigned)(y0 + min(tid & 63, nry - 1));
  auto load_chunk = [&](int k0, double (&pa)[4], double (&pb)[4]) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int e = tid + 256 * r, xx = e & 63, kk = e >> 6;   // kk: uniform per wave
      const int k = min(k0 + kk, c - 1);
      const unsigned ko = (unsigned)__builtin_amdgcn_readfirstlane(k * Emax * 8);
      const double a = nd_load(rz, ox, ko);
      const double b = nd_load(rz, oy, ko);
      const bool ok = k0 + kk < c;
      pa[r] = (ok && xx < nrx) ? a : 0.0;
      pb[r] = (ok && xx < nry) ? b : 0.0;
    }
  };
  double pza[4], pzb[4];
  load_chunk(0, pza, pzb);
#pragma unroll 1
  for (int k0 = 0; k0 < c; k0 += KC64) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int e = tid + 256 * r, xx = e & 63, kk = e >> 6;
      za[kk * KLD + xx] = pza[r];
      zb[kk * KLD + xx] = pzb[r];
    }
    __syncthreads();
    if (k0 + KC64 < c) load_chunk(k0 + KC64, pza, pzb);
    mt.step(za, zb);
    __syncthreads();
  }
  // ext = V - Z^T Z, V the children's external entries: per block column,
  // this lane's 8 entries are loaded together, then written
  // an external port is a port of one child only, so an entry of V is one
  // child's entry (or none): one load per entry, over both children's
  // blocks of the level buffer
  const int cml = min(g.cm0, g.cm1);
  const unsigned e2 = (unsigned)(g.Ein * g.Ein);
  const unsigned o0 = (unsigned)(g.cm0 - cml) * e2, o1 = (unsigned)(g.cm1 - cml) * e2;
  const __amdgpu_buffer_rsrc_t ry =
      nd_rsrc(na.buf_in + g.la * na.in_stride + (int64_t)cml * e2,
              (unsigned)(abs(g.cm1 - g.cm0) + 1) * e2 * 8u);
  double* ext = na.buf_out + g.la * na.out_stride + (int64_t)g.m * Emax * Emax;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int y = y0 + mt.col(j);
    const int yy = min(y, E - 1);
    const int pb0 = invt[0][c + yy], pb1 = invt[1][c + yy];
    double vv[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int x = min(x0 + mt.row(i, v), E - 1);
        const int pa0 = invt[0][c + x], pa1 = invt[1][c + x];
        // an entry that no child holds reads 0 without a memory access
        const unsigned off = (pa0 >= 0 && pb0 >= 0) ? 8u * (o0 + (unsigned)sym_at(pa0, pb0, g.Ein))
                             : (pa1 >= 0 && pb1 >= 0) ? 8u * (o1 + (unsigned)sym_at(pa1, pb1, g.Ein))
                                                      : kNdOob;
        vv[i][v] = nd_load(ry, off, 0);
      }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int x = x0 + mt.row(i, v);
        if (x < E && y < E) ext[x * Emax + y] = vv[i][v] - mt.acc[i][j][v];
      }
  }
}

}  // namespace

// Side of the blocks the first kernel reduces (one wave per block).
int nd_block_side(int T, int64_t n_arrays) {
  (void)T;
  (void)n_arrays;
  return BS;
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

// Register elimination: cut sizes with an instantiation (powers of two up to
// 64) and at most 8 waves of columns.
static bool cut_in_registers(int c, int ncol) {
  return (c == 8 || c == 16 || c == 32 || c == 64) && ncol <= 512;
}

// Merges whose Schur update runs inside k_nd_cut (its kFuse path).
static bool schur_fused(int c, int emax) {
  return (c == 8 && emax <= 48) || (c == 16 && emax <= 96) || (c == 32 && emax <= 192);
}

template <bool FINAL>
static void launch_cut(const NdArgs& na, dim3 grid, int c, int ncol, bool fused, hipStream_t s) {
  // the final step's G' product and a fused Schur update have 256 work
  // items, one per thread: at least 256 threads then
  const dim3 blk((unsigned)std::max((ncol + 63) / 64 * 64, (FINAL || fused) ? 256 : 64));
  if constexpr (FINAL) {
    if (c == 16) hipLaunchKernelGGL((k_nd_cut<16, 1>), grid, blk, 0, s, na);
    else if (c == 32) hipLaunchKernelGGL((k_nd_cut<32, 1>), grid, blk, 0, s, na);
    else hipLaunchKernelGGL((k_nd_cut<64, 1>), grid, blk, 0, s, na);
  } else {
    if (c == 8) hipLaunchKernelGGL((k_nd_cut<8, 0>), grid, blk, 0, s, na);
    else if (c == 16) hipLaunchKernelGGL((k_nd_cut<16, 0>), grid, blk, 0, s, na);
    else if (c == 32) hipLaunchKernelGGL((k_nd_cut<32, 0>), grid, blk, 0, s, na);
    else hipLaunchKernelGGL((k_nd_cut<64, 0>), grid, blk, 0, s, na);
  }
}

// Staged elimination of a dense combined matrix of side n0 whose first c
// rows are the pivots (c / 64 stages, an even count): the matrix is built in
// `a`, the stages alternate between `a` and `b`, and the last stage writes
// the merged block to `a` with row stride ldo (FINAL: G' instead).  Both
// buffers hold in_stride (= out_stride) doubles per array.
template <bool FINAL>
static void launch_staged(NdArgs na, int64_t n, int c, int n0, double* a, double* b, int ldo,
                          hipStream_t s) {
  constexpr int PANEL = 448;   // external columns per cut workgroup (with 64 pivots: 512 lanes)
  // Entries between two sinks, or between two sources, are never read: G' is
  // the sink x source block, and sinks and sources are never pivots.  The
  // final step: [row inputs (T) | sources (M) | sinks (T)]; the merge of the
  // whole grid: [cut (c) | L (T) | B (T)], B the sinks.
  const int T = na.T;
  if (FINAL) {
    na.dead[0] = T;
    na.dead[1] = T + na.ms.M;
    na.dead[2] = T + na.ms.M;
    na.dead[3] = 2 * T + na.ms.M;
  } else {
    na.dead[0] = c + T;
    na.dead[1] = c + 2 * T;
    na.dead[2] = na.dead[3] = 0;
  }
  na.dB = a;
  na.dn = n0;
  na.dldo = n0;
  hipLaunchKernelGGL((k_nd_dense0<FINAL>), dim3((unsigned)(n * ((n0 + 15) / 16))), dim3(256), 0,
                     s, na);
  const int stages = c / 64;
  for (int st = 0; st < stages; ++st) {
    const bool last = st == stages - 1;
    na.dA = (st & 1) ? b : a;
    na.dB = (st & 1) ? a : b;
    na.dn = n0 - 64 * st;
    na.dld = n0;
    na.dldo = last ? ldo : n0;
    na.dpanel = PANEL;
    const int ext = na.dn - 64;
    const unsigned npan = (unsigned)((ext + PANEL - 1) / PANEL);
    const unsigned nthr = (unsigned)((64 + std::min(PANEL, ext) + 63) / 64 * 64);
    hipLaunchKernelGGL((k_nd_cut<64, 2>), dim3((unsigned)n * npan), dim3(nthr), 0, s, na);
    if (FINAL && last) {
      const unsigned nt = (unsigned)(((na.ms.Np + 63) / 64) * ((na.ms.Mp + 63) / 64));
      hipLaunchKernelGGL(k_nd_dschur<1>, dim3((unsigned)n * nt), dim3(256), 0, s, na);
    } else {
      const unsigned nt = (unsigned)((ext + 63) / 64);
      hipLaunchKernelGGL(k_nd_dschur<0>, dim3((unsigned)n * (nt * (nt + 1) / 2)), dim3(256), 0, s,
                         na);
    }
  }
}

// Builds G' of arrays [arr0, arr0 + n) with the workspace ws (ping-pong
// level buffers and scratch, sized by nd_sizes for one array, times n).
hipError_t launch_nd_build(const MapScalars& ms, const float* W, float* gpt, int64_t arr0,
                           int64_t n, int bs, double* ws, hipStream_t s, const NdBatch* batch) {
  NdArgs na{};
  na.ms = ms;
  na.W = W;
  na.gpt = gpt;
  na.batch = batch ? *batch : NdBatch{nullptr, nullptr};
  na.arr0 = arr0;
  na.n_arrays = n;
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
    // 16 x 16 regions: the kernel makes the levels up to 16 x 16
    hipLaunchKernelGGL(k_nd_block, dim3((unsigned)(n * nsb * nsb / 4)), dim3(64 * BWAVES), 0, s,
                       na);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  double* cur = bufA;
  double* nxt = bufB;
  // the block kernel made the 16 x 16 level
  int h = 2 * bs, w = 2 * bs;
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
    const dim3 grid((unsigned)(n * nmerge));
    {
      ProfScope prof("nd_merge", s);
      if (cut_in_registers(c, c + e_layout)) {
        const int emax = 2 * (nh + nw);
        // a fused Schur update runs in the merge's own workgroup; with fewer
        // merges than half the CUs its tiles are spread over k_nd_schur's
        // workgroups instead (the 64 x 64 conv layer: 229 -> 217 us)
        const bool few = (int64_t)n * nmerge < 128;
        const bool fused = schur_fused(c, emax) && !few;
        na.fuse = fused ? 1 : 0;
        // few merges: each one's columns in panels of 64 externals over
        // several workgroups (the cut block eliminated in each)
        constexpr int kPanel = 64;
        na.npan = few ? (e_layout + kPanel - 1) / kPanel : 1;
        na.dpanel = kPanel;
        launch_cut<false>(na, dim3((unsigned)(n * nmerge * na.npan)), c,
                          c + (few ? std::min(kPanel, e_layout) : e_layout), fused, s);
        na.npan = 1;
        if (!fused) {
          const int nt = (emax + 63) / 64;
          hipLaunchKernelGGL(k_nd_schur, dim3((unsigned)(n * nmerge * (nt * (nt + 1) / 2))),
                             dim3(256), 0, s, na);
        }
      } else if (c == C2) {
        const int emax = 2 * (nh + nw);
        const unsigned npan = (unsigned)((emax + P2 - 1) / P2);
        hipLaunchKernelGGL((k_nd_cut2<false>), dim3((unsigned)(n * nmerge) * npan), dim3(2 * CP2),
                           0, s, na);
        const int nt = (emax + 63) / 64;
        hipLaunchKernelGGL(k_nd_schur, dim3((unsigned)(n * nmerge * (nt * (nt + 1) / 2))),
                           dim3(256), 0, s, na);
      } else if (nmerge == 1 && c % 128 == 0 && (int64_t)(c + e_layout) * (c + e_layout) <= si &&
                 c + e_layout <= MAXSLOT2) {
        // the combined matrix in nxt, the stages in nxt / cur (the children
        // are dead once it is built), the merged block back in nxt
        launch_staged<false>(na, n, c, c + e_layout, nxt, cur, 2 * (nh + nw), s);
      } else {
        hipLaunchKernelGGL(k_nd_merge, grid, dim3(NTH),
                           (unsigned)((KB * KB + 2 * KB * 64) * sizeof(double)), s, na);
      }
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
    if (na.T <= 64 && cut_in_registers(na.T, 2 * na.T + ms.M)) {
      launch_cut<true>(na, dim3((unsigned)n), na.T, 2 * na.T + ms.M, false, s);
    } else if (na.T == C2) {
      hipLaunchKernelGGL((k_nd_cut2<true>), dim3((unsigned)n), dim3(2 * CP2), 0, s, na);
      const unsigned nt = (unsigned)(((ms.Np + 63) / 64) * ((ms.Mp + 63) / 64));
      hipLaunchKernelGGL(k_nd_gprod, dim3((unsigned)n * nt), dim3(256), 0, s, na);
    } else if (na.T % 128 == 0 && (int64_t)(2 * na.T + ms.M) * (2 * na.T + ms.M) <= si) {
      // the combined matrix in the free buffer, the stages in it and cur
      launch_staged<true>(na, n, na.T, 2 * na.T + ms.M, nxt, cur, 0, s);
    } else {
      hipLaunchKernelGGL(k_nd_final, dim3((unsigned)n), dim3(NTH),
                         (unsigned)((KB * KB + 2 * KB * 64) * sizeof(double)), s, na);
    }
  }
  return hipGetLastError();
}

}  // namespace rxnn
