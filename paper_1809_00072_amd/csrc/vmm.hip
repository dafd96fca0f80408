// Evaluation phase of one layer (RxNN Sec. V-A "peripheral models", Eq. 14,
// Sec. VI): DAC -> I = V . G' per crossbar array -> ADC -> digital
// accumulation over row tiles, slices and the differential pair -> scale.
//
// Two kernels per call.
//
// k_dac converts every layer input once into its row voltage V (the DAC
// transfer table lives in LDS).  For a convolution it writes V into a
// zero-bordered copy of the NCHW input (pad pixels on every side), so the
// patch gather of the evaluation kernel needs no bounds tests: a padded pixel
// is input 0, whose DAC output is 0 V.
//
// k_xbar_vmm: one workgroup (4 waves) owns BM = 128 product rows and BN
// output columns of one column tile, and walks every row tile r of that
// column tile (or a contiguous share of them when the row tiles are split
// across workgroups).  The work is a sequence of stages (r, pair of arrays,
// 64-input chunk):
//   * the V chunk (BM x 64) is staged in LDS.  For a convolution the rows are
//     gathered from the padded V tensor (patch column k = (ci kh + ky) kw +
//     kx, patch row bv = (n H_out + oy) W_out + ox): a per-layer table gives
//     the offset of column k inside a pixel's window, which is the same for
//     the whole wave, so a gathered element costs one buffer load with a
//     scalar offset and no vector instruction; the patch matrix is never
//     written to memory;
//   * both arrays' G'^T chunks (BN x 64) are staged in LDS;
//   * the global loads of stage s + 1 are issued into registers before the
//     MFMA loop of stage s, so they are in flight while it runs;
//   * v_mfma_f32_16x16x4f32 accumulates I for both arrays in fp32, the two
//     arrays sharing every V operand read;
//   * once the tile's M inputs are consumed, every current goes through the
//     ADC: one LDS read of a bucket table gives the code at the bucket's
//     lower edge and the next threshold, one comparison finishes the code,
//     and the difference of the pair's codes is added to an int32
//     accumulator with the pair's digital weight 2^(b_s s).
// On gfx950 the fp32 matrix instructions and vector instructions of a SIMD
// do not overlap, so every vector instruction in the stage loop costs matrix
// time: the kernel keeps them to the ADC (about six per conversion) and a
// few per stage.
// Integer accumulation makes the result independent of the order of row
// tiles and arrays, so splitting the row tiles over workgroups and combining
// with int32 atomics gives bit-identical results.
// Tiles are numbered XCD-locally (consecutive tiles on one XCD and its L2),
// and 32 x 32 crossbars are walked in groups of 2 x 2 arrays, one 64 x 64
// tile with the ADC after each row tile's 32 inputs.
//
// K-order inside a 16-deep MFMA block: lane l in sub-step s multiplies the
// elements k = 4 (l / 16) + s of its row and column, so each lane fetches
// four consecutive k with one 16-byte LDS read for both operands.

#include <algorithm>

#include "common.h"

namespace rxnn {
namespace {

constexpr int BM = 128;       // product rows per workgroup
constexpr int KC = 64;        // inputs (k) staged per chunk
constexpr int LDK = KC + 4;   // LDS row stride in floats
constexpr int NTHR = 256;
constexpr int XPT = BM * KC / NTHR;  // V elements staged per thread
// Buffer offset of an element that is not loaded: at or beyond the end of every
// buffer (all are below 2^31 bytes), so the load returns 0 without a memory access.
constexpr int kOob = (int)0x80000000u;

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct ConvGeom {
  int c_in, h, w, kh, kw, stride, pad, ho, wo, hp, wp;   // hp, wp: padded input sides
};

// Tiles as the evaluation kernel walks them: the layer's own (R, C, M, N,
// Mp, Np), or, for 32 x 32 crossbars, groups of 2 x 2 arrays seen as one
// 64 x 64 tile (grouped mode).
struct TileGeo {
  int R, C, M, N, Mp, Np;
};

struct VmmArgs {
  MapScalars ms;
  TileGeo tg;
  PeriphScalars ps;
  ConvGeom cg;
  const float* gpt;
  const float* V;       // DAC output: FC Bv x ldx (zero past P); conv the padded NCHW tensor
  int64_t ldx, Bv;
  float* Y;
  int64_t hw_out;
  int32_t* iacc;
  float* dbg_I;
  int32_t* dbg_code;
  const int* ktab;      // conv: per (row tile, input) byte offset inside the window
  const float2* adc_tab;  // ADC bucket table, n_buckets + 2 entries (k_adc_table)
  const float* gload;   // divider DAC: row loads [C][R][A][Mp]
  FastDiv fd_hw, fd_wo; // conv: division by H_out W_out and by W_out (product rows < 2^31)
  int n_cb;             // column blocks (tiles along y)
  int workers;          // 0: one workgroup per tile; > 0: persistent workgroups
  int64_t dp_tiles;     // persistent: tiles [0, dp_tiles) are whole-tile work (direct
                        // writes); the rest is shared evenly by (tile, row tile) units
                        // accumulated with int32 atomics
};

__device__ __forceinline__ double bend(double u, double b) { return u - (b * u) * (1.0 - u); }

// Workgroups are dispatched to the 8 XCDs in turn (workgroup i of a grid of n
// to XCD i mod 8), and every XCD has its own L2.  This renumbering gives XCD x
// the contiguous range of n / 8 (+1) logical numbers that starts at
// x (n / 8) + min(x, n mod 8); it is a bijection of [0, n).
__device__ __forceinline__ int64_t xcd_local(int64_t i, int64_t n) {
  const int64_t q = n >> 3, r = n & 7, x = i & 7, j = i >> 3;
  return x * q + min(x, r) + j;
}

// Buffer descriptor of a workgroup-uniform range; readfirstlane keeps it in
// scalar registers (a descriptor the compiler cannot prove uniform costs a
// loop over the distinct values at every load).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const void* p, int64_t bytes) {
  const uint64_t a = (uint64_t)p;
  const uint64_t au = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(a >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((int)a);
  return __builtin_amdgcn_make_buffer_rsrc((void*)au, (short)0,
                                           __builtin_amdgcn_readfirstlane((int)bytes), 0x00020000);
}

// ---------------------------------------------------------------------------
// DAC of every layer input (Sec. IV-A 'Non-ideal DAC'): code =
// clamp(rint(x s_in), 0, L), V = fp32(v_read phi(code / L)); ideal: V =
// max(x, 0) v_read / x_max.  Convolution inputs go to the padded layout.
// ---------------------------------------------------------------------------
// n_out: rows Bv (FC; cg.c_in = P, cg.wp = row stride of V) or planes n c_in
// (convolution)
template <bool CONV>
__global__ __launch_bounds__(256) void k_dac(PeriphScalars ps, ConvGeom cg, FastDiv fd_wp,
                                             FastDiv fd_pp, const float* __restrict__ X,
                                             float* __restrict__ V, int64_t n_out) {
  __shared__ float lut[256];
  if (ps.dac_bits > 0) {
    const int L = ps.dac_levels;
    for (int k = threadIdx.x; k <= L; k += blockDim.x)
      lut[k] = (float)(ps.v_read * bend((double)k / (double)L, ps.dac_bend));
  }
  __syncthreads();
  // the divider DAC's voltage depends on the array a row feeds: the pass then
  // writes the code, which the evaluation kernel converts per array
  auto dac = [&](float x) -> float {
    if (ps.dac_bits > 0) {
      const float c = fminf(fmaxf(rintf(x * ps.dac_s_in), 0.0f), (float)ps.dac_levels);
      return ps.ldac ? c : lut[(int)c];
    }
    return fmaxf(x, 0.0f) * ps.s_v_ideal;
  };
  if (CONV) {
    // the threads stride over the whole padded tensor (every plane of every
    // image) eight elements at a time, so that their loads are in flight
    // together; plane, row and column by invariant-divisor multiplies
    // (the tensor holds fewer than 2^32 elements)
    const uint32_t plane_p = (uint32_t)(cg.hp * cg.wp);
    const uint32_t total = (uint32_t)(n_out * plane_p);
    const uint32_t stride = gridDim.x * blockDim.x;
    for (uint32_t e0 = blockIdx.x * blockDim.x + threadIdx.x; e0 < total; e0 += 8 * stride) {
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t e = e0 + j * stride;
        const uint32_t plane = div_by(e, fd_pp);
        const uint32_t rem = e - plane * plane_p;
        const int yp = (int)div_by(rem, fd_wp), xp = (int)rem - yp * cg.wp;
        const int iy = yp - cg.pad, ix = xp - cg.pad;
        x[j] = (e < total && iy >= 0 && iy < cg.h && ix >= 0 && ix < cg.w)
                   ? X[(size_t)plane * cg.h * cg.w + iy * cg.w + ix] : 0.0f;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (e0 + j * stride < total) V[e0 + j * stride] = dac(x[j]);
    }
  } else {
    // rows b over blockIdx.y: V[b][p] = DAC(X[b][p]) for p < P, 0 up to ldv
    const int P = cg.c_in, ldv = cg.wp;
    for (int64_t b = blockIdx.x; b < n_out; b += gridDim.x)
      for (int p = threadIdx.x; p < ldv; p += blockDim.x)
        V[b * ldv + p] = p < P ? dac(X[b * P + p]) : 0.0f;
  }
}

// ---------------------------------------------------------------------------
// ADC bucket table (Sec. IV-A 'Non-ideal ADC'; one workgroup).  Thresholds
// t_1 .. t_L = fp32(I_FS phi((k - 1/2) / L)) from the fp64 formula.  Entry b:
// c = #{k : t_k <= (b - 1) w} and t_{c+1}.  The bucket width w is at most
// 1 / 3.25 of the smallest threshold spacing: I / w rounded in fp32 lands in
// bucket floor(I / w) or a neighbour, which leaves at most one threshold
// between the entry's edge and I, so code(I) = c + (I >= t_{c+1}).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_adc_table(PeriphScalars ps, float2* __restrict__ tab) {
  __shared__ float thr[257];
  const int L = ps.adc_levels;
  for (int k = threadIdx.x; k <= L + 1; k += blockDim.x) {
    float t;
    if (k == 0) t = -__builtin_inff();
    else if (k == L + 1) t = __builtin_inff();
    else t = (float)(ps.i_fs * bend(((double)k - 0.5) / (double)L, ps.adc_bend));
    thr[k] = t;
  }
  __syncthreads();
  for (int b = threadIdx.x; b < ps.n_buckets + 2; b += blockDim.x) {
    const double edge = (double)(b - 1) * ps.bucket_w;
    int lo = 0, hi = L;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if ((double)thr[mid] <= edge) lo = mid; else hi = mid - 1;
    }
    tab[b] = make_float2(__int_as_float(lo), thr[lo + 1]);
  }
}

// LDAC (the load-dependent divider DAC): V holds codes c, and every array p of
// the pair converts them with its rows' loads, staged per chunk as
// h_p[k] = (g_pd + G_Load,p,k) L / (g_on V_DD):
//   V = c / (c / V_DD + h_p[k]) = V_DD g(c) / (g(c) + g_pd + G_Load).
// GRP (grouped mode, 32 x 32 crossbars): a tile of the walk is 64 x 64 and
// holds the arrays of row tiles 2 r, 2 r + 1 and column tiles 2 c, 2 c + 1;
// a stage stages all four arrays of each side of the pair, and the ADC runs
// after each physical row tile's 32 inputs.
template <int BN, bool CONV, bool QADC, bool DEBUG, bool LDAC, bool GRP>
__global__ __launch_bounds__(NTHR, 2) void k_xbar_vmm(VmmArgs va) {
  constexpr int NT = BN / 16;   // column fragments per wave
  constexpr int MT = 2;         // row fragments per wave (32 rows)
  constexpr int GV4 = BN / 8;   // float4 of G' staged per thread
  __shared__ __attribute__((aligned(16))) float Vs[BM * LDK];
  __shared__ __attribute__((aligned(16))) float Gs[2 * BN * LDK];
  __shared__ __attribute__((aligned(16))) float Hs[LDAC ? 2 * KC : 4];
  extern __shared__ float2 adct[];   // ADC table, n_buckets + 2 entries

  static_assert(!GRP || (BN == 64 && !DEBUG && !LDAC), "grouped mode: 64-wide blocks only");
  const MapScalars& ms = va.ms;
  const TileGeo& tg = va.tg;
  const PeriphScalars& ps = va.ps;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, li = lane & 15;
  const int nblk_per_tile = tg.Np / BN;

  // ---- ADC table (built by k_adc_table) -------------------------------------
  if (QADC) {
    for (int b = tid; b < ps.n_buckets + 2; b += NTHR) adct[b] = va.adc_tab[b];
  }

  const unsigned b_max = (unsigned)ps.n_buckets;
  auto adc = [&](float I) -> int {
    const unsigned b = min((unsigned)(I * ps.bucket_inv_w), b_max);
    const float2 e = adct[b];
    return __float_as_int(e.x) + (I >= e.y ? 1 : 0);
  };
  __syncthreads();

  // One tile: product rows [b0, b0 + BM) x columns [n0, n0 + BN) of column
  // tile c, row tiles [r_begin, r_end).
  auto run_tile = [&](int64_t b0_in, int c_in, int n0_in, int r_begin_in, int r_end_in,
                      bool atomic) __attribute__((always_inline)) {
  // the tile parameters are the same for the whole workgroup; readfirstlane
  // lets the compiler keep everything derived from them in scalar registers
  const int64_t b0 = (int64_t)__builtin_amdgcn_readfirstlane((int)(b0_in >> 32)) << 32 |
                     (uint32_t)__builtin_amdgcn_readfirstlane((int)b0_in);
  const int c = __builtin_amdgcn_readfirstlane(c_in);
  const int n0 = __builtin_amdgcn_readfirstlane(n0_in);
  const int r_begin = __builtin_amdgcn_readfirstlane(r_begin_in);
  const int r_end = __builtin_amdgcn_readfirstlane(r_end_in);
  // ---- per-thread staging geometry ----------------------------------------
  // Staging loads are raw buffer loads: an SGPR descriptor, a 32-bit VGPR
  // offset and an SGPR offset.  FC: lanes run along k (coalesced rows of V),
  // the SGPR offset steps the rows.  Conv: lanes run along the product rows
  // (consecutive output pixels) and every wave shares one k, whose window
  // offset is the SGPR offset.
  const int k4_fc = tid & 15, row_fc = tid >> 4;   // FC: 4 inputs of rows row_fc + 16 i
  const int row_cv = tid & (BM - 1);
  const int kq_cv = __builtin_amdgcn_readfirstlane(tid >> 7);  // conv: first quad of 4 k
  int xbase = 0;             // conv: byte offset of the pixel's window origin
  int fc_off[XPT / 4];       // FC: byte offsets of this thread's rows
  __amdgpu_buffer_rsrc_t xsrc;
  const int n_rows = (int)min((int64_t)BM, va.Bv - b0);
  if (CONV) {
    const int hw = va.cg.ho * va.cg.wo;
    const int64_t chw = (int64_t)va.cg.c_in * va.cg.hp * va.cg.wp;
    const int img_first = (int)div_by((uint32_t)b0, va.fd_hw);
    const int img_last = (int)div_by((uint32_t)(b0 + n_rows - 1), va.fd_hw);
    xsrc = uniform_rsrc(va.V + img_first * chw, (img_last - img_first + 1) * chw * 4);
    // rows past the batch read the last real row (their outputs are dropped)
    const int bv = (int)b0 + min(row_cv, n_rows - 1);
    const int img = (int)div_by((uint32_t)bv, va.fd_hw);
    const int pix = bv - img * hw;
    const int oy = (int)div_by((uint32_t)pix, va.fd_wo), ox = pix - oy * va.cg.wo;
    xbase = (int)(((int64_t)(img - img_first) * chw + (int64_t)oy * va.cg.stride * va.cg.wp +
                   (int64_t)ox * va.cg.stride) * 4);
  } else {
    xsrc = uniform_rsrc(va.V + b0 * va.ldx, (int64_t)n_rows * va.ldx * 4);
#pragma unroll
    for (int it = 0; it < XPT / 4; ++it)
      fc_off[it] = (int)(((row_fc + 16 * it) * va.ldx + 4 * k4_fc) * 4);
  }

  const int n_pairs = ms.A / 2;
  // Stages run over (row tile, pair, chunk).  Chunks that hold only padded
  // inputs (V = 0) are skipped: only the last row tile has them.
  const int nkc = (tg.Mp + KC - 1) / KC;
  const int nkc_last = min(nkc, (int)((ms.P - (int64_t)(tg.R - 1) * tg.M + KC - 1) / KC));
  const int per_r = n_pairs * nkc;
  const int n_stages = r_end == tg.R ? (r_end - 1 - r_begin) * per_r + n_pairs * nkc_last
                                     : (r_end - r_begin) * per_r;
  const int tile_elems = ms.Np * ms.Mp;
  // Stages in order: row tile r, then pair ap, then chunk kci of the nk
  // chunks of r (all workgroup-uniform).
  struct Stage {
    int r, ap, kci, nk;
  };
  auto first_stage = [&]() {
    return Stage{r_begin, 0, 0, r_begin == tg.R - 1 ? nkc_last : nkc};
  };
  auto next_stage = [&](Stage t) {
    if (++t.kci == t.nk) {
      t.kci = 0;
      if (++t.ap == n_pairs) {
        t.ap = 0;
        ++t.r;
        t.nk = t.r == tg.R - 1 ? nkc_last : nkc;
      }
    }
    return t;
  };
  (void)per_r;
  // G' staging: thread tid loads inputs 4 (tid % 16) .. + 3 of column
  // tid / 16 + 16 j of array p of the pair, j + p BN / 16 = it; only the
  // column and array move with it, so they go into the uniform offset
  const int goff_v = ((tid >> 4) * ms.Mp + 4 * (tid & 15)) * 4;
  // grouped mode (32 x 32 arrays of 1024 elements): input 4 (tid % 16) of the
  // group is in row tile 2 r + (tid % 16) / 8; that array sits A arrays after
  // the first row tile's
  const int goff_g = ((((tid & 15) >> 3) * ms.A * tile_elems) + (tid >> 4) * 32 +
                      4 * (tid & 7)) * 4;

  float xr[XPT];
  f32x4 gr[GV4];
  float hr = 0.0f;   // LDAC: the load of row kc0 + (tid % KC) of array tid / KC of the pair

  auto load_stage = [&](Stage st) {
    const int r = st.r, ap = st.ap, kci = st.kci, nk = st.nk;
    const int kc0 = kci * KC;
    if (ap == 0 || nk > 1) {
      if (CONV) {
        // this thread gathers k = 4 (kq_cv + 2 q) .. + 3, q = 0 .. 7, of its
        // pixel; table entries of missing inputs point at the window origin
        // and are zeroed when staged
        // the table is read-only for the kernel: reading it through the
        // constant address space gives scalar loads
        typedef const __attribute__((address_space(4))) int cint4;
        cint4* kt = (cint4*)(uintptr_t)(va.ktab + __builtin_amdgcn_readfirstlane(
                                                    r * (nkc * KC) + kc0 + 4 * kq_cv));
#pragma unroll
        for (int q = 0; q < XPT / 4; ++q)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            xr[4 * q + j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                xsrc, xbase, kt[8 * q + j], 0));
      } else {
        // 16 bytes per lane; V is zero past P, inputs past the tile's M meet
        // zero G' rows or G' loads past the tile; rows past the batch are
        // beyond the descriptor and read 0
        const int soff = __builtin_amdgcn_readfirstlane((r * tg.M + kc0) * 4);
#pragma unroll
        for (int it = 0; it < XPT / 4; ++it) {
          const f32x4 x4 = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
              xsrc, fc_off[it], soff, 0));
          xr[4 * it] = x4[0];
          xr[4 * it + 1] = x4[1];
          xr[4 * it + 2] = x4[2];
          xr[4 * it + 3] = x4[3];
        }
      }
    }
    if (GRP) {
      // the pair's arrays of row tiles 2 r, 2 r + 1 and column tiles 2 c,
      // 2 c + 1; a missing row or column tile (odd R or C) is read as zeros:
      // its lanes take the out-of-range offset in their own (VGPR) offset,
      // which the buffer's range check always covers
      const int64_t a0 = ((int64_t)(2 * c) * ms.R + 2 * r) * ms.A + 2 * ap;
      const int64_t left = ((int64_t)ms.C * ms.R * ms.A - a0) * tile_elems * 4;
      const __amdgpu_buffer_rsrc_t gq =
          uniform_rsrc(va.gpt + a0 * tile_elems, min(left, (int64_t)0x7fffffff));
      const bool row_absent = 2 * r + ((tid & 15) >> 3) >= ms.R;
#pragma unroll
      for (int it = 0; it < GV4; ++it) {
        const int p = it / 4, dc = (it % 4) >> 1, nb = 16 * (it & 1);
        const bool absent = row_absent || 2 * c + dc >= ms.C;
        const int soff = absent ? 0 : __builtin_amdgcn_readfirstlane(
            (((dc * ms.R * ms.A) + p) * tile_elems + nb * 32) * 4);
        gr[it] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
            gq, absent ? kOob : goff_g, soff, 0));
      }
      return;
    }
    const int64_t arr0 = ((int64_t)c * ms.R + r) * ms.A + 2 * ap;
    __amdgpu_buffer_rsrc_t gsrc = uniform_rsrc(va.gpt + arr0 * tile_elems, (int64_t)2 * tile_elems * 4);
    if (kc0 + KC <= ms.Mp) {
      // a full chunk: every load is inside the pair's G'
#pragma unroll
      for (int it = 0; it < GV4; ++it) {
        const int p = it / (BN / 16), nb = 16 * (it % (BN / 16));
        const int soff =
            __builtin_amdgcn_readfirstlane((p * tile_elems + (n0 + nb) * ms.Mp + kc0) * 4);
        gr[it] = __builtin_bit_cast(f32x4,
                                    __builtin_amdgcn_raw_buffer_load_b128(gsrc, goff_v, soff, 0));
      }
    } else {
#pragma unroll
      for (int it = 0; it < GV4; ++it) {
        const int e4 = tid + NTHR * it;
        const int p = e4 / (BN * (KC / 4));
        const int rm = e4 % (BN * (KC / 4));
        const int n = rm / (KC / 4), k4 = rm % (KC / 4);
        const int kidx = kc0 + 4 * k4;
        const int off = kidx < ms.Mp ? (p * tile_elems + (n0 + n) * ms.Mp + kidx) * 4 : kOob;
        gr[it] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(gsrc, off, 0, 0));
      }
    }
    if (LDAC && tid < 2 * KC) {
      const int kidx = kc0 + (tid & (KC - 1));
      hr = kidx < ms.Mp ? va.gload[(arr0 + (tid >> 6)) * ms.Mp + kidx] : 0.0f;
    }
  };

  auto store_stage = [&](Stage st) {
    const int r = st.r, ap = st.ap, kci = st.kci, nk = st.nk;
    if (ap == 0 || nk > 1) {
      if (CONV) {
        // inputs past the tile's or the layer's end are 0 (only in a chunk
        // that is not full, a uniform condition)
        const int kc0 = kci * KC;
        const int nvalid = min(tg.M - kc0, (int)(ms.P - (int64_t)r * tg.M) - kc0);
        if (nvalid < KC) {
#pragma unroll
          for (int q = 0; q < XPT / 4; ++q)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              if (4 * (kq_cv + 2 * q) + j >= nvalid) xr[4 * q + j] = 0.0f;
        }
#pragma unroll
        for (int q = 0; q < XPT / 4; ++q)
          *(f32x4*)&Vs[row_cv * LDK + 4 * (kq_cv + 2 * q)] =
              f32x4{xr[4 * q], xr[4 * q + 1], xr[4 * q + 2], xr[4 * q + 3]};
      } else {
#pragma unroll
        for (int it = 0; it < XPT / 4; ++it)
          *(f32x4*)&Vs[(row_fc + 16 * it) * LDK + 4 * k4_fc] =
              f32x4{xr[4 * it], xr[4 * it + 1], xr[4 * it + 2], xr[4 * it + 3]};
      }
    }
#pragma unroll
    for (int it = 0; it < GV4; ++it) {
      const int e4 = tid + NTHR * it;
      const int p = e4 / (BN * (KC / 4));
      const int rm = e4 % (BN * (KC / 4));
      const int n = rm / (KC / 4), k4 = rm % (KC / 4);
      *(f32x4*)&Gs[(p * BN + n) * LDK + 4 * k4] = gr[it];
    }
    if (LDAC && tid < 2 * KC) Hs[tid] = (ps.dac_gpd + hr) * ps.dac_hs;
  };

  // ---- accumulators -----------------------------------------------------
  int32_t iacc[MT][NT][4];
  float facc[MT][NT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int v = 0; v < 4; ++v) { iacc[mt][nt][v] = 0; facc[mt][nt][v] = 0.0f; }
  f32x4 acc[2][MT][NT];

  Stage cur = first_stage();
  if (n_stages > 0) load_stage(cur);
  for (int s = 0; s < n_stages; ++s) {
    const int r = cur.r, ap = cur.ap, kci = cur.kci, nk = cur.nk;
    const Stage nxt = next_stage(cur);
    const int kc0 = kci * KC;
    __syncthreads();
    store_stage(cur);
    __syncthreads();
    if (s + 1 < n_stages) load_stage(nxt);
    cur = nxt;
    auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) acc[p][mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    if (kci == 0) zero_acc();
    auto block = [&](int kb) {
      f32x4 af[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        af[mt] = *(const f32x4*)&Vs[(wave * 32 + mt * 16 + li) * LDK + kb + 4 * g];
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        f32x4 bf[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          bf[nt] = *(const f32x4*)&Gs[(p * BN + nt * 16 + li) * LDK + kb + 4 * g];
        f32x4 vf[MT];
        if (LDAC) {
          const f32x4 hv = *(const f32x4*)&Hs[p * KC + kb + 4 * g];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              vf[mt][j] = af[mt][j] *
                          __builtin_amdgcn_rcpf(__builtin_fmaf(af[mt][j], ps.dac_inv_vdd, hv[j]));
        } else {
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) vf[mt] = af[mt];
        }
#pragma unroll
        for (int ss = 0; ss < 4; ++ss)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
              acc[p][mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  vf[mt][ss], bf[nt][ss], acc[p][mt][nt], 0, 0, 0);
      }
    };
    // ---- ADC and digital accumulation (physical row tile rp) ----------------
    auto convert = [&](int rp) __attribute__((always_inline)) {
      const int sh = ms.slice_bits * ap;   // the pair's weight is +-2^sh
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float Ip = acc[0][mt][nt][v], In = acc[1][mt][nt][v];
            int cp = 0, cn = 0;
            if (QADC) {
              cp = adc(Ip);
              cn = adc(In);
              iacc[mt][nt][v] += (cp - cn) << sh;
            } else {
              facc[mt][nt][v] += (float)(1 << sh) * Ip;
              facc[mt][nt][v] += -(float)(1 << sh) * In;
            }
            if (DEBUG) {
              const int64_t bv = b0 + wave * 32 + mt * 16 + 4 * g + v;
              const int n = n0 + nt * 16 + li;
              if (bv < va.Bv && n < ms.N) {
                const int64_t slot = (((int64_t)rp * ms.C + c) * ms.A + 2 * ap) * va.Bv + bv;
                if (va.dbg_I) {
                  va.dbg_I[slot * ms.N + n] = Ip;
                  va.dbg_I[(slot + va.Bv) * ms.N + n] = In;
                }
                if (va.dbg_code) {
                  va.dbg_code[slot * ms.N + n] = cp;
                  va.dbg_code[(slot + va.Bv) * ms.N + n] = cn;
                }
              }
            }
          }
    };
    if (GRP) {
      // inputs 0 .. 31 belong to row tile 2 r, 32 .. 63 to row tile 2 r + 1
      // (absent when R is odd and r is the last)
      const int nh = 2 * r + 1 < ms.R ? 2 : 1;
#pragma unroll 1
      for (int h = 0; h < nh; ++h) {
        if (h) zero_acc();
        block(32 * h);
        block(32 * h + 16);
        convert(2 * r + h);
      }
      continue;
    }
    const int kb_end = min(KC, tg.Mp - kc0);
    for (int kb = 0; kb < kb_end; kb += 16) block(kb);
    if (kci != nk - 1) continue;
    convert(r);
}

  // ---- output ---------------------------------------------------------------
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;
  float scale = 0.0f;
  if (wmax > 0.0) {
    const double s_w_eff = ms.sw_num / wmax;
    scale = QADC ? (float)(ps.lsb / (ps.s_v * s_w_eff)) : (float)(1.0 / (ps.s_v * s_w_eff));
  }
  // Y is Bv x Q, or NCHW with H_out W_out = hw_out: the element of (bv, q)
  // is row_base(bv) + q times the column stride.  The int32 workspace is
  // Bv x Q (lanes along q: coalesced atomics).
  const int64_t qstride = va.hw_out > 0 ? va.hw_out : 1;
  if (CONV && !DEBUG && !atomic) {
    // NCHW output: a lane's results are 4 rows of one output channel, so a
    // direct store would scatter each instruction over 16 channels.  Each
    // wave passes its 32 x BN block through LDS (the V staging buffer, free
    // once every wave is past its last stage) and then writes 32
    // consecutive pixels of each channel per instruction.
    constexpr int TS = 33;   // LDS column stride of the transposed block
    static_assert(4 * BN * TS <= BM * LDK, "the transposed blocks fit the V buffer");
    __syncthreads();
    float* tb = Vs + wave * (BN * TS);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          tb[(nt * 16 + li) * TS + mt * 16 + 4 * g + v] =
              QADC ? (float)iacc[mt][nt][v] * scale : facc[mt][nt][v] * scale;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int row = lane & 31;
    const int64_t bv = b0 + wave * 32 + row;
    int64_t row_base = 0;
    if (bv < va.Bv) {
      const int img = (int)div_by((uint32_t)bv, va.fd_hw);   // hw_out = H_out W_out
      row_base = (int64_t)img * ms.Q * va.hw_out + (bv - (int64_t)img * va.hw_out);
    }
#pragma unroll 4
    for (int j = 0; j < BN / 2; ++j) {
      const int col = 2 * j + (lane >> 5);
      const int n = n0 + col;
      const int64_t q = (int64_t)c * tg.N + n;
      if (bv < va.Bv && n < tg.N && q < ms.Q) va.Y[row_base + q * qstride] = tb[col * TS + row];
    }
    return;
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t bv = b0 + wave * 32 + mt * 16 + 4 * g + v;
      if (bv >= va.Bv) continue;
      int64_t row_base;
      if (va.hw_out > 0) {
        const int img = (int)div_by((uint32_t)bv, va.fd_hw);   // hw_out = H_out W_out
        row_base = (int64_t)img * ms.Q * va.hw_out + (bv - (int64_t)img * va.hw_out);
      } else {
        row_base = bv * ms.Q;
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int n = n0 + nt * 16 + li;
        const int64_t q = (int64_t)c * tg.N + n;
        if (n >= tg.N || q >= ms.Q) continue;
        const int64_t e = row_base + q * qstride;
        if (atomic) {
          atomicAdd(&va.iacc[bv * ms.Q + q], iacc[mt][nt][v]);
        } else {
          va.Y[e] = QADC ? (float)iacc[mt][nt][v] * scale : facc[mt][nt][v] * scale;
        }
      }
    }
  };

  auto tile_at = [&](int bx, int cb, int r_begin, int r_end, bool atomic)
                     __attribute__((always_inline)) {
    // column blocks: every block of a full column tile, and of the last tile
    // only those that hold real output columns (padded columns are discarded)
    const int c = min(cb / nblk_per_tile, tg.C - 1);
    run_tile((int64_t)bx * BM, c, (cb - c * nblk_per_tile) * BN, r_begin, r_end, atomic);
  };
  // One workgroup per tile, or persistent workers: worker w first takes the
  // whole tiles w, w + W, ... below dp_tiles (the full rounds of the GPU), then
  // the units (tile, row tile) of the remaining tiles in the range
  // [U w / W, U (w + 1) / W) (tile-major), which may cover parts of tiles.
  // Tile and worker numbers are XCD-local (xcd_local): neighbouring tiles,
  // which share the halo rows of a convolution's input and, in a layer with
  // several column blocks, the same input rows, run on one XCD and its L2.
  int64_t u, u1, t_dp, dp_end;
  bool shared_units = false;
  if (va.workers == 0) {
    const int64_t lin = blockIdx.x + (int64_t)blockIdx.y * gridDim.x;
    u = xcd_local(lin, (int64_t)gridDim.x * gridDim.y) * tg.R;
    u1 = u + tg.R;
    t_dp = dp_end = 0;
  } else {
    const int64_t w = xcd_local(blockIdx.x, va.workers);
    const int64_t n_tiles = (int64_t)((va.Bv + BM - 1) / BM) * va.n_cb;
    const int64_t U = (n_tiles - va.dp_tiles) * tg.R;
    u = va.dp_tiles * tg.R + U * w / va.workers;
    u1 = va.dp_tiles * tg.R + U * (w + 1) / va.workers;
    t_dp = w;
    dp_end = va.dp_tiles;
    shared_units = true;
  }
  for (;;) {
    int64_t t;
    int r0, r1;
    bool atomic;
    if (t_dp < dp_end) {
      t = t_dp;
      r0 = 0;
      r1 = tg.R;
      atomic = false;
      t_dp += va.workers;
    } else if (u < u1) {
      t = u / tg.R;
      r0 = (int)(u - t * tg.R);
      r1 = (int)min((int64_t)tg.R, r0 + (u1 - u));
      atomic = shared_units;
      u += r1 - r0;
    } else {
      break;
    }
    tile_at((int)(t / va.n_cb), (int)(t % va.n_cb), r0, r1, atomic);
  }
}

// Y = fp32(acc) * scale_out from the Bv x Q int32 workspace: FC (Y has the
// same layout) elementwise.
__global__ __launch_bounds__(256) void k_finish(MapScalars ms, PeriphScalars ps,
                                                int32_t* __restrict__ iacc,
                                                float* __restrict__ Y, int64_t n) {
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;
  float scale = 0.0f;
  if (wmax > 0.0) scale = (float)(ps.lsb / (ps.s_v * (ms.sw_num / wmax)));
  const int64_t n4 = n >> 2;
  int4* a4 = reinterpret_cast<int4*>(iacc);
  float4* y4 = reinterpret_cast<float4*>(Y);
  const bool aligned = ((uintptr_t)Y & 15) == 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (aligned) {
    for (; e < n4; e += stride) {
      const int4 a = a4[e];
      a4[e] = make_int4(0, 0, 0, 0);   // the workspace is left zeroed for the next call
      y4[e] = make_float4((float)a.x * scale, (float)a.y * scale, (float)a.z * scale,
                          (float)a.w * scale);
    }
    e = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  }
  for (; e < n; e += stride) {
    Y[e] = (float)iacc[e] * scale;
    iacc[e] = 0;
  }
}

// Convolution: 64 x 64 blocks of the workspace go through LDS, so that both
// the Bv x Q reads and the NCHW writes are coalesced.
__global__ __launch_bounds__(256) void k_finish_nchw(MapScalars ms, PeriphScalars ps,
                                                     int32_t* __restrict__ iacc,
                                                     float* __restrict__ Y, int64_t row0,
                                                     int64_t Bv, int64_t hw, FastDiv fd_hw) {
  __shared__ int32_t tile[64][65];
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;
  float scale = 0.0f;
  if (wmax > 0.0) scale = (float)(ps.lsb / (ps.s_v * (ms.sw_num / wmax)));
  const int64_t bv0 = row0 + (int64_t)blockIdx.x * 64;
  const int64_t q0 = (int64_t)blockIdx.y * 64;
  const int t = threadIdx.x & 63, u = threadIdx.x >> 6;
  // all sixteen reads first (in flight together), then the zeroing writes
  int32_t v[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int i = u + 4 * j;
    v[j] = (bv0 + i < Bv && q0 + t < ms.Q) ? iacc[(bv0 + i) * ms.Q + q0 + t] : 0;
  }
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int i = u + 4 * j;
    tile[i][t] = v[j];
    if (bv0 + i < Bv && q0 + t < ms.Q) iacc[(bv0 + i) * ms.Q + q0 + t] = 0;   // left zeroed
  }
  __syncthreads();
  const int64_t bv = bv0 + t;
  if (bv >= Bv) return;
  const int64_t img = div_by((uint32_t)bv, fd_hw), pix = bv - img * hw;   // Bv < 2^31
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int i = u + 4 * j;
    if (q0 + i < ms.Q) Y[(img * ms.Q + q0 + i) * hw + pix] = (float)tile[t][i] * scale;
  }
}

// Table of the patch columns of a convolution, per row tile r of the walk
// (tg: a grouped tile spans two row tiles) and tile input kk < nkc KC: byte
// offset of input p = r M + kk inside an output pixel's window of the padded
// input; an input past the tile or the layer gets 0 (it is zeroed when
// staged).
__global__ void k_conv_ktab(MapScalars ms, TileGeo tg, ConvGeom cg, int kcp, int* tab) {
  const int64_t n = (int64_t)tg.R * kcp;
  const int khw = cg.kh * cg.kw;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(e / kcp), kk = (int)(e - (int64_t)r * kcp);
    const int64_t p = (int64_t)r * tg.M + kk;
    int v = 0;
    if (kk < tg.M && p < ms.P) {
      const int ci = (int)(p / khw), tap = (int)(p - (int64_t)ci * khw);
      const int ky = tap / cg.kw, kx = tap - ky * cg.kw;
      v = ((ci * cg.hp + ky) * cg.wp + kx) * 4;
    }
    tab[e] = v;
  }
}

// The ADC table is dynamic LDS (up to kMaxBuckets + 2 entries of 8 bytes);
// the limit is raised once per instantiation.
template <typename K>
hipError_t allow_adc_table(K kernel) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize,
                             (kMaxBuckets + 2) * (int)sizeof(float2));
}

template <int BN, bool CONV, bool QADC, bool DEBUG, bool LDAC, bool GRP = false>
hipError_t launch_one(const VmmArgs& va, dim3 grid, hipStream_t s) {
  auto kern = k_xbar_vmm<BN, CONV, QADC, DEBUG, LDAC, GRP>;
  static const hipError_t attr = allow_adc_table(kern);
  if (attr != hipSuccess) return attr;
  const size_t shm = QADC ? (size_t)(va.ps.n_buckets + 2) * sizeof(float2) : 0;
  hipLaunchKernelGGL(kern, grid, dim3(NTHR), shm, s, va);
  return hipGetLastError();
}

template <int BN, bool CONV, bool QADC>
hipError_t launch_t(const VmmArgs& va, dim3 grid, hipStream_t s, bool debug) {
  if (va.ps.ldac)
    return debug ? launch_one<BN, CONV, QADC, true, true>(va, grid, s)
                 : launch_one<BN, CONV, QADC, false, true>(va, grid, s);
  return debug ? launch_one<BN, CONV, QADC, true, false>(va, grid, s)
               : launch_one<BN, CONV, QADC, false, false>(va, grid, s);
}

template <int BN>
hipError_t launch_bn(const VmmArgs& va, dim3 grid, hipStream_t s, bool conv, bool qadc,
                     bool debug, bool grp) {
  if constexpr (BN == 64) {
    if (grp) {
      if (conv)
        return qadc ? launch_one<64, true, true, false, false, true>(va, grid, s)
                    : launch_one<64, true, false, false, false, true>(va, grid, s);
      return qadc ? launch_one<64, false, true, false, false, true>(va, grid, s)
                  : launch_one<64, false, false, false, false, true>(va, grid, s);
    }
  }
  if (conv) {
    return qadc ? launch_t<BN, true, true>(va, grid, s, debug)
                : launch_t<BN, true, false>(va, grid, s, debug);
  }
  return qadc ? launch_t<BN, false, true>(va, grid, s, debug)
              : launch_t<BN, false, false>(va, grid, s, debug);
}

int pick_bn(int Np) {
  if (Np % 64 == 0) return 64;
  if (Np % 32 == 0) return 32;
  return 16;
}

// Column blocks of the grid: every block of a full column tile, and of the
// last tile only those holding real outputs (all of them for the debug entry,
// which reports the padded columns' currents too).
int col_blocks(const MapScalars& ms, const TileGeo& tg, int bn, bool debug) {
  const int64_t q_last = ms.Q - (int64_t)(tg.C - 1) * tg.N;
  const int blk_last = debug ? tg.Np / bn : (int)((q_last + bn - 1) / bn);
  return (tg.C - 1) * (tg.Np / bn) + blk_last;
}

TileGeo tile_geo(const MapScalars& ms, bool grp) {
  if (grp) return TileGeo{(ms.R + 1) / 2, (ms.C + 1) / 2, 64, 64, 64, 64};
  return TileGeo{ms.R, ms.C, ms.M, ms.N, ms.Mp, ms.Np};
}

// Workgroups of the quantising evaluation kernel resident on the device at once.
template <int BN, bool CONV, bool LDAC, bool GRP = false>
int64_t slots_t(const PeriphScalars& ps) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  auto kern = k_xbar_vmm<BN, CONV, true, false, LDAC, GRP>;
  if (allow_adc_table(kern) != hipSuccess) return 0;
  const size_t shm = (size_t)(ps.n_buckets + 2) * sizeof(float2);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kern),
                                                   NTHR, shm) != hipSuccess)
    return 0;
  return (int64_t)cus * per_cu;
}

template <bool LDAC>
int64_t slots_l(int bn, bool conv, const PeriphScalars& ps) {
  if (bn == 64) return conv ? slots_t<64, true, LDAC>(ps) : slots_t<64, false, LDAC>(ps);
  if (bn == 32) return conv ? slots_t<32, true, LDAC>(ps) : slots_t<32, false, LDAC>(ps);
  return conv ? slots_t<16, true, LDAC>(ps) : slots_t<16, false, LDAC>(ps);
}

int64_t slots_for(int bn, bool conv, bool grp, const PeriphScalars& ps) {
  if (grp) return conv ? slots_t<64, true, false, true>(ps) : slots_t<64, false, false, true>(ps);
  return ps.ldac ? slots_l<true>(bn, conv, ps) : slots_l<false>(bn, conv, ps);
}

// Row loads of the arrays, fp64 sums over each array's stored columns (the
// padded storage columns are zero).  Workgroup (x, y): array x, rows
// 64 y .. 64 y + 63; its four waves take every fourth column and combine
// their partial sums in LDS.
__global__ __launch_bounds__(256) void k_gload(const float* __restrict__ gpt, int Np, int Mp,
                                               float* __restrict__ gload) {
  __shared__ double part[4][64];
  const int64_t arr = blockIdx.x;
  const int m = blockIdx.y * 64 + (threadIdx.x & 63), jq = threadIdx.x >> 6;
  double acc = 0.0;
  if (m < Mp) {
    const float* g = gpt + arr * ((int64_t)Np * Mp) + m;
#pragma unroll 4
    for (int j = jq; j < Np; j += 4) acc += (double)g[(int64_t)j * Mp];
  }
  part[jq][threadIdx.x & 63] = acc;
  __syncthreads();
  if (jq == 0 && m < Mp) {
    const int t = threadIdx.x;
    gload[arr * Mp + m] = (float)(((part[0][t] + part[1][t]) + part[2][t]) + part[3][t]);
  }
}

ConvGeom conv_geom(const rxnn_conv_desc& cd) {
  ConvGeom cg;
  cg.c_in = cd.c_in;
  cg.h = cd.h;
  cg.w = cd.w;
  cg.kh = cd.kh;
  cg.kw = cd.kw;
  cg.stride = cd.stride;
  cg.pad = cd.pad;
  cg.ho = (cd.h + 2 * cd.pad - cd.kh) / cd.stride + 1;
  cg.wo = (cd.w + 2 * cd.pad - cd.kw) / cd.stride + 1;
  cg.hp = cd.h + 2 * cd.pad;
  cg.wp = cd.w + 2 * cd.pad;
  return cg;
}

}  // namespace

// Grouped mode for 32 x 32 crossbars (not for the debug entry, whose
// per-array outputs follow the layer's own tiles, nor for the divider DAC).
bool use_groups(const MapScalars& ms, const PeriphScalars& ps, bool debug) {
  return ms.M == 32 && ms.N == 32 && ms.Mp == 32 && ms.Np == 32 && !ps.ldac && !debug;
}

VmmPlan vmm_plan(const MapScalars& ms, const PeriphScalars& ps, int64_t Bv, bool conv,
                 bool grp) {
  VmmPlan pl{0, 0, 0};
  const TileGeo tg = tile_geo(ms, grp);
  // fp32 accumulation (ideal ADC) keeps one workgroup per tile: a fixed order
  if (ps.adc_bits == 0 || tg.R < 2 || Bv <= 0) return pl;
  const int bn = pick_bn(tg.Np);
  const int n_cb = col_blocks(ms, tg, bn, false);
  const int64_t tiles = ((Bv + BM - 1) / BM) * n_cb;
  const int64_t slots = slots_for(bn, conv, grp, ps);
  if (slots <= 0) return pl;
  // one workgroup per tile fills the last round of the GPU only partly; when
  // that wastes more than 10 %, the full rounds stay whole-tile work and the
  // remaining tiles are shared evenly by (tile, row tile) units
  const int64_t rounds = (tiles + slots - 1) / slots;
  if ((double)tiles >= 0.9 * (double)(rounds * slots)) return pl;
  const int64_t dp = ((tiles / slots) * slots / n_cb) * n_cb;   // whole row blocks
  const int64_t units = (tiles - dp) * tg.R;
  pl.workers = (int)(units + dp < slots ? units + dp : slots);
  pl.dp_tiles = dp;
  pl.row0 = (dp / n_cb) * BM;
  return pl;
}

int64_t fc_ldv(const MapScalars& ms) {
  return ((int64_t)ms.R * ms.M + KC + 3) / 4 * 4;
}

int64_t dac_elems(const MapScalars& ms, const rxnn_conv_desc* conv, int64_t Bv) {
  if (!conv) return Bv * fc_ldv(ms);
  return (int64_t)conv->n * conv->c_in * (conv->h + 2 * conv->pad) * (conv->w + 2 * conv->pad);
}

hipError_t launch_dac(const MapScalars& ms, const PeriphScalars& ps,
                      const rxnn_conv_desc* conv, const float* X, int64_t Bv, float* V,
                      hipStream_t s) {
  if (Bv <= 0) return hipSuccess;
  if (conv) {
    const ConvGeom cg = conv_geom(*conv);
    const int64_t planes = (int64_t)conv->n * conv->c_in;
    const int64_t total = planes * cg.hp * cg.wp;
    if (total >= ((int64_t)1 << 32) - 8 * 256 * 2048) return hipErrorInvalidValue;
    const int64_t blocks = std::min<int64_t>(2048, (total + 8 * 256 - 1) / (8 * 256));
    hipLaunchKernelGGL(k_dac<true>, dim3((unsigned)std::max<int64_t>(1, blocks)), dim3(256), 0,
                       s, ps, cg, fast_div((uint32_t)cg.wp),
                       fast_div((uint32_t)(cg.hp * cg.wp)), X, V, planes);
  } else {
    ConvGeom cg{};
    cg.c_in = (int)ms.P;
    cg.wp = (int)fc_ldv(ms);
    hipLaunchKernelGGL(k_dac<false>, dim3((unsigned)(Bv < 8192 ? Bv : 8192)), dim3(256), 0, s,
                       ps, cg, FastDiv{1, 0, 0}, FastDiv{1, 0, 0}, X, V, Bv);
  }
  return hipGetLastError();
}

hipError_t launch_adc_table(const PeriphScalars& ps, float2* tab, hipStream_t s) {
  hipLaunchKernelGGL(k_adc_table, dim3(1), dim3(256), 0, s, ps, tab);
  return hipGetLastError();
}

hipError_t launch_xbar_vmm(const MapScalars& ms, const PeriphScalars& ps, const float* gpt,
                           const VmmLaunch& vl, const VmmPlan& plan, hipStream_t s) {
  const int workers = plan.workers;
  VmmArgs va;
  va.ms = ms;
  va.ps = ps;
  va.cg = vl.conv ? conv_geom(*vl.conv) : ConvGeom{0, 0, 0, 0, 0, 1, 0, 1, 1, 0, 0};
  va.gpt = gpt;
  va.V = vl.V;
  va.ldx = vl.ldx;
  va.Bv = vl.Bv;
  va.Y = vl.Y;
  va.hw_out = vl.hw_out;
  va.iacc = vl.iacc;
  va.dbg_I = vl.dbg_I;
  va.dbg_code = vl.dbg_code;
  va.ktab = vl.ktab;
  va.adc_tab = vl.adc_tab;
  va.gload = vl.gload;
  va.fd_hw = fast_div((uint32_t)(va.cg.ho * va.cg.wo));
  va.fd_wo = fast_div((uint32_t)va.cg.wo);
  const bool debug = vl.dbg_I != nullptr || vl.dbg_code != nullptr;
  va.tg = tile_geo(ms, vl.grp);
  const int bn = pick_bn(va.tg.Np);
  va.n_cb = col_blocks(ms, va.tg, bn, debug);
  va.workers = workers;
  va.dp_tiles = plan.dp_tiles;
  const dim3 grid = workers > 0 ? dim3((unsigned)workers)
                                : dim3((unsigned)((vl.Bv + BM - 1) / BM), (unsigned)va.n_cb);
  const bool qadc = ps.adc_bits > 0;
  const bool conv = vl.conv != nullptr;
  if (bn == 64) return launch_bn<64>(va, grid, s, conv, qadc, debug, vl.grp);
  if (bn == 32) return launch_bn<32>(va, grid, s, conv, qadc, debug, false);
  return launch_bn<16>(va, grid, s, conv, qadc, debug, false);
}

hipError_t launch_gload(const MapScalars& ms, const float* gpt, float* gload, hipStream_t s) {
  const int64_t n_arrays = (int64_t)ms.R * ms.C * ms.A;
  const dim3 grid((unsigned)n_arrays, (unsigned)((ms.Mp + 63) / 64));
  hipLaunchKernelGGL(k_gload, grid, dim3(256), 0, s, gpt, ms.Np, ms.Mp, gload);
  return hipGetLastError();
}

int ktab_entries(const MapScalars& ms, bool grp) {
  const TileGeo tg = tile_geo(ms, grp);
  return tg.R * (((tg.Mp + KC - 1) / KC) * KC);
}

hipError_t launch_conv_ktab(const MapScalars& ms, const rxnn_conv_desc& cd, bool grp, int* tab,
                            hipStream_t s) {
  const TileGeo tg = tile_geo(ms, grp);
  const int kcp = ((tg.Mp + KC - 1) / KC) * KC;
  const int64_t n = (int64_t)tg.R * kcp;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(k_conv_ktab, dim3((unsigned)blocks), dim3(256), 0, s, ms, tg, conv_geom(cd),
                     kcp, tab);
  return hipGetLastError();
}

hipError_t launch_finish(const MapScalars& ms, const PeriphScalars& ps, int32_t* iacc,
                         int64_t row0, int64_t Bv, float* Y, int64_t hw_out, hipStream_t s) {
  if (Bv <= row0) return hipSuccess;
  if (hw_out > 0) {
    const dim3 grid((unsigned)((Bv - row0 + 63) / 64), (unsigned)((ms.Q + 63) / 64));
    hipLaunchKernelGGL(k_finish_nchw, grid, dim3(256), 0, s, ms, ps, iacc, Y, row0, Bv, hw_out,
                       fast_div((uint32_t)hw_out));
    return hipGetLastError();
  }
  iacc += row0 * ms.Q;
  Y += row0 * ms.Q;
  const int64_t n = (Bv - row0) * ms.Q;
  int64_t blocks = (n / 4 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_finish, dim3((unsigned)blocks), dim3(256), 0, s, ms, ps, iacc, Y, n);
  return hipGetLastError();
}

}  // namespace rxnn
