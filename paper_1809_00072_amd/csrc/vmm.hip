// Evaluation phase of one layer (RxNN Sec. V-A "peripheral models", Eq. 14,
// Sec. VI): DAC -> I = V . G' per crossbar array -> ADC -> digital
// accumulation over row tiles, slices and the differential pair -> scale.
//
// One workgroup (4 waves) owns BM = 128 product rows and BN output columns of
// one column tile, and walks every row tile r of that column tile (or a
// contiguous share of them when the row tiles are split across workgroups).
// The work is a sequence of stages (r, pair of arrays, 64-input chunk):
//   * the DAC output V (BM x 64) of the chunk is staged in LDS: inputs are
//     quantised to a code and replaced by the DAC table entry (the table lives
//     in LDS).  For a convolution the inputs are gathered straight from the
//     NCHW tensor (patch column k = (ci kh + ky) kw + kx, patch row
//     bv = (n H_out + oy) W_out + ox, zero outside the image): the patch
//     matrix is never written to memory;
//   * both arrays' G'^T chunks (BN x 64) are staged in LDS;
//   * the global loads of stage s + 1 are issued into registers before the
//     MFMA loop of stage s, so they are in flight while it runs;
//   * v_mfma_f32_16x16x4f32 accumulates I for both arrays in fp32, the two
//     arrays sharing every V operand read;
//   * once the tile's M inputs are consumed, every current goes through the
//     ADC (a bucket table gives a code that is exact or one too low, one
//     comparison with the threshold table finishes it) and is added to an
//     int32 accumulator with the array's digital weight (+-2^(b_s s)).
// Integer accumulation makes the result independent of the order of row
// tiles and arrays, so splitting the row tiles over workgroups and combining
// with int32 atomics gives bit-identical results.
//
// K-order inside a 16-deep MFMA block: lane l in sub-step s multiplies the
// elements k = 4 (l / 16) + s of its row and column, so each lane fetches
// four consecutive k with one 16-byte LDS read for both operands.

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
  int c_in, h, w, kh, kw, stride, pad, ho, wo;
};

struct VmmArgs {
  MapScalars ms;
  PeriphScalars ps;
  ConvGeom cg;
  const float* gpt;
  const float* X;
  int64_t ldx, Bv;
  float* Y;
  int64_t hw_out;
  int32_t* iacc;
  float* dbg_I;
  int32_t* dbg_code;
  const int2* ktab;   // conv, kh kw <= 31: per (row tile, input) {byte offset, tap}
  int r_per_split;
};

__device__ __forceinline__ double bend(double u, double b) { return u - (b * u) * (1.0 - u); }

// bucket[b] = #{k : t_k <= (b - 1) w}: with w at most a quarter of the
// smallest threshold spacing, the exact code is bucket[b] or bucket[b] + 1.
__device__ __forceinline__ int adc_code(float I, const float* thr, const unsigned char* bucket,
                                        float inv_w, int nb) {
  const float t = I * inv_w;
  const int b = (int)fminf(fmaxf(t, 0.0f), (float)(nb - 1));
  const int c = bucket[b];
  return c + (I >= thr[c + 1] ? 1 : 0);
}

// CV: 0 fully connected; 1 convolution, patch columns decomposed in the
// kernel; 2 convolution, patch columns read from the per-layer table.
template <int BN, int CV, bool QADC, bool DEBUG>
__global__ __launch_bounds__(NTHR, 2) void k_xbar_vmm(VmmArgs va) {
  constexpr bool CONV = CV > 0;
  constexpr int NT = BN / 16;   // column fragments per wave
  constexpr int MT = 2;         // row fragments per wave (32 rows)
  constexpr int GV4 = BN / 8;   // float4 of G' staged per thread
  __shared__ __attribute__((aligned(16))) float Vs[BM * LDK];
  __shared__ __attribute__((aligned(16))) float Gs[2 * BN * LDK];
  __shared__ float lut[256];
  __shared__ float thr[258];
  __shared__ unsigned char bucket[kMaxBuckets];

  const MapScalars& ms = va.ms;
  const PeriphScalars& ps = va.ps;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, li = lane & 15;
  const int64_t b0 = (int64_t)blockIdx.x * BM;
  // column blocks: every block of a full column tile, and of the last tile
  // only those that hold real output columns (padded columns are discarded)
  const int nblk_per_tile = ms.Np / BN;
  const int c = min((int)blockIdx.y / nblk_per_tile, ms.C - 1);
  const int n0 = ((int)blockIdx.y - c * nblk_per_tile) * BN;
  const int r_begin = blockIdx.z * va.r_per_split;
  const int r_end = min(ms.R, r_begin + va.r_per_split);

  // ---- DAC and ADC tables (fp64 formulas, rounded to fp32) ----------------
  if (ps.dac_bits > 0) {
    const int L = ps.dac_levels;
    for (int k = tid; k <= L; k += NTHR)
      lut[k] = (float)(ps.v_read * bend((double)k / (double)L, ps.dac_bend));
  }
  if (QADC) {
    const int L = ps.adc_levels;
    for (int k = tid; k <= L + 1; k += NTHR) {
      float t;
      if (k == 0) t = -__builtin_inff();
      else if (k == L + 1) t = __builtin_inff();
      else t = (float)(ps.i_fs * bend(((double)k - 0.5) / (double)L, ps.adc_bend));
      thr[k] = t;
    }
    __syncthreads();
    for (int b = tid; b < ps.n_buckets; b += NTHR) {
      const double edge = (double)(b - 1) * ps.bucket_w;
      int lo = 0, hi = L;  // count of k in 1..L with thr[k] <= edge
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((double)thr[mid] <= edge) lo = mid; else hi = mid - 1;
      }
      bucket[b] = (unsigned char)lo;
    }
  }

  // ---- per-thread staging geometry ----------------------------------------
  // Staging loads are raw buffer loads: an SGPR descriptor, a 32-bit VGPR
  // offset and (FC) an SGPR offset per row step, so no 64-bit address is kept
  // per element.  Lanes whose element lies outside the input issue no load.
  // FC: lanes run along k (coalesced rows of X).  Conv: lanes run along the
  // product rows (consecutive output pixels), every wave shares one k.
  const int kk_fc = tid & 63, row_fc = tid >> 6;
  const int row_cv = tid & (BM - 1);
  const int kq_cv = __builtin_amdgcn_readfirstlane(tid >> 7);  // conv: first quad of 4 k
  int xrow_off = 0;          // conv: element offset of (img, iy0, ix0) from the WG base
  unsigned yok = 0, xok = 0;  // conv: bit ky (kx) set when that tap row (column) is inside the image
  unsigned tapbad = ~0u;     // table mode: bit ky kw + kx set when that tap is outside the image
                             // (bit 31, the table's code for a missing input, always set)
  __amdgpu_buffer_rsrc_t xsrc;
  int n_rows = (int)min((int64_t)BM, va.Bv - b0);
  if (CONV) {
    const int hw = va.cg.ho * va.cg.wo;
    const int64_t chw = (int64_t)va.cg.c_in * va.cg.h * va.cg.w;
    const int64_t img_first = b0 / hw;
    const int64_t img_last = (b0 + n_rows - 1) / hw;
    // table mode: the descriptor starts pad (w + 1) elements before the first
    // image, so that every lane's base offset is non-negative
    const int64_t shift = CV == 2 ? (int64_t)va.cg.pad * (va.cg.w + 1) : 0;
    xsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(va.X + img_first * chw - shift), (short)0,
                                             (int)(((img_last - img_first + 1) * chw + shift) * 4),
                                             0x00020000);
    if (row_cv < n_rows) {
      const int64_t bv = b0 + row_cv;
      const int64_t img = bv / hw;
      const int pix = (int)(bv - img * hw);
      const int oy = pix / va.cg.wo, ox = pix - oy * va.cg.wo;
      const int iy0 = oy * va.cg.stride - va.cg.pad;
      const int ix0 = ox * va.cg.stride - va.cg.pad;
      xrow_off = (int)((img - img_first) * chw) + iy0 * va.cg.w + ix0;
      for (int t = 0; t < va.cg.kh; ++t)
        if (iy0 + t >= 0 && iy0 + t < va.cg.h) yok |= 1u << t;
      for (int t = 0; t < va.cg.kw; ++t)
        if (ix0 + t >= 0 && ix0 + t < va.cg.w) xok |= 1u << t;
      if (CV == 2) {
        xrow_off = (xrow_off + (int)shift) * 4;   // byte offset from the shifted descriptor
        tapbad = 1u << 31;
        for (int ty = 0; ty < va.cg.kh; ++ty)
          for (int tx = 0; tx < va.cg.kw; ++tx)
            if (!((yok >> ty) & (xok >> tx) & 1u)) tapbad |= 1u << (ty * va.cg.kw + tx);
      }
    }
  } else {
    xsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(va.X + b0 * va.ldx), (short)0,
                                             (int)((int64_t)n_rows * va.ldx * 4), 0x00020000);
  }

  const int n_pairs = ms.A / 2;
  // Stages run over (row tile, pair, chunk).  Chunks that hold only padded
  // inputs (V = 0) are skipped: only the last row tile has them.
  const int nkc = (ms.Mp + KC - 1) / KC;
  const int nkc_last = min(nkc, (int)((ms.P - (int64_t)(ms.R - 1) * ms.M + KC - 1) / KC));
  const int per_r = n_pairs * nkc;
  const int n_stages = r_end == ms.R ? (r_end - 1 - r_begin) * per_r + n_pairs * nkc_last
                                     : (r_end - r_begin) * per_r;
  // stage s -> row tile r, pair ap, chunk kci of the nk chunks of r
  auto decode = [&](int s, int& r, int& ap, int& kci, int& nk) {
    const int rr = s / per_r;
    const int rem = s - rr * per_r;
    r = r_begin + rr;
    nk = r == ms.R - 1 ? nkc_last : nkc;
    ap = rem / nk;
    kci = rem - ap * nk;
  };
  const int tile_elems = ms.Np * ms.Mp;

  float xr[XPT];
  f32x4 gr[GV4];

  auto load_stage = [&](int s) {
    int r, ap, kci, nk;
    decode(s, r, ap, kci, nk);
    const int kc0 = kci * KC;
    if (ap == 0 || nk > 1) {
      if (CV == 2) {
        // this thread gathers k = 4 (kq_cv + 2 q) .. + 3, q = 0 .. 7, of its
        // pixel.  The table gives, per k, the byte offset of the input element
        // relative to the pixel's window (a scalar, the same for the wave) and
        // its tap; a tap outside the image (or code 31, no input) turns the
        // lane's offset out of range, so the load returns 0.
        const int2* kt = va.ktab + (int64_t)r * (nkc * KC) + kc0 + 4 * kq_cv;
#pragma unroll
        for (int q = 0; q < XPT / 4; ++q)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int2 e = kt[8 * q + j];
            const int voff = (int)((((tapbad >> e.y) & 1u) << 31) | (unsigned)xrow_off);
            xr[4 * q + j] = __builtin_bit_cast(float,
                __builtin_amdgcn_raw_buffer_load_b32(xsrc, voff, e.x, 0));
          }
      } else if (CONV) {
        // this thread gathers k = 4 (kq_cv + 2 q) .. + 3, q = 0 .. 7, of its
        // pixel.  The tap (ky, kx) and the input offset of k advance in scalar
        // registers (k is the same for the whole wave); an element outside the
        // image or beyond the layer's inputs gets an out-of-range buffer offset,
        // for which the load returns 0 without touching memory.
        const int khw = va.cg.kh * va.cg.kw, hw_in = va.cg.h * va.cg.w;
        const int kbase = r * ms.M + kc0;
        const int nvalid = min(ms.M - kc0, (int)ms.P - kbase);   // valid k of this chunk
        const int k0 = kbase + 4 * kq_cv;
        const int ci = k0 / khw;
        const int tap = k0 - ci * khw;
        int ky = tap / va.cg.kw, kx = tap - ky * va.cg.kw;
        int off = (ci * va.cg.h + ky) * va.cg.w + kx;
        auto step = [&]() {
          ++off;
          if (++kx == va.cg.kw) {
            kx = 0;
            off += va.cg.w - va.cg.kw;
            if (++ky == va.cg.kh) {
              ky = 0;
              off += hw_in - va.cg.kh * va.cg.w;
            }
          }
        };
#pragma unroll
        for (int q = 0; q < XPT / 4; ++q) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bool kok = 4 * (kq_cv + 2 * q) + j < nvalid;
            const bool ok = kok && (((yok >> ky) & (xok >> kx)) & 1);
            xr[4 * q + j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                xsrc, ok ? (xrow_off + off) * 4 : kOob, 0, 0));
            step();
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) step();   // the other half-wave group's quad
        }
      } else {
        // lanes along k; a lane beyond the layer's inputs gets an out-of-range
        // offset (the load returns 0), rows beyond the batch are skipped
        const int km = kc0 + kk_fc;
        const int p = r * ms.M + km;
        const bool kok = km < ms.M && p < (int)ms.P;
        const int voff = kok ? (int)((row_fc * va.ldx + p) * 4) : kOob;
#pragma unroll
        for (int it = 0; it < XPT; ++it) {
          float x = 0.0f;
          if (row_fc + 4 * it < n_rows)   // uniform over the wave
            x = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                              xsrc, voff, (int)(4 * it * va.ldx * 4), 0));
          xr[it] = x;
        }
      }
    }
    const int64_t arr0 = ((int64_t)c * ms.R + r) * ms.A + 2 * ap;
    __amdgpu_buffer_rsrc_t gsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(va.gpt + arr0 * tile_elems), (short)0, 2 * tile_elems * 4, 0x00020000);
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
  };

  auto dac = [&](float x) -> float {
    if (ps.dac_bits > 0) {
      const float t = rintf(x * ps.dac_s_in);
      const int code = (int)fminf(fmaxf(t, 0.0f), (float)ps.dac_levels);
      return lut[code];
    }
    return fmaxf(x, 0.0f) * ps.s_v_ideal;
  };

  auto store_stage = [&](int s) {
    int r, ap, kci, nk;
    decode(s, r, ap, kci, nk);
    if (ap == 0 || nk > 1) {
      if (CONV) {
#pragma unroll
        for (int q = 0; q < XPT / 4; ++q)
          *(f32x4*)&Vs[row_cv * LDK + 4 * (kq_cv + 2 * q)] =
              f32x4{dac(xr[4 * q]), dac(xr[4 * q + 1]), dac(xr[4 * q + 2]), dac(xr[4 * q + 3])};
      } else {
#pragma unroll
        for (int it = 0; it < XPT; ++it) Vs[(row_fc + 4 * it) * LDK + kk_fc] = dac(xr[it]);
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

  __syncthreads();
  if (n_stages > 0) load_stage(0);
  for (int s = 0; s < n_stages; ++s) {
    int r, ap, kci, nk;
    decode(s, r, ap, kci, nk);
    const int kc0 = kci * KC;
    __syncthreads();
    store_stage(s);
    __syncthreads();
    if (s + 1 < n_stages) load_stage(s + 1);
    if (kci == 0) {
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) acc[p][mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int kb_end = min(KC, ms.Mp - kc0);
    for (int kb = 0; kb < kb_end; kb += 16) {
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
#pragma unroll
        for (int ss = 0; ss < 4; ++ss)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
              acc[p][mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  af[mt][ss], bf[nt][ss], acc[p][mt][nt], 0, 0, 0);
      }
    }
    if (kci != nk - 1) continue;

    // ---- ADC and digital accumulation -------------------------------------
    const int wpos = 1 << (ms.slice_bits * ap);
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int wgt = p ? -wpos : wpos;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float I = acc[p][mt][nt][v];
            int code = 0;
            if (QADC) {
              code = adc_code(I, thr, bucket, ps.bucket_inv_w, ps.n_buckets);
              iacc[mt][nt][v] += wgt * code;
            } else {
              facc[mt][nt][v] += (float)wgt * I;
            }
            if (DEBUG) {
              const int64_t bv = b0 + wave * 32 + mt * 16 + 4 * g + v;
              const int n = n0 + nt * 16 + li;
              if (bv < va.Bv && n < ms.N) {
                const int64_t slot = (((int64_t)r * ms.C + c) * ms.A + 2 * ap + p) * va.Bv + bv;
                if (va.dbg_I) va.dbg_I[slot * ms.N + n] = I;
                if (va.dbg_code) va.dbg_code[slot * ms.N + n] = code;
              }
            }
          }
    }
  }

  // ---- output ---------------------------------------------------------------
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;
  float scale = 0.0f;
  if (wmax > 0.0) {
    const double s_w_eff = ms.sw_num / wmax;
    scale = QADC ? (float)(ps.lsb / (ps.s_v * s_w_eff)) : (float)(1.0 / (ps.s_v * s_w_eff));
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t bv = b0 + wave * 32 + mt * 16 + 4 * g + v;
        const int n = n0 + nt * 16 + li;
        const int64_t q = (int64_t)c * ms.N + n;
        if (bv >= va.Bv || n >= ms.N || q >= ms.Q) continue;
        if (va.iacc) {
          atomicAdd(&va.iacc[bv * ms.Q + q], iacc[mt][nt][v]);
          continue;
        }
        const float y = QADC ? (float)iacc[mt][nt][v] * scale : facc[mt][nt][v] * scale;
        if (va.hw_out > 0) {
          const int64_t img = bv / va.hw_out, pix = bv - img * va.hw_out;
          va.Y[(img * ms.Q + q) * va.hw_out + pix] = y;
        } else {
          va.Y[bv * ms.Q + q] = y;
        }
      }
}

template <typename IDX>
__global__ void k_finish(MapScalars ms, PeriphScalars ps, const int32_t* __restrict__ iacc,
                         IDX Bv, float* __restrict__ Y, IDX hw_out) {
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;
  float scale = 0.0f;
  if (wmax > 0.0) scale = (float)(ps.lsb / (ps.s_v * (ms.sw_num / wmax)));
  const IDX Q = (IDX)ms.Q;
  const IDX total = Bv * Q;
  for (IDX e = (IDX)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (IDX)gridDim.x * blockDim.x) {
    const IDX bv = e / Q, q = e - bv * Q;
    const float y = (float)iacc[e] * scale;
    if (hw_out > 0) {
      const IDX img = bv / hw_out, pix = bv - img * hw_out;
      Y[(img * Q + q) * hw_out + pix] = y;
    } else {
      Y[e] = y;
    }
  }
}

template <int BN, int CV, bool QADC>
hipError_t launch_t(const VmmArgs& va, dim3 grid, hipStream_t s, bool debug) {
  if (debug)
    hipLaunchKernelGGL((k_xbar_vmm<BN, CV, QADC, true>), grid, dim3(NTHR), 0, s, va);
  else
    hipLaunchKernelGGL((k_xbar_vmm<BN, CV, QADC, false>), grid, dim3(NTHR), 0, s, va);
  return hipGetLastError();
}

template <int BN>
hipError_t launch_bn(const VmmArgs& va, dim3 grid, hipStream_t s, int cv, bool qadc,
                     bool debug) {
  if (cv == 2) {
    return qadc ? launch_t<BN, 2, true>(va, grid, s, debug)
                : launch_t<BN, 2, false>(va, grid, s, debug);
  }
  if (cv == 1) {
    return qadc ? launch_t<BN, 1, true>(va, grid, s, debug)
                : launch_t<BN, 1, false>(va, grid, s, debug);
  }
  return qadc ? launch_t<BN, 0, true>(va, grid, s, debug)
              : launch_t<BN, 0, false>(va, grid, s, debug);
}

// Table of the patch columns of a convolution, per row tile r and tile input
// kk < nkc KC: {byte offset of input p = r M + kk relative to the window of
// an output pixel, tap ky kw + kx}; kk >= M or p >= P gets tap 31 (no input).
__global__ void k_conv_ktab(MapScalars ms, ConvGeom cg, int kcp, int2* tab) {
  const int64_t n = (int64_t)ms.R * kcp;
  const int khw = cg.kh * cg.kw;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(e / kcp), kk = (int)(e - (int64_t)r * kcp);
    const int64_t p = (int64_t)r * ms.M + kk;
    int2 v = make_int2(0, 31);
    if (kk < ms.M && p < ms.P) {
      const int ci = (int)(p / khw), tap = (int)(p - (int64_t)ci * khw);
      const int ky = tap / cg.kw, kx = tap - ky * cg.kw;
      v = make_int2(((ci * cg.h + ky) * cg.w + kx) * 4, tap);
    }
    tab[e] = v;
  }
}

int pick_bn(int Np) {
  if (Np % 64 == 0) return 64;
  if (Np % 32 == 0) return 32;
  return 16;
}

}  // namespace

int choose_splits(const MapScalars& ms, const PeriphScalars& ps, int64_t Bv) {
  if (ps.adc_bits == 0 || ms.R < 2) return 1;
  const int bn = pick_bn(ms.Np);
  const int64_t col_blocks = (int64_t)(ms.C - 1) * (ms.Np / bn) +
                             (ms.Q - (int64_t)(ms.C - 1) * ms.N + bn - 1) / bn;
  const int64_t blocks = ((Bv + BM - 1) / BM) * col_blocks;
  if (blocks >= 512) return 1;
  int64_t want = (1024 + blocks - 1) / blocks;
  if (want > ms.R) want = ms.R;
  const int per = (int)((ms.R + want - 1) / want);
  return (ms.R + per - 1) / per;
}

hipError_t launch_xbar_vmm(const MapScalars& ms, const PeriphScalars& ps, const float* gpt,
                           const VmmLaunch& vl, int splits, hipStream_t s) {
  VmmArgs va;
  va.ms = ms;
  va.ps = ps;
  va.cg = ConvGeom{0, 0, 0, 0, 0, 1, 0, 1, 1};
  if (vl.conv) {
    const rxnn_conv_desc& cd = *vl.conv;
    va.cg.c_in = cd.c_in;
    va.cg.h = cd.h;
    va.cg.w = cd.w;
    va.cg.kh = cd.kh;
    va.cg.kw = cd.kw;
    va.cg.stride = cd.stride;
    va.cg.pad = cd.pad;
    va.cg.ho = (cd.h + 2 * cd.pad - cd.kh) / cd.stride + 1;
    va.cg.wo = (cd.w + 2 * cd.pad - cd.kw) / cd.stride + 1;
  }
  va.gpt = gpt;
  va.X = vl.X;
  va.ldx = vl.ldx;
  va.Bv = vl.Bv;
  va.Y = vl.Y;
  va.hw_out = vl.hw_out;
  va.iacc = vl.iacc;
  va.dbg_I = vl.dbg_I;
  va.dbg_code = vl.dbg_code;
  va.r_per_split = (ms.R + splits - 1) / splits;
  const int bn = pick_bn(ms.Np);
  // the debug entry reports the currents of every column, padded ones included
  const bool debug = vl.dbg_I != nullptr || vl.dbg_code != nullptr;
  const int64_t q_last = ms.Q - (int64_t)(ms.C - 1) * ms.N;   // real columns of the last tile
  const int blk_last = debug ? ms.Np / bn : (int)((q_last + bn - 1) / bn);
  dim3 grid((unsigned)((vl.Bv + BM - 1) / BM), (unsigned)((ms.C - 1) * (ms.Np / bn) + blk_last),
            (unsigned)((ms.R + va.r_per_split - 1) / va.r_per_split));
  const bool qadc = ps.adc_bits > 0;
  const int cv = vl.conv == nullptr ? 0 : (vl.ktab ? 2 : 1);
  va.ktab = vl.ktab;
  if (bn == 64) return launch_bn<64>(va, grid, s, cv, qadc, debug);
  if (bn == 32) return launch_bn<32>(va, grid, s, cv, qadc, debug);
  return launch_bn<16>(va, grid, s, cv, qadc, debug);
}

int ktab_entries(const MapScalars& ms) { return ms.R * (((ms.Mp + KC - 1) / KC) * KC); }

hipError_t launch_conv_ktab(const MapScalars& ms, const rxnn_conv_desc& cd, int2* tab,
                            hipStream_t s) {
  ConvGeom cg{cd.c_in, cd.h, cd.w, cd.kh, cd.kw, cd.stride, cd.pad, 0, 0};
  const int kcp = ((ms.Mp + KC - 1) / KC) * KC;
  const int64_t n = (int64_t)ms.R * kcp;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(k_conv_ktab, dim3((unsigned)blocks), dim3(256), 0, s, ms, cg, kcp, tab);
  return hipGetLastError();
}

hipError_t launch_finish(const MapScalars& ms, const PeriphScalars& ps, const int32_t* iacc,
                         int64_t Bv, float* Y, int64_t hw_out, hipStream_t s) {
  int64_t blocks = (Bv * ms.Q + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  if (Bv * ms.Q < ((int64_t)1 << 31))
    hipLaunchKernelGGL(k_finish<int32_t>, dim3((unsigned)blocks), dim3(256), 0, s, ms, ps, iacc,
                       (int32_t)Bv, Y, (int32_t)hw_out);
  else
    hipLaunchKernelGGL(k_finish<int64_t>, dim3((unsigned)blocks), dim3(256), 0, s, ms, ps, iacc,
                       Bv, Y, hw_out);
  return hipGetLastError();
}

}  // namespace rxnn
