// Evaluation phase of one layer (RxNN Sec. V-A "peripheral models", Eq. 14,
// Sec. VI): DAC -> I = V . G' per crossbar array -> ADC -> digital
// accumulation over row tiles, slices and the differential pair -> scale.
//
// One workgroup (4 waves) owns BM = 128 product rows and BN output columns of
// one column tile, and walks every row tile r of that column tile (or a
// contiguous share of them when the row tiles are split across workgroups).
// For each row tile and each differential pair of arrays (+, -) of a slice:
//   * the DAC output V (BM x 64 chunk of the tile's M inputs) is staged in LDS:
//     inputs are read once per row tile, quantised to a code, and replaced by
//     the DAC table entry (the table lives in LDS);
//   * both arrays' G'^T chunks (BN x 64) are staged in LDS;
//   * v_mfma_f32_16x16x4f32 accumulates I for both arrays in fp32, the two
//     arrays sharing every V operand read;
//   * once the tile's M inputs are consumed, every current goes through the
//     ADC (a bucket table gives a code within one of the exact one, two
//     comparisons against the threshold table finish it) and is added to an
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

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct VmmArgs {
  MapScalars ms;
  PeriphScalars ps;
  const float* gpt;
  const void* X;
  int64_t ldx, Bv;
  float* Y;
  int64_t hw_out;
  int32_t* iacc;
  float* dbg_I;
  int32_t* dbg_code;
  int r_per_split;
};

__device__ __forceinline__ double bend(double u, double b) { return u - (b * u) * (1.0 - u); }

__device__ __forceinline__ int adc_code(float I, const float* thr, const unsigned char* bucket,
                                        float inv_w, int nb) {
  float t = I * inv_w;
  int b = (int)fminf(fmaxf(t, 0.0f), (float)(nb - 1));
  int c = bucket[b];
  int up = I >= thr[c + 1];
  int dn = I < thr[c];
  return c + up - dn;
}

template <int BN, bool CODES, bool QADC, bool DEBUG>
__global__ __launch_bounds__(NTHR, 2) void k_xbar_vmm(VmmArgs va) {
  constexpr int NT = BN / 16;   // column fragments per wave
  constexpr int MT = 2;         // row fragments per wave (32 rows)
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
  const int nblk_per_tile = ms.Np / BN;
  const int c = blockIdx.y / nblk_per_tile;
  const int n0 = (blockIdx.y % nblk_per_tile) * BN;
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
      const double edge = (double)b * ps.bucket_w;
      int lo = 0, hi = L;  // count of k in 1..L with thr[k] <= edge
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((double)thr[mid] <= edge) lo = mid; else hi = mid - 1;
      }
      bucket[b] = (unsigned char)lo;
    }
  }

  // ---- accumulators -----------------------------------------------------
  int32_t iacc[MT][NT][4];
  float facc[MT][NT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int v = 0; v < 4; ++v) { iacc[mt][nt][v] = 0; facc[mt][nt][v] = 0.0f; }

  const int n_pairs = ms.A / 2;
  const int64_t tile_elems = (int64_t)ms.Np * ms.Mp;
  const float* Xf = (const float*)va.X;
  const unsigned char* Xc = (const unsigned char*)va.X;

  for (int r = r_begin; r < r_end; ++r) {
    for (int ap = 0; ap < n_pairs; ++ap) {
      f32x4 acc[2][MT][NT];
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) acc[p][mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

      for (int kc0 = 0; kc0 < ms.Mp; kc0 += KC) {
        const bool stage_v = (ap == 0) || (ms.Mp > KC);
        __syncthreads();
        if (stage_v) {
          // V = DAC(x) for rows b0.., inputs r*M + kc0 + kk of this row tile
          for (int e = tid; e < BM * KC; e += NTHR) {
            const int row = e / KC, kk = e % KC;
            const int64_t bv = b0 + row;
            const int km = kc0 + kk;
            const int64_t p = (int64_t)r * ms.M + km;
            float v = 0.0f;
            if (bv < va.Bv && km < ms.M && p < ms.P) {
              if (CODES) {
                v = lut[Xc[bv * va.ldx + p]];
              } else {
                const float x = Xf[bv * va.ldx + p];
                if (ps.dac_bits > 0) {
                  const float t = rintf(x * ps.dac_s_in);
                  const int code = (int)fminf(fmaxf(t, 0.0f), (float)ps.dac_levels);
                  v = lut[code];
                } else {
                  v = fmaxf(x, 0.0f) * ps.s_v_ideal;
                }
              }
            }
            Vs[row * LDK + kk] = v;
          }
        }
        // G'^T chunks of arrays 2 ap and 2 ap + 1
        for (int e = tid; e < 2 * BN * KC; e += NTHR) {
          const int p = e / (BN * KC);
          const int rem = e % (BN * KC);
          const int n = rem / KC, kk = rem % KC;
          const int64_t arr = ((int64_t)c * ms.R + r) * ms.A + 2 * ap + p;
          float gv = 0.0f;
          if (kc0 + kk < ms.Mp) gv = va.gpt[arr * tile_elems + (int64_t)(n0 + n) * ms.Mp + kc0 + kk];
          Gs[(p * BN + n) * LDK + kk] = gv;
        }
        __syncthreads();

        const int kb_end = min(KC, ms.Mp - kc0);
        for (int kb = 0; kb < kb_end; kb += 16) {
          f32x4 af[MT], bf[2][NT];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            af[mt] = *(const f32x4*)&Vs[(wave * 32 + mt * 16 + li) * LDK + kb + 4 * g];
#pragma unroll
          for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
              bf[p][nt] = *(const f32x4*)&Gs[(p * BN + nt * 16 + li) * LDK + kb + 4 * g];
#pragma unroll
          for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
              for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                  acc[p][mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                      af[mt][s], bf[p][nt][s], acc[p][mt][nt], 0, 0, 0);
        }
      }

      // ---- ADC and digital accumulation -----------------------------------
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
          const int64_t img = bv / va.hw_out, pix = bv % va.hw_out;
          va.Y[(img * ms.Q + q) * va.hw_out + pix] = y;
        } else {
          va.Y[bv * ms.Q + q] = y;
        }
      }
}

__global__ void k_finish(MapScalars ms, PeriphScalars ps, const int32_t* __restrict__ iacc,
                         int64_t Bv, float* __restrict__ Y, int64_t hw_out) {
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;
  float scale = 0.0f;
  if (wmax > 0.0) scale = (float)(ps.lsb / (ps.s_v * (ms.sw_num / wmax)));
  const int64_t total = Bv * ms.Q;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t bv = e / ms.Q, q = e % ms.Q;
    const float y = (float)iacc[e] * scale;
    if (hw_out > 0) {
      const int64_t img = bv / hw_out, pix = bv % hw_out;
      Y[(img * ms.Q + q) * hw_out + pix] = y;
    } else {
      Y[e] = y;
    }
  }
}

template <int BN, bool CODES, bool QADC>
hipError_t launch_t(const VmmArgs& va, dim3 grid, hipStream_t s, bool debug) {
  if (debug)
    hipLaunchKernelGGL((k_xbar_vmm<BN, CODES, QADC, true>), grid, dim3(NTHR), 0, s, va);
  else
    hipLaunchKernelGGL((k_xbar_vmm<BN, CODES, QADC, false>), grid, dim3(NTHR), 0, s, va);
  return hipGetLastError();
}

template <int BN>
hipError_t launch_bn(const VmmArgs& va, dim3 grid, hipStream_t s, bool codes, bool qadc,
                     bool debug) {
  if (codes) {
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

}  // namespace

int choose_splits(const MapScalars& ms, const PeriphScalars& ps, int64_t Bv) {
  if (ps.adc_bits == 0 || ms.R < 2) return 1;
  const int64_t blocks = ((Bv + BM - 1) / BM) * (int64_t)ms.C * (ms.Np / pick_bn(ms.Np));
  if (blocks >= 1024) return 1;
  int64_t want = (1024 + blocks - 1) / blocks;
  if (want > ms.R) want = ms.R;
  // equal shares of row tiles
  const int per = (int)((ms.R + want - 1) / want);
  return (ms.R + per - 1) / per;
}

hipError_t launch_xbar_vmm(const MapScalars& ms, const PeriphScalars& ps, const float* gpt,
                           const VmmLaunch& vl, int splits, hipStream_t s) {
  VmmArgs va;
  va.ms = ms;
  va.ps = ps;
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
  dim3 grid((unsigned)((vl.Bv + BM - 1) / BM), (unsigned)(ms.C * (ms.Np / bn)),
            (unsigned)((ms.R + va.r_per_split - 1) / va.r_per_split));
  const bool qadc = ps.adc_bits > 0;
  const bool debug = vl.dbg_I != nullptr || vl.dbg_code != nullptr;
  if (bn == 64) return launch_bn<64>(va, grid, s, vl.x_codes, qadc, debug);
  if (bn == 32) return launch_bn<32>(va, grid, s, vl.x_codes, qadc, debug);
  return launch_bn<16>(va, grid, s, vl.x_codes, qadc, debug);
}

hipError_t launch_finish(const MapScalars& ms, const PeriphScalars& ps, const int32_t* iacc,
                         int64_t Bv, float* Y, int64_t hw_out, hipStream_t s) {
  int64_t blocks = (Bv * ms.Q + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_finish, dim3((unsigned)blocks), dim3(256), 0, s, ms, ps, iacc, Bv, Y,
                     hw_out);
  return hipGetLastError();
}

}  // namespace rxnn
