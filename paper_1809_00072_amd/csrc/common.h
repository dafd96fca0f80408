// Internal declarations shared by the HIP sources of librxnn (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/rxnn.h"

namespace rxnn {

constexpr uint64_t kLayerMagic = 0x52784e4e4c617972ull;  // "RxNNLayr"
constexpr int kMaxXbar = 256;       // largest crossbar side
constexpr int kMaxSweep = 64;       // largest side of the row-sweep build (zero resistances)
constexpr int kMaxBits = 8;         // largest DAC / ADC resolution
constexpr int kMaxBuckets = 2048;   // largest ADC bucket table (u8 entries)

// Scalars of one mapping, shared by the build, the evaluation and the finish
// kernels.  w_max is either fixed by the caller (wmax_fixed > 0) or reduced on
// the device into *d_wmax before the build runs.
struct MapScalars {
  int M, N, R, C, A, Mp, Np;   // crossbar, tile grid, arrays per position, padded tile
  int64_t P, Q;
  double g_min, g_max, r_driver, r_sense, r_row, r_col;
  int weight_bits, slice_bits, n_slices;
  float wmax_fixed;
  const float* d_wmax;
  double sw_num;               // s_w' = sw_num / w_max (siemens per unit weight)
  const float* vf;             // per-device variation factors [C][R][A][M][N] (or null)
  double vf_sigma;             // > 0 (vf null): generated factors N(1, vf_sigma^2)
  uint64_t vf_seed;
  const double* lut;           // device characteristic samples (or null: linear)
  int lut_n;
};

// Division by a launch-invariant divisor d >= 1 of any 32-bit n, by a
// multiply-high and a shift (Granlund and Montgomery, "Division by invariant
// integers using multiplication", PLDI 1994, Sec. 4): with l = ceil(log2 d)
// and m = floor(2^32 (2^l - d) / d) + 1, n / d = (mulhi(n, m) + n) >> l.
struct FastDiv {
  uint32_t d, m, l;
};

inline FastDiv fast_div(uint32_t d) {
  uint32_t l = 0;
  while (l < 32 && ((uint64_t)1 << l) < d) ++l;
  const uint64_t m = ((((uint64_t)1 << l) - d) << 32) / d + 1;
  return FastDiv{d, (uint32_t)m, l};
}

__device__ __forceinline__ uint32_t div_by(uint32_t n, FastDiv f) {
  return (uint32_t)(((uint64_t)__umulhi(n, f.m) + n) >> f.l);
}

// Peripheral constants prepared on the host from rxnn_periph_params; the
// per-code tables are rebuilt from them on the device.
struct PeriphScalars {
  int dac_bits, adc_bits;      // 0 = ideal
  int dac_levels, adc_levels;  // 2^bits - 1
  float dac_s_in;              // fp32(L / x_max)
  float s_v_ideal;             // fp32(v_read / x_max)
  double v_read, dac_bend, adc_bend;
  double i_fs;                 // ADC full scale, v_read * M * g_max
  double lsb;                  // i_fs / L
  double s_v;                  // v_read / x_max
  int n_buckets;               // ADC bucket table size
  float bucket_inv_w;          // fp32(n_buckets / i_fs)
  double bucket_w;             // i_fs / n_buckets
  // load-dependent divider DAC: V = c / (c / V_DD + (g_pd + G_Load) L / (g_on V_DD))
  int ldac;                    // 1: the DAC pass writes codes, the evaluation converts
  float dac_inv_vdd;           // fp32(1 / V_DD)
  float dac_hs;                // fp32(L / (g_on V_DD))
  float dac_gpd;               // fp32(g_pd)
};

}  // namespace rxnn

struct rxnn_layer {
  uint64_t magic;
  int device;
  rxnn_xbar_params params;
  rxnn::MapScalars ms;
  float* gpt;          // G' of every array, [C][R][A][Np][Mp] fp32, transposed per array
  float* d_wmax;       // [0] w_max; [1], [2] accumulator and ticket counter of its reduction
  void* ws;            // scratch of the evaluation calls
  size_t ws_bytes;
  bool ws_dirty;       // ws may hold non-zero words (new, or a call did not finish)
  double* nd_ws;       // nested-dissection build workspace (null: row sweep)
  int64_t nd_chunk;    // arrays built per pass over the workspace
  int nd_bs;           // side of the blocks reduced in LDS
  int* ktab;           // patch-column table of the last convolution geometry (or null)
  int64_t ktab_cap;    // entries allocated
  int ktab_key[7];     // c_in, h, w, kh, kw, pad, grouped walk the table was built for
  float* vbuf;         // DAC output of the current call (padded for a convolution)
  size_t vbuf_bytes;
  float* d_vf;         // the layer's copy of the variation factors (or null)
  double* d_lut;       // the layer's copy of the characteristic table (or null)
  float* bw_ws;        // backward-pass scratch (clipped inputs, patches, gradient rows)
  size_t bw_bytes;
  float* gload;        // row loads sum_j G'_ij per array, [C][R][A][Mp] (divider DAC), or null
  bool gload_valid;    // gload matches the stored G'
  float2* adct;        // ADC bucket table of the quantising evaluation (or null)
  double adct_key[5];  // adc_levels, n_buckets, i_fs, adc_bend, bucket_w it was built for
};

namespace rxnn {

// ---- launchers (each returns the hipError_t of its launch) -----------------

hipError_t launch_absmax(const float* W, int64_t n, unsigned* out, hipStream_t s);
hipError_t launch_fill_u32(unsigned* p, int64_t n, unsigned v, hipStream_t s);
hipError_t launch_gprime_build(const MapScalars& ms, const float* W, float* gpt,
                               hipStream_t s);
int nd_side(int M, int N);
int nd_block_side(int T, int64_t n_arrays);
void nd_sizes(int T, int M, int bs, int64_t* in_stride, int64_t* out_stride,
              int64_t* scr_stride);
// A build over the arrays of several layers that share the crossbar size and
// its resistances (one launch sequence for all of them): per layer its
// scalars, weights and G' buffer; per array of the batch, (layer, array).
struct NdBatchLayer {
  MapScalars ms;
  const float* W;
  float* gpt;
};
struct NdBatch {
  const NdBatchLayer* layers;   // device
  const int2* ent;              // device: batch array -> (layer slot, array of that layer)
};
hipError_t launch_nd_build(const MapScalars& ms, const float* W, float* gpt, int64_t arr0,
                           int64_t n, int bs, double* ws, hipStream_t s,
                           const NdBatch* batch = nullptr);
// blocks of the w_max reduction of n weights; w_max of every layer of a batch
// in two launches (layer l: blocks [start[l], start[l + 1]), start on the device)
int absmax_blocks(int64_t n);
hipError_t launch_absmax_batch(const NdBatchLayer* layers, const int* start, int n_layers,
                               int total_blocks, hipStream_t s);

struct VmmLaunch {
  const float* V;       // DAC output: FC Bv x ldx rows (ldx = fc_ldv); conv the padded NCHW tensor
  const rxnn_conv_desc* conv;  // null for FC
  int64_t ldx;          // row stride of X in elements (FC)
  int64_t Bv;           // rows of the product
  float* Y;
  int64_t hw_out;       // 0: Y is Bv x Q row-major; > 0: NCHW with H_out W_out = hw_out
  int32_t* iacc;        // split accumulation workspace (Bv x Q int32) or null
  float* dbg_I;         // [R][C][A][Bv][N] or null
  int32_t* dbg_code;    // [R][C][A][Bv][N] or null
  const int* ktab;      // conv: patch-column table
  const float* gload;   // divider DAC: row loads [C][R][A][Mp]
  bool grp;             // grouped mode (use_groups)
  const float2* adc_tab;  // quantising ADC: the bucket table of launch_adc_table
};
// Schedule of the evaluation kernel.  workers = 0: one workgroup per tile.
// workers > 0: persistent workgroups; tiles [0, dp_tiles) are whole-tile work,
// the rest (output rows [row0, Bv)) is shared by (tile, row tile) units that
// accumulate in the int32 workspace (zeroed first, converted by finish).
struct VmmPlan {
  int workers;
  int64_t dp_tiles;
  int64_t row0;
};
hipError_t launch_xbar_vmm(const MapScalars& ms, const PeriphScalars& ps, const float* gpt,
                           const VmmLaunch& vl, const VmmPlan& plan, hipStream_t s);
// grouped evaluation: 2 x 2 arrays of 32 x 32 crossbars walked as one 64 x 64
// tile (the patch-column table follows the walk)
bool use_groups(const MapScalars& ms, const PeriphScalars& ps, bool debug);
int ktab_entries(const MapScalars& ms, bool grp);
hipError_t launch_conv_ktab(const MapScalars& ms, const rxnn_conv_desc& cd, bool grp, int* tab,
                            hipStream_t s);
// DAC output: FC rows of fc_ldv(ms) floats (zero past P); conv the input with
// pad pixels on every side
int64_t fc_ldv(const MapScalars& ms);
// ADC bucket table of the quantising evaluation (n_buckets + 2 float2 entries)
hipError_t launch_adc_table(const PeriphScalars& ps, float2* tab, hipStream_t s);
int64_t dac_elems(const MapScalars& ms, const rxnn_conv_desc* conv, int64_t Bv);
hipError_t launch_dac(const MapScalars& ms, const PeriphScalars& ps,
                      const rxnn_conv_desc* conv, const float* X, int64_t Bv, float* V,
                      hipStream_t s);
hipError_t launch_finish(const MapScalars& ms, const PeriphScalars& ps, int32_t* iacc,
                         int64_t row0, int64_t Bv, float* Y, int64_t hw_out, hipStream_t s);
VmmPlan vmm_plan(const MapScalars& ms, const PeriphScalars& ps, int64_t Bv, bool conv,
                 bool grp);
// row loads of every array: gload[arr][m] = sum over columns of G'[arr][m][.]
hipError_t launch_gload(const MapScalars& ms, const float* gpt, float* gload, hipStream_t s);

// backward pass of re-training (backward.hip): implicit-GEMM kernels on the
// fp32 matrix cores; a fully connected layer is the 1 x 1 convolution of
// B images of 1 x 1 pixels.  dW's contraction over the output pixels is split
// into `nsplit` ranges (of `kc` pixels for the generic kernel; kc = 0 selects
// the 3 x 3 kernel, which splits whole 64-pixel chunks); with nsplit > 1 the
// partial products (nsplit P Q floats) are summed and masked by
// launch_bw_reduce_w.  vec_ok: X, dY and W are 16-byte aligned.
struct BwPlan {
  int nsplit, kc;
};
BwPlan bw_plan(const rxnn_conv_desc& cd, int P, int Q, bool vec_ok);
hipError_t launch_bw_dw(const rxnn_conv_desc& cd, int P, int Q, float x_max, const float* X,
                        const float* dY, const float* W, const MapScalars& ms, const BwPlan& plan,
                        float* out, hipStream_t s);
hipError_t launch_bw_dx(const rxnn_conv_desc& cd, int P, int Q, float x_max, const float* X,
                        const float* dY, const float* W, float* dX, hipStream_t s);
hipError_t launch_bw_reduce_w(const float* part, int nparts, const float* W, int64_t n,
                              const MapScalars& ms, float* dW, hipStream_t s);

// ---- kernel timing (api.hip) ------------------------------------------------
// `bytes`: the launch's algorithmic HBM bytes, summed per kernel name for the
// achieved bandwidth of memory-bound kernels (0 where it is not counted).
struct ProfScope {
  ProfScope(const char* name, hipStream_t s, double bytes = 0.0);
  ~ProfScope();
  const char* name_;
  hipStream_t s_;
  double bytes_;
  hipEvent_t a_, b_;
  bool on_;
};

}  // namespace rxnn
