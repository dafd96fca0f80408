/*
 * rxnn.h -- C ABI of the MI355X (gfx950) Fast Crossbar Model library.
 *
 * The library evaluates DNN layers on simulated resistive crossbars the way
 * the Fast Crossbar Model (FCM) of RxNN (arXiv 1809.00072) defines it:
 *
 *   phase 1, model generation (Sec. V-A, generator steps 1-3):
 *     the P x Q weight matrix is cut into M x N crossbar tiles (zero padded),
 *     every tile becomes one or more conductance arrays (a differential pair
 *     per weight slice), and every array's conductances G become the
 *     equivalent non-ideal conductance matrix G' of the resistive network
 *     with driver, wire and sense resistances (Sec. V-B, Eqs. 2-14).
 *   phase 2, evaluation (Sec. V-A "peripheral models", Eq. 14, Sec. VI):
 *     DAC transfer of the layer inputs, I = V . G' per array, ADC transfer
 *     and quantisation, and digital accumulation of the codes over row tiles,
 *     slices and the differential pair.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Device pointers are HIP device memory of the current device (e.g. the
 *   data_ptr() of a torch tensor on "cuda"); host pointers are ordinary host
 *   memory.  Every array is dense and row-major unless stated.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   Every call is asynchronous and stream ordered unless stated: the caller
 *   keeps its inputs alive and its outputs untouched until the stream has
 *   reached the call.
 * - Calls on one rxnn_layer are not thread safe and must be ordered on one
 *   stream: the layer owns a scratch workspace that its calls reuse.
 * - No exception crosses the ABI.  Arguments are validated before any launch;
 *   a failure returns a negative rxnn_status and leaves a message that
 *   rxnn_last_error() returns (per thread).  HIP failures map to RXNN_EHIP.
 *
 * Tile-local orientation (the reading of Eqs. 2-8): row 0 of a tile is the
 * paper's row 1, the row farthest from the sense amplifiers; column 0 is the
 * paper's column 1, the column nearest the row drivers.
 */
#ifndef RXNN_H
#define RXNN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RXNN_OK = 0,
  RXNN_EINVAL = -1,       /* an argument is out of range or inconsistent      */
  RXNN_ENOMEM = -2,       /* a device allocation failed                       */
  RXNN_EHIP = -3,         /* a HIP runtime call failed                        */
  RXNN_EUNSUPPORTED = -4  /* valid, but not supported by this library         */
} rxnn_status;

/* Opaque handle of one mapped layer: owns the tiled G' buffer on the device. */
typedef struct rxnn_layer rxnn_layer;

/*
 * Crossbar and device parameters (Sec. III, IV-A, V-A generator steps 1-2).
 *
 * rows, cols       crossbar size M x N, each 1..256.  Sizes above 64 need
 *                  r_row, r_col and r_sense > 0 (else RXNN_EUNSUPPORTED).
 * g_min, g_max     conductance range of one device in siemens, 0 < g_min < g_max.
 * r_driver         Thevenin resistance of each row driver (ohm, >= 0).  It sits
 *                  in series with the first row-wire segment, so the
 *                  load-dependent DAC output of Sec. IV-A is part of G'.
 * r_sense          sense resistance between each column's last node and the
 *                  virtual ground (ohm, >= 0).
 * r_row, r_col     resistance of one row-wire / column-wire segment (ohm, >= 0).
 * weight_bits      0: continuous conductances; else the magnitude |w| is
 *                  quantised to 2^weight_bits - 1 levels (1..16).
 * bits_per_slice   0: one slice of weight_bits bits; else the level is cut
 *                  into weight_bits / bits_per_slice slices of that many bits,
 *                  each on its own differential pair (shift-and-add).
 * w_max            |w| that maps to g_max; <= 0 means max|W| of the layer,
 *                  computed on the device at mapping time.
 * variation        device, fp32, one variation factor per device in the
 *                  layout [C][R][A][M][N] (tile column, tile row, array,
 *                  device row, device column; padded positions included), or
 *                  NULL.  Copied on `stream` at mapping time and kept by the
 *                  layer (a remap reuses it): every device's conductance is
 *                  multiplied by its factor (Sec. V-A generator step 2).
 * variation_sigma  with variation NULL: > 0 draws each device's factor as
 *                  max(0, 1 + variation_sigma z), z standard normal from
 *                  Philox-4x64-10 (counter (d, 0, 0, 0), key (variation_seed,
 *                  0), d = ((c R + r) A + a) M N + i N + j) and Box-Muller on
 *                  its first two words: u1 = ((x0 >> 11) + 1) 2^-53,
 *                  u2 = (x1 >> 11) 2^-53, z = sqrt(-2 ln u1) cos(2 pi u2).
 *                  0: no variation.  Sec. IV-B studies sigma / mu = 0.1.
 * variation_seed   key of the generated factors.
 * g_lut, g_lut_n   host, the device characteristic: g_lut_n (2..4096) samples
 *                  in [0, 1] of the normalised conductance (G - g_min) /
 *                  (g_max - g_min) at levels k / (g_lut_n - 1), linear in
 *                  between (copied).  NULL (g_lut_n 0): the linear device.
 *
 * Mapping of one weight w (fp64):
 *   continuous: G+ = g_min + s_w max(w,0), G- = g_min + s_w max(-w,0),
 *               s_w = (g_max - g_min) / w_max.
 *   quantised:  q = min(L_w, rint(|w| * (L_w / w_max))), L_w = 2^weight_bits - 1,
 *               slice s digit d_s = (q >> (b_s s)) & (2^b_s - 1); the side of
 *               sign(w) gets g_min + d_s dG, the other side g_min,
 *               dG = (g_max - g_min) / (2^b_s - 1).
 *   with g_lut: the level u = min(max(+-w, 0) / w_max, 1) (continuous) or
 *               d_s / (2^b_s - 1) (quantised) gives G = g_min + (g_max -
 *               g_min) f(u); the output scale keeps the linear device's s_w'.
 *   then every G is multiplied by its device's variation factor.
 * Arrays at one tile position are ordered a = 2 s + side (side 0 = positive,
 * slice 0 least significant); array a carries the digital weight
 * (side ? -1 : +1) * 2^(b_s s).  Zero-padded positions hold weight 0, i.e.
 * devices at g_min that still load the network.
 */
typedef struct {
  int32_t rows, cols;
  double g_min, g_max;
  double r_driver, r_sense, r_row, r_col;
  int32_t weight_bits;
  int32_t bits_per_slice;
  double w_max;
  const float* variation;
  double variation_sigma;
  uint64_t variation_seed;
  const double* g_lut;
  int32_t g_lut_n;
} rxnn_xbar_params;

/*
 * Peripheral (DAC / ADC) parameters (Sec. IV-A "non-ideal DAC", Sec. V-A
 * "peripheral models"; the curves are a stated reading of a figure that the
 * paper's text does not reproduce).  phi_b(u) = u - b u (1 - u).
 *
 * DAC (dac_bits 1..8): code c = clamp(rint(fp32(x) * s_in), 0, L) with
 *   s_in = fp32(L / x_max), L = 2^dac_bits - 1, one fp32 multiply rounded to
 *   nearest even; row voltage V = fp32(v_read * phi_{dac_bend}(c / L)).
 *   dac_bits = 0: ideal DAC, V = max(x, 0) * fp32(v_read / x_max).
 * ADC (adc_bits 1..8): I_FS = v_read * M * g_max, L = 2^adc_bits - 1,
 *   thresholds t_k = fp32(I_FS * phi_{adc_bend}((k - 1/2) / L)), k = 1..L;
 *   code = #{k : fp32(I) >= t_k}.  adc_bits = 0: ideal ADC (the current
 *   itself is accumulated).
 * x_max > 0, v_read > 0, 0 <= dac_bend < 1, |adc_bend| <= 0.5.
 *
 * Load-dependent DAC (the resistive divider of Sec. IV-A and Sec. V-A),
 * selected by dac_g_pd > 0: the DAC output node sits between the supply V_DD
 * through an input-dependent conductance g(c) = (c / L) dac_g_on and ground
 * through the pull-down dac_g_pd, and drives the row into the load G_Load,i =
 * sum_j G'_ij of the array it feeds (each array's rows see their own load):
 *   V_i = V_DD g(c_i) / (g(c_i) + dac_g_pd + G_Load,i),
 *   V_DD = v_read (dac_g_on + dac_g_pd) / dac_g_on (the unloaded DAC reaches
 *   v_read at full scale).
 * The divider stands in for the driver: the layer must have been mapped with
 * r_driver = 0 (RXNN_EINVAL otherwise).  Requires dac_bits > 0, dac_g_on > 0
 * and dac_bend = 0; the code c is the quantiser's above.  The evaluation
 * kernel converts codes to voltages per array in fp32 (one reciprocal per
 * element); the layer keeps the rows' loads (n_arrays x M floats, from the
 * stored G', recomputed after a remap).  dac_g_pd = 0 selects the static DAC
 * above and ignores dac_g_on.  Siemens; finite and >= 0.
 *
 * Output scale: with the quantising ADC, Y = fp32(acc) * fp32(LSB / (s_v s_w'))
 * where acc = sum over row tiles and arrays of weight(a) * code, LSB = I_FS / L,
 * s_v = v_read / x_max and s_w' = s_w (continuous) or dG L_w / w_max
 * (quantised).  With the ideal ADC, Y = sum weight(a) I / (s_v s_w').
 */
typedef struct {
  int32_t dac_bits;
  double x_max, v_read, dac_bend;
  int32_t adc_bits;
  double adc_bend;
  double dac_g_on, dac_g_pd;
} rxnn_periph_params;

/* Convolution shape: input NCHW n x c_in x h x w, weight c_out x c_in x kh x kw,
 * square stride and zero padding. */
typedef struct {
  int32_t n, c_in, h, w, c_out, kh, kw, stride, pad;
} rxnn_conv_desc;

/*
 * Phase 1, model generation (Sec. V-A generator steps 1-3; G -> G' is the
 * network of Sec. V-B solved exactly).
 *   params  host pointer, copied.
 *   W       device, fp32 P x Q row-major (P layer inputs, Q layer outputs),
 *           read on `stream`, not retained.  For torch.nn.Linear pass
 *           weight.t().contiguous(); for a conv pass weight.reshape(c_out,-1)
 *           transposed.
 *   out     receives the new handle; free it with rxnn_free_layer.
 * G' is built in fp64 and stored as fp32.  Returns RXNN_EINVAL for a bad
 * argument, RXNN_EUNSUPPORTED for sizes beyond the library's limits, RXNN_ENOMEM.
 */
rxnn_status rxnn_map_layer(const rxnn_xbar_params* params, const float* W,
                           int64_t P, int64_t Q, void* stream, rxnn_layer** out);

/*
 * Phase 1 again for new weights of the same shape: rebuilds every array's G'
 * of `layer` in place from W (device fp32 P x Q, as for rxnn_map_layer), with
 * the parameters the layer was mapped with (w_max recomputed from W when it
 * was not fixed).  Allocates nothing; stream ordered.  Used where the model
 * is regenerated every step (re-training with the crossbar in the loop).
 */
rxnn_status rxnn_remap_layer(rxnn_layer* layer, const float* W, void* stream);

/*
 * Phase 1 for several layers at once: rxnn_remap_layer of every layers[i]
 * from W[i] (device fp32, P_i x Q_i row-major, as for rxnn_map_layer), as one
 * launch sequence over the arrays of all of them, so that each level of the
 * G' build runs as one large grid (the per-level grids of one small layer
 * leave most of the GPU idle).  Same results as rxnn_remap_layer, bit for bit.
 *   layers  host array of n (>= 1) distinct live handles on one device, all
 *           mapped with the same crossbar size (rows, cols) and the same
 *           r_driver, r_sense, r_row and r_col, each of them > 0 for r_row,
 *           r_col and r_sense (the nested-dissection build); weights, sizes,
 *           w_max, slicing, device table and variation may differ.
 *   W       host array of n device pointers.
 * The library keeps, per device, the batch's layer, array and w_max-block
 * tables (copied from host memory on `stream`; every layer's w_max is
 * reduced in one pass) and one build workspace of at most 24 GiB,
 * grown on demand and held until the process ends; batches whose workspace
 * would exceed it are built in chunks.  Calls that overlap on one device
 * (different streams) race on these.  RXNN_EINVAL for a bad argument or a
 * mismatch, RXNN_ENOMEM when the tables or workspace cannot grow.
 */
rxnn_status rxnn_remap_layers(rxnn_layer* const* layers, const float* const* W, int32_t n,
                              void* stream);

/*
 * Phase 2 for a fully connected layer: DAC -> V . G' (Eq. 14) -> ADC ->
 * accumulation over row tiles and arrays -> scale.
 *   X  device fp32 B x P row-major; Y  device fp32 B x Q row-major.
 *   B >= 0 (B = 0 is a no-op).
 * The layer keeps a DAC output buffer (B x (R M + 64) floats) and, when the
 * evaluation is shared across persistent workgroups, an int32 B x Q
 * workspace; both grow on demand (RXNN_ENOMEM when they cannot).  It also
 * keeps the quantising ADC's bucket table (16 KiB, rebuilt on `stream` when
 * the peripheral parameters change).  Calls on one layer that overlap on
 * different streams race on these buffers.
 * RXNN_EUNSUPPORTED when P >= 2^22 (32-bit buffer offsets).
 */
rxnn_status rxnn_crossbar_vmm(const rxnn_layer* layer, const rxnn_periph_params* periph,
                              const float* X, int64_t B, float* Y, void* stream);

/*
 * rxnn_crossbar_vmm without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, kernels and results as
 * rxnn_crossbar_vmm (bit for bit).  Every evaluation buffer of the call (the
 * ADC bucket table, the divider DAC's row loads, the shared-tile int32
 * workspace and the DAC output) lives in one fixed device array of 64 MiB
 * that the library holds on each device it runs on until the process ends;
 * the call needs about 4 (B (R M + 64) + B Q) bytes plus the tables
 * (16 KiB; divider DAC: 4 R C A M bytes) and returns RXNN_EINVAL, launching
 * nothing, when that exceeds 64 MiB.  The tables are rebuilt and the
 * workspace cleared by kernels in every call (no memset nodes).  All calls on
 * one device share the array, which keeps the last call's contents: calls
 * that overlap on one device (different streams, threads or layers) race,
 * and must be ordered by the caller.
 */
rxnn_status rxnn_crossbar_vmm_noalloc(const rxnn_layer* layer, const rxnn_periph_params* periph,
                                      const float* X, int64_t B, float* Y, void* stream);

/*
 * Phase 2 for a convolution evaluated as a matrix product over unrolled
 * patches (Sec. VI): patch column k = (ci kh + ky) kw + kx, patch row
 * bv = (n H_out + oy) W_out + ox, padded pixels are 0.  The layer must have
 * been mapped with P = c_in kh kw and Q = c_out.
 *   X  device fp32 NCHW input; Y  device fp32 NCHW output n x c_out x H_out x W_out.
 * The patch matrix is never written: the layer keeps a DAC output buffer
 * (the input with pad zero pixels on every side), a table of patch-column
 * offsets (rebuilt when the geometry changes) and, as for the FC entry, an
 * int32 workspace when needed.  RXNN_EUNSUPPORTED when P >= 2^22, when
 * the padded images one 128-pixel block touches exceed 2 GiB, or when the
 * zero-bordered input holds 2^32 - 2^23 elements or more.
 */
rxnn_status rxnn_conv_layer(const rxnn_layer* layer, const rxnn_periph_params* periph,
                            const rxnn_conv_desc* conv, const float* X, float* Y,
                            void* stream);

/*
 * Backward pass of model-in-the-loop re-training (Sec. VI, re-training with
 * RxNN: crossbar forward pass, floating-point backward pass, data kept within
 * the range constraints).  The gradients flow through the layer's ideal fp32
 * weights with straight-through DAC and ADC; inputs the DAC clips and weights
 * beyond the layer's w_max get no gradient:
 *   dX = (dY W^T) * [0 <= x <= x_max]
 *   dW = clip(X, 0, x_max)^T dY * [|w| <= w_max]
 * where x_max is the periph's x_max for a quantising DAC and +inf for the
 * ideal one (which only drops negative inputs), and w_max is the one the
 * layer was mapped with.
 *   W   device fp32 P x Q row-major: the ideal weights the layer was mapped
 *       from (the same layout as for rxnn_map_layer).
 *   X   device fp32 forward input (FC: B x P row-major; conv: NCHW).
 *   dY  device fp32 gradient of the forward output (FC: B x Q; conv: NCHW
 *       n x c_out x H_out x W_out).
 *   dX  device fp32, the layout of X, overwritten; dW device fp32 P x Q,
 *       overwritten.  Either may be NULL to skip it.
 * All buffers are read and written on `stream`.  The two contractions run as
 * implicit GEMMs on the fp32 matrix cores: dW's gathers the clipped input
 * patches and the output gradient tile by tile, dX's gathers the output
 * gradient per kernel tap, so no unrolled patch matrix is formed.  An FC layer
 * runs as the 1 x 1 convolution of B images of 1 x 1 pixels.  When dW's
 * contraction over the Bv = n H_out W_out output pixels is split across
 * workgroups (at most 64 ranges, at most 2^24 floats of partial products), the
 * partials live in a layer-owned scratch buffer that grows on demand
 * (RXNN_ENOMEM when it cannot); calls on one layer that overlap on different
 * streams race on it.  Both sums are taken in fp32 in an order that differs
 * from a sequential one.  x_max enters the kernels rounded to fp32.
 * RXNN_EUNSUPPORTED when a pixel count, P, kh kw Q or an image's c_in H W
 * reaches 2^31 - 64, or a gradient has 2^24 tiles of 64 x 64 or more.
 * RXNN_EINVAL for bad arguments or a
 * convolution that does not match the layer; B = 0 or Bv = 0, or dX and dW
 * both NULL, is a no-op.
 */
rxnn_status rxnn_fc_backward(const rxnn_layer* layer, const rxnn_periph_params* periph,
                             const float* W, const float* X, const float* dY, int64_t B,
                             float* dX, float* dW, void* stream);
rxnn_status rxnn_conv_backward(const rxnn_layer* layer, const rxnn_periph_params* periph,
                               const rxnn_conv_desc* conv, const float* W, const float* X,
                               const float* dY, float* dX, float* dW, void* stream);

/*
 * Parity/debug exports.
 * rxnn_get_gprime copies the M x N fp32 G' of array `array` at tile
 *   (row_tile, col_tile) to host memory `host_out` (row-major, G'[i][j] = the
 *   column-j current for 1 V on row i).  It synchronises the device.
 * rxnn_set_gprime overwrites that array's G' from host memory (synchronous);
 *   for tests that feed a known G' to the evaluation kernels.
 * rxnn_vmm_debug runs rxnn_crossbar_vmm and also writes, for every row tile r,
 *   column tile c and array a, the fp32 pre-ADC currents and the ADC codes:
 *   I_preadc and codes are device buffers laid out [R][C][A][B][N] (either may
 *   be NULL).  Codes are 0 with the ideal ADC.
 * rxnn_layer_info returns P, Q, M, N, R, C, A (host pointer to 7 int64).
 * rxnn_layer_wmax returns the w_max the layer was mapped with (synchronises).
 */
rxnn_status rxnn_get_gprime(const rxnn_layer* layer, int64_t row_tile, int64_t col_tile,
                            int64_t array, float* host_out);
rxnn_status rxnn_set_gprime(rxnn_layer* layer, int64_t row_tile, int64_t col_tile,
                            int64_t array, const float* host_in);
rxnn_status rxnn_vmm_debug(const rxnn_layer* layer, const rxnn_periph_params* periph,
                           const float* X, int64_t B, float* Y, float* I_preadc,
                           int32_t* codes, void* stream);
rxnn_status rxnn_layer_info(const rxnn_layer* layer, int64_t* info7);
rxnn_status rxnn_layer_wmax(const rxnn_layer* layer, double* w_max);

/* Releases the handle and its device memory (synchronises its device).
 * NULL and already released handles are ignored. */
void rxnn_free_layer(rxnn_layer* layer);

/*
 * Kernel timing, for measurement.  rxnn_profile_enable(1): the library
 * brackets each kernel it launches with HIP events on the launch stream;
 * rxnn_profile_enable(2): only the evaluation kernel ("xbar_vmm"), which
 * keeps the other launches back to back (an event pair leaves the GPU idle
 * for several microseconds); 0 switches timing off, any other level is
 * RXNN_EINVAL.  The elapsed time is accumulated per kernel name: "wmax" (w_max reduction), "nd_block",
 * "nd_merge", "nd_final" (G' build by nested dissection), "gprime_sweep" (G'
 * build by the row sweep), "dac" (DAC of the inputs), "ktab" (patch-column
 * table), "xbar_vmm" (evaluation), "fill" (clearing of a new evaluation
 * workspace), "finish" (workspace of the shared tiles to Y, which also
 * leaves the workspace zeroed), "bw_dw", "bw_dx" (the backward pass's
 * contractions) and "bw_reduce" (the sum of dW's split partial products,
 * which counts 4 bytes per partial read, W read and dW written).  rxnn_profile_read synchronises, folds pending events
 * into the totals and returns total milliseconds and launch count.
 * rxnn_profile_bytes returns, for the same timed launches, the sum of their
 * algorithmic HBM bytes where the library counts them ("dac": 4 bytes per
 * input read plus 4 per DAC output written; "finish": 12 bytes per output it
 * converts, the int32 read, its zeroing and the fp32 write), else 0; divided
 * by rxnn_profile_read's time it is the kernel's achieved bandwidth.  Both
 * take a NUL-terminated kernel name and host output pointers (RXNN_EINVAL
 * when NULL).
 */
rxnn_status rxnn_profile_enable(int32_t on);
rxnn_status rxnn_profile_reset(void);
rxnn_status rxnn_profile_read(const char* kernel, double* total_ms, int64_t* count);
rxnn_status rxnn_profile_bytes(const char* kernel, double* bytes);

const char* rxnn_status_string(rxnn_status status);
const char* rxnn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RXNN_H */
