// C ABI of librxnn: argument validation, layer handles, workspaces, launches
// and optional kernel timing.  The kernels live in gprime.hip (model
// generation) and vmm.hip (evaluation, with the convolution's patch gather).

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <set>
#include <string>
#include <vector>

#include "common.h"

using namespace rxnn;

// Fixed scratch of rxnn_crossbar_vmm_noalloc: every evaluation buffer of a
// call (ADC table, row loads, shared-tile workspace, DAC output) is carved
// out of this array, so the entry point allocates nothing.  Each device the
// library runs on holds its own copy until the process ends.  Host code must
// not pass the array's name to a kernel: its device address comes from
// hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

thread_local std::string g_err;
std::mutex g_mu;
std::set<const rxnn_layer*> g_live;

rxnn_status fail(rxnn_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
rxnn_status fail(rxnn_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_TRY(expr)                                                                        \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess)                                                                    \
      return fail(RXNN_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));                 \
  } while (0)

bool finite_nonneg(double v) { return isfinite(v) && v >= 0.0; }

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

bool live(const rxnn_layer* L) {
  if (!L) return false;
  std::lock_guard<std::mutex> g(g_mu);
  return g_live.count(L) && L->magic == kLayerMagic;
}

// Makes the layer's device current for the scope of a call.
struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) { ok = false; return; }
    if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
  }
  ~DeviceGuard() {
    int cur;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

// The nested-dissection build needs finite wire, driver and sense conductances.
bool nd_ok(const rxnn_xbar_params* p) {
  return p->r_row > 0.0 && p->r_col > 0.0 && p->r_sense > 0.0;
}

constexpr size_t kNdBudget = (size_t)1 << 30;  // bytes of build workspace per layer
constexpr int kMaxLut = 4096;                  // samples of a device characteristic table

rxnn_status check_xbar(const rxnn_xbar_params* p) {
  if (!p) return fail(RXNN_EINVAL, "params is NULL");
  if (p->rows < 1 || p->cols < 1)
    return fail(RXNN_EINVAL, "crossbar size %dx%d must be positive", p->rows, p->cols);
  if (p->rows > 256 || p->cols > 256)
    return fail(RXNN_EINVAL, "crossbar size %dx%d exceeds 256", p->rows, p->cols);
  if (!(isfinite(p->g_min) && p->g_min > 0.0 && isfinite(p->g_max) && p->g_max > p->g_min))
    return fail(RXNN_EINVAL, "need 0 < g_min < g_max (got %g, %g)", p->g_min, p->g_max);
  if (!finite_nonneg(p->r_driver) || !finite_nonneg(p->r_sense) || !finite_nonneg(p->r_row) ||
      !finite_nonneg(p->r_col))
    return fail(RXNN_EINVAL, "resistances must be finite and >= 0");
  if (p->weight_bits < 0 || p->weight_bits > 16)
    return fail(RXNN_EINVAL, "weight_bits %d not in 0..16", p->weight_bits);
  if (p->weight_bits == 0 && p->bits_per_slice != 0)
    return fail(RXNN_EINVAL, "bits_per_slice needs weight_bits > 0");
  if (p->bits_per_slice < 0 || p->bits_per_slice > p->weight_bits)
    return fail(RXNN_EINVAL, "bits_per_slice %d not in 0..weight_bits", p->bits_per_slice);
  if (p->bits_per_slice > 0 && p->weight_bits % p->bits_per_slice)
    return fail(RXNN_EINVAL, "weight_bits %d is not a multiple of bits_per_slice %d",
                p->weight_bits, p->bits_per_slice);
  if (!isfinite(p->w_max)) return fail(RXNN_EINVAL, "w_max must be finite");
  if (p->w_max > 3.0e38) return fail(RXNN_EINVAL, "w_max exceeds the fp32 range");
  if (!(isfinite(p->variation_sigma) && p->variation_sigma >= 0.0))
    return fail(RXNN_EINVAL, "variation_sigma must be finite and >= 0");
  if (p->variation && p->variation_sigma > 0.0)
    return fail(RXNN_EINVAL, "give either variation factors or variation_sigma, not both");
  if (p->g_lut) {
    if (p->g_lut_n < 2 || p->g_lut_n > kMaxLut)
      return fail(RXNN_EINVAL, "g_lut_n %d not in 2..%d", p->g_lut_n, kMaxLut);
    for (int k = 0; k < p->g_lut_n; ++k)
      if (!(isfinite(p->g_lut[k]) && p->g_lut[k] >= 0.0 && p->g_lut[k] <= 1.0))
        return fail(RXNN_EINVAL, "g_lut[%d] = %g is not in [0, 1]", k, p->g_lut[k]);
  } else if (p->g_lut_n != 0) {
    return fail(RXNN_EINVAL, "g_lut_n must be 0 without g_lut");
  }
  if (!nd_ok(p) && (p->rows > kMaxSweep || p->cols > kMaxSweep))
    return fail(RXNN_EUNSUPPORTED,
                "crossbars above %dx%d need positive wire, driver and sense resistances",
                kMaxSweep, kMaxSweep);
  return RXNN_OK;
}

// A convolution's shape, and that it matches the layer (P = c_in kh kw, Q = c_out).
rxnn_status check_conv(const MapScalars& ms, const rxnn_conv_desc* conv) {
  if (!conv) return fail(RXNN_EINVAL, "conv is NULL");
  const rxnn_conv_desc cd = *conv;
  if (cd.n < 0 || cd.c_in < 1 || cd.h < 1 || cd.w < 1 || cd.c_out < 1 || cd.kh < 1 ||
      cd.kw < 1 || cd.stride < 1 || cd.pad < 0)
    return fail(RXNN_EINVAL, "invalid convolution shape");
  if (cd.h + 2 * cd.pad < cd.kh || cd.w + 2 * cd.pad < cd.kw)
    return fail(RXNN_EINVAL, "kernel larger than the padded input");
  if (ms.P != (int64_t)cd.c_in * cd.kh * cd.kw || ms.Q != cd.c_out)
    return fail(RXNN_EINVAL, "layer is %lldx%lld but the convolution needs %lldx%d",
                (long long)ms.P, (long long)ms.Q, (long long)cd.c_in * cd.kh * cd.kw, cd.c_out);
  return RXNN_OK;
}

rxnn_status make_periph(const rxnn_periph_params* pp, const MapScalars& ms, PeriphScalars* out) {
  if (!pp) return fail(RXNN_EINVAL, "periph is NULL");
  if (pp->dac_bits < 0 || pp->dac_bits > kMaxBits)
    return fail(RXNN_EINVAL, "dac_bits %d not in 0..%d", pp->dac_bits, kMaxBits);
  if (pp->adc_bits < 0 || pp->adc_bits > kMaxBits)
    return fail(RXNN_EINVAL, "adc_bits %d not in 0..%d", pp->adc_bits, kMaxBits);
  if (!(isfinite(pp->x_max) && pp->x_max > 0.0))
    return fail(RXNN_EINVAL, "x_max must be finite and > 0");
  if (!(isfinite(pp->v_read) && pp->v_read > 0.0))
    return fail(RXNN_EINVAL, "v_read must be finite and > 0");
  if (!(isfinite(pp->dac_bend) && pp->dac_bend >= 0.0 && pp->dac_bend < 1.0))
    return fail(RXNN_EINVAL, "dac_bend must be in [0, 1)");
  if (!(isfinite(pp->adc_bend) && fabs(pp->adc_bend) <= 0.5))
    return fail(RXNN_EINVAL, "|adc_bend| must be <= 0.5");
  if (!(isfinite(pp->dac_g_on) && pp->dac_g_on >= 0.0 && isfinite(pp->dac_g_pd) &&
        pp->dac_g_pd >= 0.0))
    return fail(RXNN_EINVAL, "dac_g_on and dac_g_pd must be finite and >= 0");
  if (pp->dac_g_pd > 0.0) {
    if (!(pp->dac_g_on > 0.0)) return fail(RXNN_EINVAL, "the divider DAC needs dac_g_on > 0");
    if (pp->dac_bits == 0) return fail(RXNN_EINVAL, "the divider DAC needs dac_bits > 0");
    if (pp->dac_bend != 0.0) return fail(RXNN_EINVAL, "the divider DAC needs dac_bend = 0");
  }
  PeriphScalars ps;
  memset(&ps, 0, sizeof ps);
  ps.dac_bits = pp->dac_bits;
  ps.adc_bits = pp->adc_bits;
  ps.dac_levels = (1 << pp->dac_bits) - 1;
  ps.adc_levels = (1 << pp->adc_bits) - 1;
  ps.v_read = pp->v_read;
  ps.dac_bend = pp->dac_bend;
  ps.adc_bend = pp->adc_bend;
  ps.dac_s_in = pp->dac_bits ? (float)((double)ps.dac_levels / pp->x_max) : 0.0f;
  ps.s_v_ideal = (float)(pp->v_read / pp->x_max);
  ps.s_v = pp->v_read / pp->x_max;
  if (pp->dac_g_pd > 0.0) {
    const double vdd = pp->v_read * (pp->dac_g_on + pp->dac_g_pd) / pp->dac_g_on;
    ps.ldac = 1;
    ps.dac_inv_vdd = (float)(1.0 / vdd);
    ps.dac_hs = (float)((double)ps.dac_levels / (pp->dac_g_on * vdd));
    ps.dac_gpd = (float)pp->dac_g_pd;
  }
  ps.i_fs = pp->v_read * (double)ms.M * ms.g_max;
  if (pp->adc_bits) {
    ps.lsb = ps.i_fs / (double)ps.adc_levels;
    // bucket width w <= 1 / 3.25 of the smallest threshold spacing
    // (1 - |bend|) I_FS / L: a current rounded into a neighbouring bucket
    // still leaves at most one threshold between the bucket's lower edge and
    // the current, so the bucket's code is exact or one too low
    const double need = 3.25 * ps.adc_levels / (1.0 - fabs(pp->adc_bend));
    const int nb = (int)ceil(need) < 16 ? 16 : (int)ceil(need);
    if (nb > kMaxBuckets) return fail(RXNN_EINVAL, "ADC bucket table too large");
    ps.n_buckets = nb;
    ps.bucket_inv_w = (float)((double)nb / ps.i_fs);
    ps.bucket_w = ps.i_fs / (double)nb;
  }
  *out = ps;
  return RXNN_OK;
}

// ---- kernel timing ------------------------------------------------------------
struct Pending {
  std::string name;
  hipEvent_t a, b;
  double bytes;
};
struct ProfTotal {
  double ms = 0.0;
  int64_t count = 0;
  double bytes = 0.0;
};
int g_prof = 0;   // 0 off, 1 every kernel, 2 the evaluation kernel only
std::vector<Pending> g_pending;
std::map<std::string, ProfTotal> g_prof_tot;

// Frees every device buffer of a layer and the handle itself.
void release_buffers(rxnn_layer* L) {
  void* bufs[] = {L->gpt,  L->d_wmax, L->ws,    L->nd_ws, L->ktab,
                  L->vbuf, L->d_vf,   L->d_lut, L->bw_ws, L->gload, L->adct};
  for (void* b : bufs)
    if (b) (void)hipFree(b);
  L->magic = 0;
  delete L;
}

rxnn_status grow_ws(rxnn_layer* L, size_t bytes) {
  if (L->ws_bytes >= bytes) return RXNN_OK;
  if (L->ws) HIP_TRY(hipFree(L->ws));
  L->ws = nullptr;
  L->ws_bytes = 0;
  void* p = nullptr;
  if (hipMalloc(&p, bytes) != hipSuccess) {
    (void)hipGetLastError();
    return fail(RXNN_ENOMEM, "cannot allocate %zu bytes of workspace", bytes);
  }
  L->ws = p;
  L->ws_bytes = bytes;
  L->ws_dirty = true;
  return RXNN_OK;
}

// Largest |acc| = R * L_adc * sum_s 2^(b_s s) must fit int32.
rxnn_status check_acc_range(const MapScalars& ms, const PeriphScalars& ps) {
  if (!ps.adc_bits) return RXNN_OK;
  double w = 0.0;
  for (int s = 0; s < ms.n_slices; ++s) w += ldexp(1.0, ms.slice_bits * s);
  const double mx = (double)ms.R * ps.adc_levels * w;
  if (mx >= 2147483647.0)
    return fail(RXNN_EUNSUPPORTED, "accumulated codes can reach %.3g, beyond int32", mx);
  return RXNN_OK;
}

// Device buffers of one evaluation call: the layer's own (grown on demand,
// cached across calls) or carved out of the fixed scratch array.
struct EvalBufs {
  float2* adct = nullptr;     // ADC bucket table
  bool adct_build = false;    // (re)build it in this call
  float* gload = nullptr;     // divider DAC: row loads of every array
  bool gload_build = false;
  int32_t* iacc = nullptr;    // shared-tile int32 workspace (null: no split)
  int64_t iacc_clear = 0;     // words of it to clear before the evaluation kernel
  float* vbuf = nullptr;      // DAC output
};

// The layer-owned buffers for a call with `workers` shared-tile workers and
// n_v DAC outputs (allocates what is missing or too small).
rxnn_status layer_bufs(const rxnn_layer* L, const PeriphScalars& ps, int workers, int64_t Bv,
                       int64_t n_v, EvalBufs* b) {
  const MapScalars& ms = L->ms;
  rxnn_layer* Lm = const_cast<rxnn_layer*>(L);
  if (ps.ldac) {
    if (!Lm->gload) {
      void* p = nullptr;
      const size_t bytes = (size_t)ms.R * ms.C * ms.A * ms.Mp * sizeof(float);
      if (hipMalloc(&p, bytes) != hipSuccess) {
        (void)hipGetLastError();
        return fail(RXNN_ENOMEM, "cannot allocate %zu bytes for the row loads", bytes);
      }
      Lm->gload = (float*)p;
    }
    b->gload = Lm->gload;
    b->gload_build = !Lm->gload_valid;
  }
  if (ps.adc_bits > 0) {
    // the ADC's bucket table, rebuilt when the converter changes
    const double key[5] = {(double)ps.adc_levels, (double)ps.n_buckets, ps.i_fs, ps.adc_bend,
                           ps.bucket_w};
    const bool current = Lm->adct && memcmp(key, Lm->adct_key, sizeof key) == 0;
    if (!Lm->adct) {
      void* p = nullptr;
      if (hipMalloc(&p, (size_t)(kMaxBuckets + 2) * sizeof(float2)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(RXNN_ENOMEM, "cannot allocate the ADC table");
      }
      Lm->adct = (float2*)p;
    }
    b->adct = Lm->adct;
    b->adct_build = !current;
  }
  if (workers > 0) {
    rxnn_status st = grow_ws(Lm, (size_t)Bv * ms.Q * sizeof(int32_t));
    if (st) return st;
    b->iacc = (int32_t*)Lm->ws;
    // the finish kernel zeroes again every word it reads and no other word is
    // ever written, so the workspace is cleared only when new or after a call
    // that did not end
    b->iacc_clear = Lm->ws_dirty ? (int64_t)(Lm->ws_bytes / sizeof(int32_t)) : 0;
  }
  if ((size_t)n_v * sizeof(float) > L->vbuf_bytes) {
    if (Lm->vbuf) HIP_TRY(hipFree(Lm->vbuf));
    Lm->vbuf = nullptr;
    Lm->vbuf_bytes = 0;
    void* p = nullptr;
    if (hipMalloc(&p, (size_t)n_v * sizeof(float)) != hipSuccess) {
      (void)hipGetLastError();
      return fail(RXNN_ENOMEM, "cannot allocate %zu bytes for the DAC output",
                  (size_t)n_v * sizeof(float));
    }
    Lm->vbuf = (float*)p;
    Lm->vbuf_bytes = (size_t)n_v * sizeof(float);
  }
  b->vbuf = L->vbuf;
  return RXNN_OK;
}

// The same buffers carved out of `base` (kScratchBytes, 256-byte aligned):
// every table is rebuilt and the workspace cleared in every call, since
// calls on other layers share the scratch.  RXNN_EINVAL when they do not fit.
rxnn_status scratch_bufs(const rxnn_layer* L, const PeriphScalars& ps, int workers, int64_t Bv,
                         int64_t n_v, unsigned char* base, EvalBufs* b) {
  const MapScalars& ms = L->ms;
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  size_t off = 0;
  if (ps.adc_bits > 0) {
    b->adct = (float2*)(base + off);
    b->adct_build = true;
    off += up((size_t)(kMaxBuckets + 2) * sizeof(float2));
  }
  if (ps.ldac) {
    b->gload = (float*)(base + off);
    b->gload_build = true;
    off += up((size_t)ms.R * ms.C * ms.A * ms.Mp * sizeof(float));
  }
  if (workers > 0) {
    b->iacc = (int32_t*)(base + off);
    b->iacc_clear = Bv * ms.Q;
    off += up((size_t)Bv * ms.Q * sizeof(int32_t));
  }
  b->vbuf = (float*)(base + off);
  off += up((size_t)n_v * sizeof(float));
  if (off > kScratchBytes)
    return fail(RXNN_EINVAL,
                "the call needs %zu bytes of scratch, more than the fixed %zu (B x (R M + 64) "
                "DAC outputs, B x Q workspace words and the tables); use rxnn_crossbar_vmm or a "
                "smaller batch",
                off, kScratchBytes);
  return RXNN_OK;
}

// Device address of the scratch array on device `dev` (current), looked up
// once per device.
constexpr int kMaxDevices = 64;
unsigned char* g_scratch_ptr[kMaxDevices];

rxnn_status scratch_address(int dev, unsigned char** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(RXNN_EUNSUPPORTED, "device %d out of range", dev);
  std::lock_guard<std::mutex> g(g_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(RXNN_EHIP, "hipGetSymbolAddress of the scratch array failed: %s",
                  hipGetErrorString(e));
    g_scratch_ptr[dev] = (unsigned char*)p;
  }
  *out = g_scratch_ptr[dev];
  return RXNN_OK;
}

rxnn_status run_vmm(const rxnn_layer* L, const PeriphScalars& ps, const float* X,
                    const rxnn_conv_desc* conv, int64_t Bv, float* Y, int64_t hw_out,
                    float* dbgI, int32_t* dbgC, hipStream_t s, const int* ktab = nullptr,
                    unsigned char* scratch_base = nullptr) {
  const MapScalars& ms = L->ms;
  // the divider stands in for the driver; the rows' loads follow G'
  if (ps.ldac && ms.r_driver != 0.0)
    return fail(RXNN_EINVAL, "the divider DAC needs a layer mapped with r_driver = 0");
  const bool grp = use_groups(ms, ps, dbgI || dbgC);
  VmmPlan plan{0, 0, 0};
  if (!(dbgI || dbgC)) plan = vmm_plan(ms, ps, Bv, conv != nullptr, grp);
  const int workers = plan.workers;
  const int64_t n_v = dac_elems(ms, conv, Bv);
  EvalBufs b;
  rxnn_status st = scratch_base ? scratch_bufs(L, ps, workers, Bv, n_v, scratch_base, &b)
                                : layer_bufs(L, ps, workers, Bv, n_v, &b);
  if (st) return st;
  rxnn_layer* Lw = const_cast<rxnn_layer*>(L);
  if (b.gload_build) {
    {
      ProfScope t("gload", s);
      HIP_TRY(launch_gload(ms, L->gpt, b.gload, s));
    }
    if (!scratch_base) Lw->gload_valid = true;
  }
  if (b.adct_build) {
    {
      ProfScope t("adc_table", s);
      HIP_TRY(launch_adc_table(ps, b.adct, s));
    }
    if (!scratch_base) {
      const double key[5] = {(double)ps.adc_levels, (double)ps.n_buckets, ps.i_fs, ps.adc_bend,
                             ps.bucket_w};
      memcpy(Lw->adct_key, key, sizeof key);
    }
  }
  {
    // algorithmic bytes: every input read once, every V element written once
    const double n_in = conv ? (double)conv->n * conv->c_in * conv->h * conv->w : (double)Bv * ms.P;
    ProfScope t("dac", s, 4.0 * (n_in + (double)n_v));
    HIP_TRY(launch_dac(ms, ps, conv, X, Bv, b.vbuf, s));
  }
  VmmLaunch vl;
  vl.V = b.vbuf;
  vl.conv = conv;
  vl.ldx = conv ? 0 : fc_ldv(ms);
  vl.Bv = Bv;
  vl.Y = Y;
  vl.hw_out = hw_out;
  vl.iacc = b.iacc;
  vl.dbg_I = dbgI;
  vl.dbg_code = dbgC;
  vl.ktab = ktab;
  vl.gload = b.gload;
  vl.grp = grp;
  vl.adc_tab = b.adct;
  if (workers > 0) {
    if (b.iacc_clear > 0) {
      ProfScope z("fill", s);
      HIP_TRY(launch_fill_u32((unsigned*)b.iacc, b.iacc_clear, 0u, s));
    }
    if (!scratch_base) Lw->ws_dirty = true;   // until the finish kernel has been launched
  }
  {
    ProfScope t("xbar_vmm", s);
    HIP_TRY(launch_xbar_vmm(ms, ps, L->gpt, vl, plan, s));
  }
  if (workers > 0) {
    // per output of a shared tile: the int32 read, its zeroing write, the fp32 write
    ProfScope t("finish", s, 12.0 * (double)(Bv - plan.row0) * (double)ms.Q);
    HIP_TRY(launch_finish(ms, ps, b.iacc, plan.row0, Bv, Y, hw_out, s));
    if (!scratch_base) Lw->ws_dirty = false;
  }
  return RXNN_OK;
}

rxnn_status vmm_common(const rxnn_layer* layer, const rxnn_periph_params* periph,
                       const float* X, int64_t B, float* Y, float* dbgI, int32_t* dbgC,
                       void* stream) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  if (B < 0) return fail(RXNN_EINVAL, "B must be >= 0");
  if (B > 0 && (!X || !Y)) return fail(RXNN_EINVAL, "X and Y must not be NULL");
  rxnn_layer* L = const_cast<rxnn_layer*>(layer);
  PeriphScalars ps;
  rxnn_status st = make_periph(periph, L->ms, &ps);
  if (st) return st;
  if ((st = check_acc_range(L->ms, ps))) return st;
  // the evaluation kernel addresses a 128-row block of X with 32-bit byte offsets
  if (L->ms.P >= (int64_t)1 << 22)
    return fail(RXNN_EUNSUPPORTED, "P must be below 2^22 for the evaluation kernel");
  if (B == 0) return RXNN_OK;
  DeviceGuard dg(L->device);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layer's device");
  hipStream_t s = (hipStream_t)stream;
  return run_vmm(L, ps, X, nullptr, B, Y, 0, dbgI, dbgC, s);
}

// w_max (fixed or reduced from W) followed by the G' build of every array.
// w_max of a layer: the fixed one, or max |W| reduced on the device.
hipError_t launch_wmax(rxnn_layer* L, const float* W, hipStream_t s) {
  const MapScalars& ms = L->ms;
  ProfScope t("wmax", s);
  if (ms.wmax_fixed > 0.0f)
    return launch_fill_u32((unsigned*)L->d_wmax, 1, __builtin_bit_cast(unsigned, ms.wmax_fixed), s);
  return launch_absmax(W, ms.P * ms.Q, (unsigned*)L->d_wmax, s);
}

hipError_t build_gprime(rxnn_layer* L, const float* W, hipStream_t s) {
  L->gload_valid = false;   // the row loads follow G'
  const MapScalars& ms = L->ms;
  hipError_t e = launch_wmax(L, W, s);
  if (e == hipSuccess) {
    if (!L->nd_ws) {
      ProfScope t("gprime_sweep", s);
      return launch_gprime_build(ms, W, L->gpt, s);
    }
    const int64_t n_arrays = (int64_t)ms.R * ms.C * ms.A;
    for (int64_t a0 = 0; a0 < n_arrays && e == hipSuccess; a0 += L->nd_chunk) {
      const int64_t n = n_arrays - a0 < L->nd_chunk ? n_arrays - a0 : L->nd_chunk;
      e = launch_nd_build(ms, W, L->gpt, a0, n, L->nd_bs, L->nd_ws, s);
    }
  }
  return e;
}

}  // namespace

namespace rxnn {

ProfScope::ProfScope(const char* name, hipStream_t s, double bytes)
    : name_(name), s_(s), bytes_(bytes), on_(false) {
  if (!g_prof || (g_prof == 2 && strcmp(name, "xbar_vmm") != 0)) return;
  // no system-scope fence: a timing event then costs no cache flush on the GPU
  if (hipEventCreateWithFlags(&a_, hipEventDisableSystemFence) != hipSuccess) return;
  if (hipEventCreateWithFlags(&b_, hipEventDisableSystemFence) != hipSuccess) {
    (void)hipEventDestroy(a_);
    return;
  }
  if (hipEventRecord(a_, s_) != hipSuccess) {
    (void)hipEventDestroy(a_);
    (void)hipEventDestroy(b_);
    return;
  }
  on_ = true;
}

ProfScope::~ProfScope() {
  if (!on_) return;
  if (hipEventRecord(b_, s_) != hipSuccess) {
    (void)hipEventDestroy(a_);
    (void)hipEventDestroy(b_);
    return;
  }
  std::lock_guard<std::mutex> g(g_mu);
  g_pending.push_back(Pending{name_, a_, b_, bytes_});
}

}  // namespace rxnn

extern "C" {

const char* rxnn_status_string(rxnn_status st) {
  switch (st) {
    case RXNN_OK: return "ok";
    case RXNN_EINVAL: return "invalid argument";
    case RXNN_ENOMEM: return "out of device memory";
    case RXNN_EHIP: return "HIP runtime error";
    case RXNN_EUNSUPPORTED: return "unsupported by this library";
  }
  return "unknown status";
}

const char* rxnn_last_error(void) { return g_err.c_str(); }

rxnn_status rxnn_map_layer(const rxnn_xbar_params* params, const float* W, int64_t P, int64_t Q,
                           void* stream, rxnn_layer** out) {
  if (!out) return fail(RXNN_EINVAL, "out is NULL");
  *out = nullptr;
  rxnn_status st = check_xbar(params);
  if (st) return st;
  if (P < 1 || Q < 1) return fail(RXNN_EINVAL, "P and Q must be >= 1");
  if (P > (int64_t)1 << 31 || Q > (int64_t)1 << 31)
    return fail(RXNN_EINVAL, "P and Q must be <= 2^31");
  if (!W) return fail(RXNN_EINVAL, "W is NULL");
  MapScalars ms;
  memset(&ms, 0, sizeof ms);
  ms.M = params->rows;
  ms.N = params->cols;
  ms.P = P;
  ms.Q = Q;
  ms.R = (int)((P + ms.M - 1) / ms.M);
  ms.C = (int)((Q + ms.N - 1) / ms.N);
  ms.weight_bits = params->weight_bits;
  ms.slice_bits = params->weight_bits
                      ? (params->bits_per_slice ? params->bits_per_slice : params->weight_bits)
                      : 0;
  ms.n_slices = params->weight_bits ? params->weight_bits / ms.slice_bits : 1;
  if (ms.slice_bits * (ms.n_slices - 1) > 24)
    return fail(RXNN_EUNSUPPORTED, "slice weights beyond 2^24 are not supported");
  ms.A = 2 * ms.n_slices;
  ms.Mp = (int)round_up(ms.M, 16);
  ms.Np = (int)round_up(ms.N, 16);
  ms.g_min = params->g_min;
  ms.g_max = params->g_max;
  ms.r_driver = params->r_driver;
  ms.r_sense = params->r_sense;
  ms.r_row = params->r_row;
  ms.r_col = params->r_col;
  if (ms.slice_bits == 0) {
    ms.sw_num = ms.g_max - ms.g_min;
  } else {
    const double dG = (ms.g_max - ms.g_min) / (double)((1 << ms.slice_bits) - 1);
    ms.sw_num = dG * (double)((1 << ms.weight_bits) - 1);
  }
  ms.wmax_fixed = params->w_max > 0.0 ? (float)params->w_max : 0.0f;
  if (params->w_max > 0.0 && !(ms.wmax_fixed > 0.0f))
    return fail(RXNN_EINVAL, "w_max underflows fp32");

  int dev;
  HIP_TRY(hipGetDevice(&dev));
  const size_t gbytes = (size_t)ms.C * ms.R * ms.A * ms.Np * ms.Mp * sizeof(float);
  rxnn_layer* L = new (std::nothrow) rxnn_layer();
  if (!L) return fail(RXNN_ENOMEM, "host allocation failed");
  memset(L, 0, sizeof *L);
  L->device = dev;
  L->params = *params;
  L->params.variation = nullptr;   // the layer keeps its own copies
  L->params.g_lut = nullptr;
  if (hipMalloc((void**)&L->gpt, gbytes) != hipSuccess) {
    (void)hipGetLastError();
    release_buffers(L);
    return fail(RXNN_ENOMEM, "cannot allocate %zu bytes for G'", gbytes);
  }
  if (hipMalloc((void**)&L->d_wmax, 256) != hipSuccess) {
    (void)hipGetLastError();
    release_buffers(L);
    return fail(RXNN_ENOMEM, "cannot allocate w_max");
  }
  if (params->variation) {
    // one factor per device: [C][R][A][M][N]
    const size_t vbytes = (size_t)ms.C * ms.R * ms.A * ms.M * ms.N * sizeof(float);
    if (hipMalloc((void**)&L->d_vf, vbytes) != hipSuccess) {
      (void)hipGetLastError();
      release_buffers(L);
      return fail(RXNN_ENOMEM, "cannot allocate %zu bytes of variation factors", vbytes);
    }
    if (hipMemcpyAsync(L->d_vf, params->variation, vbytes, hipMemcpyDeviceToDevice,
                       (hipStream_t)stream) != hipSuccess) {
      (void)hipGetLastError();
      release_buffers(L);
      return fail(RXNN_EHIP, "cannot copy the variation factors");
    }
    ms.vf = L->d_vf;
  }
  ms.vf_sigma = params->variation_sigma;
  ms.vf_seed = params->variation_seed;
  if (params->g_lut) {
    const size_t lbytes = (size_t)params->g_lut_n * sizeof(double);
    if (hipMalloc((void**)&L->d_lut, lbytes) != hipSuccess) {
      (void)hipGetLastError();
      release_buffers(L);
      return fail(RXNN_ENOMEM, "cannot allocate the characteristic table");
    }
    if (hipMemcpy(L->d_lut, params->g_lut, lbytes, hipMemcpyHostToDevice) != hipSuccess) {
      (void)hipGetLastError();
      release_buffers(L);
      return fail(RXNN_EHIP, "cannot copy the characteristic table");
    }
    ms.lut = L->d_lut;
    ms.lut_n = params->g_lut_n;
  }
  if (nd_ok(params)) {
    int64_t si, so, sc;
    const int T = nd_side(ms.M, ms.N);
    const int64_t n_arrays = (int64_t)ms.R * ms.C * ms.A;
    L->nd_bs = nd_block_side(T, n_arrays);
    nd_sizes(T, ms.M, L->nd_bs, &si, &so, &sc);
    const size_t per = (size_t)(si + so + sc) * sizeof(double);
    int64_t chunk = (int64_t)(kNdBudget / per);
    if (chunk < 1) chunk = 1;
    if (chunk > n_arrays) chunk = n_arrays;
    if (hipMalloc((void**)&L->nd_ws, per * chunk) != hipSuccess) {
      (void)hipGetLastError();
      release_buffers(L);
      return fail(RXNN_ENOMEM, "cannot allocate %zu bytes of build workspace", per * chunk);
    }
    L->nd_chunk = chunk;
  }
  ms.d_wmax = L->d_wmax;
  L->ms = ms;
  L->magic = kLayerMagic;
  // the w_max reduction's accumulator and ticket counter start at zero (it
  // leaves them so after every call)
  hipError_t e = launch_fill_u32((unsigned*)L->d_wmax, 4, 0u, (hipStream_t)stream);
  if (e == hipSuccess) e = build_gprime(L, W, (hipStream_t)stream);
  if (e != hipSuccess) {
    release_buffers(L);
    return fail(RXNN_EHIP, "mapping launch failed: %s", hipGetErrorString(e));
  }
  {
    std::lock_guard<std::mutex> g(g_mu);
    g_live.insert(L);
  }
  *out = L;
  return RXNN_OK;
}

}  // extern "C"

namespace {

// Batched rebuilds: per device, the layer and array tables of the last batch
// and one build workspace, grown on demand and kept until the process ends
// (at most kBatchBudget bytes: larger batches are built in chunks).
struct BatchState {
  NdBatchLayer* d_layers = nullptr;
  int64_t layers_cap = 0;
  int2* d_ent = nullptr;
  int64_t ent_cap = 0;
  double* ws = nullptr;
  int64_t ws_cap = 0;          // doubles
  int* d_start = nullptr;      // the layers' first blocks of the batched w_max reduction
  int64_t start_cap = 0;
  std::vector<NdBatchLayer> h_layers;
  std::vector<int2> h_ent;
  std::vector<int> h_start;
};
constexpr size_t kBatchBudget = (size_t)24 << 30;
BatchState g_batch[kMaxDevices];
std::mutex g_batch_mu;

template <typename T>
rxnn_status grow_dev(T** p, int64_t* cap, int64_t need, const char* what) {
  if (*cap >= need) return RXNN_OK;
  if (*p) HIP_TRY(hipFree(*p));
  *p = nullptr;
  *cap = 0;
  if (hipMalloc((void**)p, (size_t)need * sizeof(T)) != hipSuccess) {
    (void)hipGetLastError();
    *p = nullptr;
    return fail(RXNN_ENOMEM, "cannot allocate %zu bytes for the %s",
                (size_t)need * sizeof(T), what);
  }
  *cap = need;
  return RXNN_OK;
}

bool same_network(const rxnn_layer* a, const rxnn_layer* b) {
  return a->device == b->device && a->ms.M == b->ms.M && a->ms.N == b->ms.N &&
         a->ms.r_driver == b->ms.r_driver && a->ms.r_sense == b->ms.r_sense &&
         a->ms.r_row == b->ms.r_row && a->ms.r_col == b->ms.r_col;
}

}  // namespace

extern "C" {

rxnn_status rxnn_remap_layers(rxnn_layer* const* layers, const float* const* W, int32_t n,
                              void* stream) {
  if (n < 1) return fail(RXNN_EINVAL, "n must be >= 1");
  if (!layers || !W) return fail(RXNN_EINVAL, "layers and W must not be NULL");
  for (int32_t i = 0; i < n; ++i) {
    if (!live(layers[i])) return fail(RXNN_EINVAL, "layer %d is invalid or released", i);
    if (!W[i]) return fail(RXNN_EINVAL, "W[%d] is NULL", i);
    if (!layers[i]->nd_ws)
      return fail(RXNN_EINVAL, "layer %d uses the row-sweep build (a zero wire or sense "
                  "resistance); rebuild it with rxnn_remap_layer", i);
    if (!same_network(layers[i], layers[0]))
      return fail(RXNN_EINVAL, "layer %d differs from layer 0 in device, crossbar size or "
                  "resistances", i);
    for (int32_t j = 0; j < i; ++j)
      if (layers[j] == layers[i]) return fail(RXNN_EINVAL, "layer %d appears twice", i);
  }
  const int dev = layers[0]->device;
  if (dev < 0 || dev >= kMaxDevices) return fail(RXNN_EUNSUPPORTED, "device %d out of range", dev);
  DeviceGuard dg(dev);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layers' device");
  hipStream_t s = (hipStream_t)stream;
  std::lock_guard<std::mutex> g(g_batch_mu);
  BatchState& bs = g_batch[dev];
  bs.h_layers.resize((size_t)n);
  bs.h_ent.clear();
  bs.h_start.resize((size_t)n + 1);
  bs.h_start[0] = 0;
  for (int32_t i = 0; i < n; ++i) {
    rxnn_layer* L = layers[i];
    bs.h_layers[(size_t)i] = NdBatchLayer{L->ms, W[i], L->gpt};
    const int64_t na = (int64_t)L->ms.R * L->ms.C * L->ms.A;
    for (int64_t a = 0; a < na; ++a) bs.h_ent.push_back(make_int2(i, (int)a));
    bs.h_start[(size_t)i + 1] =
        bs.h_start[(size_t)i] + (L->ms.wmax_fixed > 0.0f ? 1 : absmax_blocks(L->ms.P * L->ms.Q));
  }
  const int64_t total = (int64_t)bs.h_ent.size();
  const MapScalars& ms0 = layers[0]->ms;
  int64_t si, so, sc;
  const int T = nd_side(ms0.M, ms0.N);
  const int nbs = nd_block_side(T, total);
  nd_sizes(T, ms0.M, nbs, &si, &so, &sc);
  const int64_t per = si + so + sc;   // doubles of workspace per array
  int64_t chunk = (int64_t)(kBatchBudget / sizeof(double)) / per;
  if (chunk < 1) chunk = 1;
  if (chunk > total) chunk = total;
  rxnn_status st;
  if ((st = grow_dev(&bs.d_layers, &bs.layers_cap, n, "batch layer table"))) return st;
  if ((st = grow_dev(&bs.d_ent, &bs.ent_cap, total, "batch array table"))) return st;
  if ((st = grow_dev(&bs.ws, &bs.ws_cap, chunk * per, "batch build workspace"))) return st;
  if ((st = grow_dev(&bs.d_start, &bs.start_cap, (int64_t)n + 1, "batch w_max table"))) return st;
  // the tables go over on the stream (from pageable memory: staged before return)
  HIP_TRY(hipMemcpyAsync(bs.d_layers, bs.h_layers.data(), (size_t)n * sizeof(NdBatchLayer),
                         hipMemcpyHostToDevice, s));
  HIP_TRY(hipMemcpyAsync(bs.d_ent, bs.h_ent.data(), (size_t)total * sizeof(int2),
                         hipMemcpyHostToDevice, s));
  HIP_TRY(hipMemcpyAsync(bs.d_start, bs.h_start.data(), ((size_t)n + 1) * sizeof(int),
                         hipMemcpyHostToDevice, s));
  for (int32_t i = 0; i < n; ++i) layers[i]->gload_valid = false;   // the row loads follow G'
  {
    // every layer's w_max at once
    ProfScope t("wmax", s);
    hipError_t e = launch_absmax_batch(bs.d_layers, bs.d_start, n, bs.h_start[(size_t)n], s);
    if (e != hipSuccess) return fail(RXNN_EHIP, "w_max launch failed: %s", hipGetErrorString(e));
  }
  const NdBatch batch{bs.d_layers, bs.d_ent};
  for (int64_t a0 = 0; a0 < total; a0 += chunk) {
    const int64_t m = total - a0 < chunk ? total - a0 : chunk;
    hipError_t e = launch_nd_build(ms0, nullptr, nullptr, a0, m, nbs, bs.ws, s, &batch);
    if (e != hipSuccess)
      return fail(RXNN_EHIP, "mapping launch failed: %s", hipGetErrorString(e));
  }
  return RXNN_OK;
}

rxnn_status rxnn_remap_layer(rxnn_layer* layer, const float* W, void* stream) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  if (!W) return fail(RXNN_EINVAL, "W is NULL");
  DeviceGuard dg(layer->device);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layer's device");
  hipError_t e = build_gprime(layer, W, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RXNN_EHIP, "mapping launch failed: %s", hipGetErrorString(e));
  return RXNN_OK;
}

rxnn_status rxnn_crossbar_vmm(const rxnn_layer* layer, const rxnn_periph_params* periph,
                              const float* X, int64_t B, float* Y, void* stream) {
  return vmm_common(layer, periph, X, B, Y, nullptr, nullptr, stream);
}

rxnn_status rxnn_crossbar_vmm_noalloc(const rxnn_layer* layer, const rxnn_periph_params* periph,
                                      const float* X, int64_t B, float* Y, void* stream) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  if (B < 0) return fail(RXNN_EINVAL, "B must be >= 0");
  if (B > 0 && (!X || !Y)) return fail(RXNN_EINVAL, "X and Y must not be NULL");
  const rxnn_layer* L = layer;
  PeriphScalars ps;
  rxnn_status st = make_periph(periph, L->ms, &ps);
  if (st) return st;
  if ((st = check_acc_range(L->ms, ps))) return st;
  if (L->ms.P >= (int64_t)1 << 22)
    return fail(RXNN_EUNSUPPORTED, "P must be below 2^22 for the evaluation kernel");
  if (B == 0) return RXNN_OK;
  DeviceGuard dg(L->device);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layer's device");
  unsigned char* base = nullptr;
  if ((st = scratch_address(L->device, &base))) return st;
  return run_vmm(L, ps, X, nullptr, B, Y, 0, nullptr, nullptr, (hipStream_t)stream, nullptr,
                 base);
}

rxnn_status rxnn_vmm_debug(const rxnn_layer* layer, const rxnn_periph_params* periph,
                           const float* X, int64_t B, float* Y, float* I_preadc, int32_t* codes,
                           void* stream) {
  return vmm_common(layer, periph, X, B, Y, I_preadc, codes, stream);
}

rxnn_status rxnn_conv_layer(const rxnn_layer* layer, const rxnn_periph_params* periph,
                            const rxnn_conv_desc* conv, const float* X, float* Y,
                            void* stream) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  rxnn_layer* L = const_cast<rxnn_layer*>(layer);
  const MapScalars& ms = L->ms;
  rxnn_status cst = check_conv(ms, conv);
  if (cst) return cst;
  const rxnn_conv_desc cd = *conv;
  if (ms.P >= (int64_t)1 << 22)
    return fail(RXNN_EUNSUPPORTED, "P must be below 2^22 for the evaluation kernel");
  PeriphScalars ps;
  rxnn_status st = make_periph(periph, ms, &ps);
  if (st) return st;
  if ((st = check_acc_range(ms, ps))) return st;
  const int64_t ho = (cd.h + 2 * cd.pad - cd.kh) / cd.stride + 1;
  const int64_t wo = (cd.w + 2 * cd.pad - cd.kw) / cd.stride + 1;
  const int64_t Bv = (int64_t)cd.n * ho * wo;
  if (Bv > INT32_MAX)
    return fail(RXNN_EUNSUPPORTED, "more than 2^31 - 1 output pixels per call");
  {
    // the images one 128-pixel block of the evaluation kernel reads are
    // addressed with 32-bit byte offsets
    const int64_t span = std::min<int64_t>(cd.n, 127 / (ho * wo) + 2);
    if (span * cd.c_in * (cd.h + 2 * (int64_t)cd.pad) * (cd.w + 2 * (int64_t)cd.pad) * 4 >=
        (int64_t)1 << 31)
      return fail(RXNN_EUNSUPPORTED, "input images too large for the evaluation kernel");
  }
  if ((int64_t)cd.n * cd.c_in * (cd.h + 2 * (int64_t)cd.pad) * (cd.w + 2 * (int64_t)cd.pad) >=
      ((int64_t)1 << 32) - ((int64_t)1 << 23))
    return fail(RXNN_EUNSUPPORTED, "the zero-bordered input must hold fewer than 2^32 - 2^23 "
                "elements (32-bit indexing of the DAC pass)");
  if (Bv == 0) return RXNN_OK;
  if (!X || !Y) return fail(RXNN_EINVAL, "X and Y must not be NULL");
  DeviceGuard dg(L->device);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layer's device");
  hipStream_t s = (hipStream_t)stream;
  // patch-column table (per row tile and input: byte offset in the window of
  // the padded input), rebuilt when the geometry changes
  {
    const bool grp = use_groups(ms, ps, false);
    const int key[7] = {cd.c_in, cd.h, cd.w, cd.kh, cd.kw, cd.pad, grp ? 1 : 0};
    const int64_t n = ktab_entries(ms, grp);
    if (!L->ktab || memcmp(key, L->ktab_key, sizeof key) != 0) {
      if (L->ktab_cap < n) {
        if (L->ktab) HIP_TRY(hipFree(L->ktab));
        L->ktab = nullptr;
        L->ktab_cap = 0;
        void* p = nullptr;
        if (hipMalloc(&p, (size_t)n * sizeof(int)) != hipSuccess) {
          (void)hipGetLastError();
          return fail(RXNN_ENOMEM, "cannot allocate the patch-column table");
        }
        L->ktab = (int*)p;
        L->ktab_cap = n;
      }
      {
        ProfScope t("ktab", s);
        HIP_TRY(launch_conv_ktab(ms, cd, grp, L->ktab, s));
      }
      memcpy(L->ktab_key, key, sizeof key);
    }
  }
  const int* ktab = L->ktab;
  return run_vmm(L, ps, X, &cd, Bv, Y, ho * wo, nullptr, nullptr, s, ktab);
}

rxnn_status rxnn_get_gprime(const rxnn_layer* layer, int64_t row_tile, int64_t col_tile,
                            int64_t array, float* host_out) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  const MapScalars& ms = layer->ms;
  if (row_tile < 0 || row_tile >= ms.R || col_tile < 0 || col_tile >= ms.C || array < 0 ||
      array >= ms.A)
    return fail(RXNN_EINVAL, "tile (%lld, %lld, %lld) out of range", (long long)row_tile,
                (long long)col_tile, (long long)array);
  if (!host_out) return fail(RXNN_EINVAL, "host_out is NULL");
  DeviceGuard dg(layer->device);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layer's device");
  std::vector<float> t((size_t)ms.Np * ms.Mp);
  const int64_t arr = (col_tile * ms.R + row_tile) * ms.A + array;
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(t.data(), layer->gpt + arr * ms.Np * ms.Mp, t.size() * sizeof(float),
                    hipMemcpyDeviceToHost));
  for (int i = 0; i < ms.M; ++i)
    for (int j = 0; j < ms.N; ++j) host_out[(size_t)i * ms.N + j] = t[(size_t)j * ms.Mp + i];
  return RXNN_OK;
}

rxnn_status rxnn_set_gprime(rxnn_layer* layer, int64_t row_tile, int64_t col_tile, int64_t array,
                            const float* host_in) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  const MapScalars& ms = layer->ms;
  if (row_tile < 0 || row_tile >= ms.R || col_tile < 0 || col_tile >= ms.C || array < 0 ||
      array >= ms.A)
    return fail(RXNN_EINVAL, "tile (%lld, %lld, %lld) out of range", (long long)row_tile,
                (long long)col_tile, (long long)array);
  if (!host_in) return fail(RXNN_EINVAL, "host_in is NULL");
  DeviceGuard dg(layer->device);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layer's device");
  std::vector<float> t((size_t)ms.Np * ms.Mp, 0.0f);
  for (int i = 0; i < ms.M; ++i)
    for (int j = 0; j < ms.N; ++j) t[(size_t)j * ms.Mp + i] = host_in[(size_t)i * ms.N + j];
  const int64_t arr = (col_tile * ms.R + row_tile) * ms.A + array;
  layer->gload_valid = false;
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(layer->gpt + arr * ms.Np * ms.Mp, t.data(), t.size() * sizeof(float),
                    hipMemcpyHostToDevice));
  return RXNN_OK;
}

rxnn_status rxnn_layer_info(const rxnn_layer* layer, int64_t* info7) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  if (!info7) return fail(RXNN_EINVAL, "info is NULL");
  const MapScalars& ms = layer->ms;
  const int64_t v[7] = {ms.P, ms.Q, ms.M, ms.N, ms.R, ms.C, ms.A};
  memcpy(info7, v, sizeof v);
  return RXNN_OK;
}

rxnn_status rxnn_layer_wmax(const rxnn_layer* layer, double* w_max) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  if (!w_max) return fail(RXNN_EINVAL, "w_max is NULL");
  DeviceGuard dg(layer->device);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layer's device");
  float v = 0.0f;
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(&v, layer->d_wmax, sizeof v, hipMemcpyDeviceToHost));
  *w_max = (double)v;
  return RXNN_OK;
}

void rxnn_free_layer(rxnn_layer* layer) {
  {
    std::lock_guard<std::mutex> g(g_mu);
    if (!layer || !g_live.count(layer)) return;
    g_live.erase(layer);
  }
  DeviceGuard dg(layer->device);
  (void)hipDeviceSynchronize();
  release_buffers(layer);
}

// ---- backward pass of re-training -------------------------------------------
namespace {

rxnn_status grow_bw(rxnn_layer* L, size_t bytes) {
  if (L->bw_bytes >= bytes) return RXNN_OK;
  if (L->bw_ws) HIP_TRY(hipFree(L->bw_ws));
  L->bw_ws = nullptr;
  L->bw_bytes = 0;
  if (hipMalloc((void**)&L->bw_ws, bytes) != hipSuccess) {
    (void)hipGetLastError();
    L->bw_ws = nullptr;
    return fail(RXNN_ENOMEM, "cannot allocate %zu bytes of backward scratch", bytes);
  }
  L->bw_bytes = bytes;
  return RXNN_OK;
}

// The DAC's input range: [0, x_max] for a quantising DAC, [0, inf) for the
// ideal one.
float dac_range(const rxnn_periph_params* pp) {
  return pp->dac_bits ? (float)pp->x_max : __builtin_huge_valf();
}

// dX and dW of a convolution whose shape has been checked against the layer.
rxnn_status bw_run(rxnn_layer* L, const rxnn_periph_params* periph, const rxnn_conv_desc& cd,
                   const float* W, const float* X, const float* dY, float* dX, float* dW,
                   hipStream_t s) {
  const int64_t ho = (cd.h + 2 * cd.pad - cd.kh) / cd.stride + 1;
  const int64_t wo = (cd.w + 2 * cd.pad - cd.kw) / cd.stride + 1;
  const int64_t Bv = (int64_t)cd.n * ho * wo, npix = (int64_t)cd.n * cd.h * cd.w;
  const int64_t P = L->ms.P, Q = L->ms.Q, khw = (int64_t)cd.kh * cd.kw;
  // the kernels index pixels, patch columns, the (tap, output) reduction and
  // an image's input planes with 32-bit integers, and launch one workgroup of
  // 256 threads per 64 x 64 tile
  const int64_t kLim = INT32_MAX - 64;
  const int64_t dx_tiles = ((npix + 63) / 64) * ((cd.c_in + 63) / 64);
  const int64_t dw_tiles = ((P + 63) / 64) * ((Q + 63) / 64);
  if (Bv > kLim || npix > kLim || P > kLim || khw * Q > kLim ||
      (int64_t)cd.c_in * cd.h * cd.w > kLim || dx_tiles >= ((int64_t)1 << 24) ||
      dw_tiles >= ((int64_t)1 << 24))
    return fail(RXNN_EUNSUPPORTED, "layer too large for the backward pass");
  if (Bv == 0 || (!dX && !dW)) return RXNN_OK;
  DeviceGuard dg(L->device);
  if (!dg.ok) return fail(RXNN_EHIP, "cannot select the layer's device");
  const float xr = dac_range(periph);
  if (dW) {
    const bool vec_ok = ((uintptr_t)X | (uintptr_t)dY | (uintptr_t)W) % 16 == 0;
    const BwPlan plan = bw_plan(cd, (int)P, (int)Q, vec_ok);
    if (plan.nsplit == 1) {
      ProfScope t("bw_dw", s);
      HIP_TRY(launch_bw_dw(cd, (int)P, (int)Q, xr, X, dY, W, L->ms, plan, dW, s));
    } else {
      rxnn_status st = grow_bw(L, (size_t)plan.nsplit * P * Q * sizeof(float));
      if (st) return st;
      {
        ProfScope t("bw_dw", s);
        HIP_TRY(launch_bw_dw(cd, (int)P, (int)Q, xr, X, dY, W, L->ms, plan, L->bw_ws, s));
      }
      ProfScope t("bw_reduce", s, (double)(plan.nsplit + 2) * P * Q * sizeof(float));
      HIP_TRY(launch_bw_reduce_w(L->bw_ws, plan.nsplit, W, P * Q, L->ms, dW, s));
    }
  }
  if (dX) {
    ProfScope t("bw_dx", s);
    HIP_TRY(launch_bw_dx(cd, (int)P, (int)Q, xr, X, dY, W, dX, s));
  }
  return RXNN_OK;
}

}  // namespace

extern "C" {

rxnn_status rxnn_fc_backward(const rxnn_layer* layer, const rxnn_periph_params* periph,
                             const float* W, const float* X, const float* dY, int64_t B,
                             float* dX, float* dW, void* stream) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  rxnn_layer* L = const_cast<rxnn_layer*>(layer);
  PeriphScalars ps;
  rxnn_status st = make_periph(periph, L->ms, &ps);
  if (st) return st;
  if (B < 0) return fail(RXNN_EINVAL, "B must be >= 0");
  if (!W || !X || !dY) return fail(RXNN_EINVAL, "W, X and dY must not be NULL");
  if (B > INT32_MAX || L->ms.P > INT32_MAX || L->ms.Q > INT32_MAX)
    return fail(RXNN_EUNSUPPORTED, "B too large for the backward pass");
  // the layer as the 1 x 1 convolution of B images of 1 x 1 pixels
  rxnn_conv_desc cd;
  cd.n = (int32_t)B;
  cd.c_in = (int32_t)L->ms.P;
  cd.h = cd.w = 1;
  cd.c_out = (int32_t)L->ms.Q;
  cd.kh = cd.kw = 1;
  cd.stride = 1;
  cd.pad = 0;
  return bw_run(L, periph, cd, W, X, dY, dX, dW, (hipStream_t)stream);
}

rxnn_status rxnn_conv_backward(const rxnn_layer* layer, const rxnn_periph_params* periph,
                               const rxnn_conv_desc* conv, const float* W, const float* X,
                               const float* dY, float* dX, float* dW, void* stream) {
  if (!live(layer)) return fail(RXNN_EINVAL, "invalid or released layer handle");
  rxnn_layer* L = const_cast<rxnn_layer*>(layer);
  PeriphScalars ps;
  rxnn_status st = make_periph(periph, L->ms, &ps);
  if (st) return st;
  if ((st = check_conv(L->ms, conv))) return st;
  if (!W || !X || !dY) return fail(RXNN_EINVAL, "W, X and dY must not be NULL");
  return bw_run(L, periph, *conv, W, X, dY, dX, dW, (hipStream_t)stream);
}

}  // extern "C"

rxnn_status rxnn_profile_enable(int32_t on) {
  if (on < 0 || on > 2) return fail(RXNN_EINVAL, "profile level must be 0, 1 or 2");
  std::lock_guard<std::mutex> g(g_mu);
  g_prof = on;
  return RXNN_OK;
}

rxnn_status rxnn_profile_reset(void) {
  std::vector<Pending> p;
  {
    std::lock_guard<std::mutex> g(g_mu);
    p.swap(g_pending);
    g_prof_tot.clear();
  }
  for (auto& e : p) {
    (void)hipEventSynchronize(e.b);
    (void)hipEventDestroy(e.a);
    (void)hipEventDestroy(e.b);
  }
  return RXNN_OK;
}

// Folds the pending event pairs into the per-kernel totals.
static rxnn_status fold_pending() {
  std::vector<Pending> p;
  {
    std::lock_guard<std::mutex> g(g_mu);
    p.swap(g_pending);
  }
  for (auto& e : p) {
    float ms = 0.0f;
    HIP_TRY(hipEventSynchronize(e.b));
    HIP_TRY(hipEventElapsedTime(&ms, e.a, e.b));
    (void)hipEventDestroy(e.a);
    (void)hipEventDestroy(e.b);
    std::lock_guard<std::mutex> g(g_mu);
    auto& t = g_prof_tot[e.name];
    t.ms += ms;
    t.count += 1;
    t.bytes += e.bytes;
  }
  return RXNN_OK;
}

rxnn_status rxnn_profile_read(const char* kernel, double* total_ms, int64_t* count) {
  if (!kernel || !total_ms || !count) return fail(RXNN_EINVAL, "NULL argument");
  rxnn_status st = fold_pending();
  if (st) return st;
  std::lock_guard<std::mutex> g(g_mu);
  auto it = g_prof_tot.find(kernel);
  *total_ms = it == g_prof_tot.end() ? 0.0 : it->second.ms;
  *count = it == g_prof_tot.end() ? 0 : it->second.count;
  return RXNN_OK;
}

rxnn_status rxnn_profile_bytes(const char* kernel, double* bytes) {
  if (!kernel || !bytes) return fail(RXNN_EINVAL, "NULL argument");
  rxnn_status st = fold_pending();
  if (st) return st;
  std::lock_guard<std::mutex> g(g_mu);
  auto it = g_prof_tot.find(kernel);
  *bytes = it == g_prof_tot.end() ? 0.0 : it->second.bytes;
  return RXNN_OK;
}

}  // extern "C"
