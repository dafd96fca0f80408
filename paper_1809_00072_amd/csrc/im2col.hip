// Convolution as a matrix product over unrolled patches (RxNN Sec. VI: the
// crossbar evaluation runs on Caffe's conv-as-GEMM), fused with the DAC.
//
// Patch matrix row bv = (n H_out + oy) W_out + ox, column
// k = (ci kh + ky) kw + kx (the order of weight.reshape(c_out, -1)); pixels
// outside the input are 0.  With a quantising DAC the kernel writes the DAC
// code of every element as one byte (the evaluation kernel turns codes into
// row voltages through its table); with the ideal DAC it writes the fp32
// input values.  Rows are ldk elements apart.

#include "common.h"

namespace rxnn {
namespace {

template <bool CODES>
__global__ __launch_bounds__(256) void k_dac_im2col(rxnn_conv_desc cd, float s_in, int levels,
                                                    const float* __restrict__ X,
                                                    void* __restrict__ out, int64_t ldk,
                                                    int64_t Bv, int Kdim, int ho, int wo) {
  const int64_t total = Bv * (int64_t)Kdim;
  const int khw = cd.kh * cd.kw;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t bv = e / Kdim;
    const int k = (int)(e % Kdim);
    const int ci = k / khw, kr = k % khw, ky = kr / cd.kw, kx = kr % cd.kw;
    const int64_t img = bv / ((int64_t)ho * wo);
    const int pix = (int)(bv % ((int64_t)ho * wo));
    const int oy = pix / wo, ox = pix % wo;
    const int iy = oy * cd.stride - cd.pad + ky, ix = ox * cd.stride - cd.pad + kx;
    float x = 0.0f;
    if (iy >= 0 && iy < cd.h && ix >= 0 && ix < cd.w)
      x = X[((img * cd.c_in + ci) * cd.h + iy) * (int64_t)cd.w + ix];
    if (CODES) {
      const float t = rintf(x * s_in);
      const int code = (int)fminf(fmaxf(t, 0.0f), (float)levels);
      ((unsigned char*)out)[bv * ldk + k] = (unsigned char)code;
    } else {
      ((float*)out)[bv * ldk + k] = x;
    }
  }
}

}  // namespace

hipError_t launch_dac_im2col(const rxnn_conv_desc& cd, const PeriphScalars& ps, const float* X,
                             void* out, bool codes, int64_t ldk, hipStream_t s) {
  const int ho = (cd.h + 2 * cd.pad - cd.kh) / cd.stride + 1;
  const int wo = (cd.w + 2 * cd.pad - cd.kw) / cd.stride + 1;
  const int64_t Bv = (int64_t)cd.n * ho * wo;
  const int Kdim = cd.c_in * cd.kh * cd.kw;
  int64_t blocks = (Bv * Kdim + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (codes)
    hipLaunchKernelGGL(k_dac_im2col<true>, dim3((unsigned)blocks), dim3(256), 0, s, cd,
                       ps.dac_s_in, ps.dac_levels, X, out, ldk, Bv, Kdim, ho, wo);
  else
    hipLaunchKernelGGL(k_dac_im2col<false>, dim3((unsigned)blocks), dim3(256), 0, s, cd,
                       ps.dac_s_in, ps.dac_levels, X, out, ldk, Bv, Kdim, ho, wo);
  return hipGetLastError();
}

}  // namespace rxnn
