// Model generation: W -> G -> G' for every crossbar array of a layer
// (RxNN Sec. V-A generator steps 1-3; the network is the one of Sec. V-B).
//
// Formulation.  The paper reaches G' through one dense MN x MN inverse per
// tile (Eq. 12).  The same exact matrix is obtained here by sweeping the
// tile's rows from the one farthest from the sense amplifiers (tile row 0)
// to the last one, carrying a Norton equivalent of the rows already swept as
// seen from the N column wires:
//
//   c = w - Lambda b        c: the N column currents leaving the swept part,
//                           b: the N column-node voltages at the cut,
//                           Lambda (N x N, SPD): its admittance,
//                           w (N x M): its short-circuit currents, one column
//                           per source row (1 V on row k, 0 V elsewhere).
//
//   crossing one column-wire segment r_col:   (I + r_col Lambda) F = I,
//                                             Lambda <- F Lambda, w <- F w
//   adding row i:                             Lambda += Y_i, w[:, i] += Y_i 1
//     with Y_i = Z_i^-1 the admittance of row i seen from its column nodes,
//     Z_i = diag(1 / G[i, :]) + H,  H[j][x] = r_driver + r_row (min(j, x) + 1)
//     (the resistance the row wire shares between the paths from the driver
//     to devices j and x);
//   the sense resistors:                      Iout = (I + r_sense Lambda)^-1 w
//   and G'[k][j] = Iout[j][k].
//
// Only 1/G is ever inverted besides SPD systems, so every resistance may be
// zero (zero parasitics give G' = G).  Each SPD system is solved by
// Gauss-Jordan elimination without pivoting (safe for SPD matrices) in fp64,
// with the matrices held in registers: a 16 x 16 grid of threads, thread
// (ty, tx) owning rows ty + 16 i and columns tx + 16 j, and the pivot row and
// column broadcast through LDS, double buffered so that one barrier per pivot
// suffices.  One workgroup builds one array; arrays are independent.

#include "common.h"
#include "device_map.h"

namespace rxnn {
namespace {

constexpr int TG = 16;  // thread grid side
// Impedance of an open device: its admittance 1e-30 S is 25 orders of
// magnitude below g_min's, far below what an fp64 sum can see.
constexpr double kOpenOhm = 1e30;

__device__ __forceinline__ double device_conductance(const MapScalars& ms, const float* W,
                                                     double wmax, int r, int c, int a,
                                                     int i, int j) {
  return device_g(ms, W, wmax, ((int64_t)c * ms.R + r) * ms.A + a, i, j);
}

// Gauss-Jordan solve A Y = B in place on X = [A | B], A PS x PS SPD,
// B the remaining 2 PS columns; afterwards X[:, PS:] holds Y.
template <int PS>
__device__ __forceinline__ void gj_solve(double (&X)[PS / TG][3 * PS / TG], double* rowbuf,
                                         double* colbuf, int& parity, int ty, int tx) {
  constexpr int RI = PS / TG, CJ = 3 * PS / TG;
#pragma unroll
  for (int kb = 0; kb < RI; ++kb) {
#pragma unroll 1
    for (int kk = 0; kk < TG; ++kk) {
      double* rb = rowbuf + parity * 3 * PS;
      double* cb = colbuf + parity * PS;
      if (ty == kk) {
#pragma unroll
        for (int jj = 0; jj < CJ; ++jj) rb[tx + TG * jj] = X[kb][jj];
      }
      if (tx == kk) {
#pragma unroll
        for (int ii = 0; ii < RI; ++ii) cb[ty + TG * ii] = X[ii][kb];
      }
      __syncthreads();
      const int k = kb * TG + kk;
      const double inv = 1.0 / rb[k];
      double pc[CJ];
#pragma unroll
      for (int jj = 0; jj < CJ; ++jj) pc[jj] = rb[tx + TG * jj] * inv;
#pragma unroll
      for (int ii = 0; ii < RI; ++ii) {
        const double f = cb[ty + TG * ii];
        const bool pivot_row = (ii == kb) && (ty == kk);
#pragma unroll
        for (int jj = 0; jj < CJ; ++jj)
          X[ii][jj] = pivot_row ? pc[jj] : fma(-f, pc[jj], X[ii][jj]);
      }
      parity ^= 1;
    }
  }
}

// In-place Gauss-Jordan inversion of an SPD PS x PS matrix held as Z.
template <int PS>
__device__ __forceinline__ void gj_invert(double (&Z)[PS / TG][PS / TG], double* rowbuf,
                                          double* colbuf, int& parity, int ty, int tx) {
  constexpr int RI = PS / TG;
#pragma unroll
  for (int kb = 0; kb < RI; ++kb) {
#pragma unroll 1
    for (int kk = 0; kk < TG; ++kk) {
      double* rb = rowbuf + parity * 3 * PS;
      double* cb = colbuf + parity * PS;
      if (ty == kk) {
#pragma unroll
        for (int jj = 0; jj < RI; ++jj) rb[tx + TG * jj] = Z[kb][jj];
      }
      if (tx == kk) {
#pragma unroll
        for (int ii = 0; ii < RI; ++ii) cb[ty + TG * ii] = Z[ii][kb];
      }
      __syncthreads();
      const int k = kb * TG + kk;
      const double inv = 1.0 / rb[k];
#pragma unroll
      for (int ii = 0; ii < RI; ++ii) {
        const double f = cb[ty + TG * ii] * inv;
        const bool prow = (ii == kb) && (ty == kk);
#pragma unroll
        for (int jj = 0; jj < RI; ++jj) {
          const bool pcol = (jj == kb) && (tx == kk);
          const double rk = rb[tx + TG * jj];
          double v;
          if (prow && pcol) v = inv;
          else if (prow) v = Z[ii][jj] * inv;
          else if (pcol) v = -f;
          else v = fma(-f, rk, Z[ii][jj]);
          Z[ii][jj] = v;
        }
      }
      parity ^= 1;
    }
  }
}

template <int PS>
__global__ __launch_bounds__(TG* TG) void k_gprime_build(MapScalars ms, const float* __restrict__ W,
                                                         float* __restrict__ gpt, int64_t array0) {
  constexpr int RI = PS / TG, CJ = 3 * PS / TG, CZ = PS / TG;
  __shared__ double rowbuf[2 * 3 * PS];
  __shared__ double colbuf[2 * PS];
  const int tid = threadIdx.x, ty = tid / TG, tx = tid % TG;
  const int64_t arr = array0 + blockIdx.x;
  const int a = (int)(arr % ms.A);
  const int64_t rc = arr / ms.A;
  const int r = (int)(rc % ms.R), c = (int)(rc / ms.R);
  const double wmax = ms.wmax_fixed > 0.0f ? (double)ms.wmax_fixed : (double)*ms.d_wmax;
  const int M = ms.M, N = ms.N;
  int parity = 0;

  // X = [A | Lambda | w]; Lambda = 0, w = 0 before the first row.
  double X[RI][CJ];
#pragma unroll
  for (int ii = 0; ii < RI; ++ii)
#pragma unroll
    for (int jj = 0; jj < CJ; ++jj) X[ii][jj] = 0.0;
  double Z[RI][CZ];

#pragma unroll 1
  for (int i = 0; i < M; ++i) {
    if (i > 0 && ms.r_col > 0.0) {
      // F-step: Lambda <- (I + r_col Lambda)^-1 Lambda, w <- (I + r_col Lambda)^-1 w
#pragma unroll
      for (int ii = 0; ii < RI; ++ii)
#pragma unroll
        for (int jj = 0; jj < CZ; ++jj) {
          const int row = ty + TG * ii, col = tx + TG * jj;
          X[ii][jj] = (row == col ? 1.0 : 0.0) + ms.r_col * X[ii][CZ + jj];
        }
      gj_solve<PS>(X, rowbuf, colbuf, parity, ty, tx);
    }
    // Z_i: impedance of row i seen from its column nodes (identity on padding).
#pragma unroll
    for (int ii = 0; ii < RI; ++ii)
#pragma unroll
      for (int jj = 0; jj < CZ; ++jj) {
        const int row = ty + TG * ii, col = tx + TG * jj;
        double z;
        if (row < N && col < N) {
          z = ms.r_driver + ms.r_row * (double)(min(row, col) + 1);
          if (row == col) {
            // a device of zero conductance (a variation factor of 0) is an
            // open circuit: kOpenOhm stands for its infinite impedance
            const double g = device_conductance(ms, W, wmax, r, c, a, i, row);
            z += g > 0.0 ? 1.0 / g : kOpenOhm;
          }
        } else {
          z = (row == col) ? 1.0 : 0.0;
        }
        Z[ii][jj] = z;
      }
    gj_invert<PS>(Z, rowbuf, colbuf, parity, ty, tx);
    // Lambda += Y_i ; w[:, i] += Y_i 1 (sum over the real columns only)
#pragma unroll
    for (int ii = 0; ii < RI; ++ii) {
      double s = 0.0;
#pragma unroll
      for (int jj = 0; jj < CZ; ++jj) {
        const int col = tx + TG * jj;
        if (col < N) s += Z[ii][jj];
        X[ii][CZ + jj] += Z[ii][jj];
      }
#pragma unroll
      for (int off = TG / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, TG);
#pragma unroll
      for (int jj = 0; jj < CZ; ++jj) {
        const int col = tx + TG * jj;
        if (col == i) X[ii][2 * CZ + jj] += s;
      }
    }
  }

  if (ms.r_sense > 0.0) {
#pragma unroll
    for (int ii = 0; ii < RI; ++ii)
#pragma unroll
      for (int jj = 0; jj < CZ; ++jj) {
        const int row = ty + TG * ii, col = tx + TG * jj;
        X[ii][jj] = (row == col ? 1.0 : 0.0) + ms.r_sense * X[ii][CZ + jj];
      }
    gj_solve<PS>(X, rowbuf, colbuf, parity, ty, tx);
  }

  // G'^T[j][k] = Iout[j][k], stored [Np][Mp] with zero padding.
  float* out = gpt + arr * (int64_t)ms.Np * ms.Mp;
#pragma unroll
  for (int ii = 0; ii < RI; ++ii)
#pragma unroll
    for (int jj = 0; jj < CZ; ++jj) {
      const int j = ty + TG * ii, k = tx + TG * jj;
      if (j < ms.Np && k < ms.Mp)
        out[(int64_t)j * ms.Mp + k] = (j < N && k < M) ? (float)X[ii][2 * CZ + jj] : 0.0f;
    }
}

// max |W| as the bit pattern of a non-negative float (ordered like the
// value): wave then workgroup reduction, one atomic per workgroup
// out[0] = max |W| as fp32 bits (non-negative floats order like their bits),
// in one launch: every workgroup folds its maximum into out[1] and takes a
// ticket from out[2]; the workgroup with the last ticket moves the maximum to
// out[0].  Both words are left at zero for the next call (atomicInc wraps the
// ticket counter at the grid size; the last workgroup swaps the maximum out),
// so they only need clearing once, when the buffer is allocated.
__global__ __launch_bounds__(256) void k_absmax(const float* __restrict__ W, int64_t n,
                                                unsigned* out) {
  __shared__ unsigned wm[4];
  unsigned m = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // eight loads in flight per thread
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += 8 * stride) {
    unsigned v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t i = i0 + j * stride;
      v[j] = i < n ? __float_as_uint(fabsf(W[i])) : 0u;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) m = max(m, v[j]);
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    atomicMax(&out[1], max(max(wm[0], wm[1]), max(wm[2], wm[3])));
    __threadfence();
    if (atomicInc(&out[2], gridDim.x - 1) == gridDim.x - 1) {
      __threadfence();
      out[0] = atomicExch(&out[1], 0u);
    }
  }
}

// w_max of every layer of a batch in two launches.  k_wmax_init sets each
// layer's w_max to its fixed value or to 0; k_absmax_batch then gives layer l
// the blocks [start[l], start[l + 1]) (as many as its own reduction would
// launch), and each block folds its max |W| into w_max by one atomic max on
// the bits (|w| as unsigned bits orders as |w| does), without fences or a
// last-block step.
__global__ void k_wmax_init(const NdBatchLayer* __restrict__ layers, int n_layers) {
  const int l = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (l >= n_layers) return;
  const MapScalars& ms = layers[l].ms;
  unsigned* out = reinterpret_cast<unsigned*>(const_cast<float*>(ms.d_wmax));
  out[0] = ms.wmax_fixed > 0.0f ? __float_as_uint(ms.wmax_fixed) : 0u;
}

__global__ __launch_bounds__(256) void k_absmax_batch(const NdBatchLayer* __restrict__ layers,
                                                      const int* __restrict__ start,
                                                      int n_layers) {
  __shared__ unsigned wm[4];
  __shared__ int sl;
  // the layer whose block range holds this block: the ranges partition the
  // grid, so exactly one thread finds it (one round of loads, not a chain)
  for (int base = 0; base < n_layers; base += (int)blockDim.x) {
    const int t = base + (int)threadIdx.x;
    if (t < n_layers && start[t] <= (int)blockIdx.x && (int)blockIdx.x < start[t + 1]) sl = t;
  }
  __syncthreads();
  const int l = sl;
  const MapScalars& ms = layers[l].ms;
  if (ms.wmax_fixed > 0.0f) return;
  unsigned* out = reinterpret_cast<unsigned*>(const_cast<float*>(ms.d_wmax));
  const int b = (int)blockIdx.x - start[l], nb = start[l + 1] - start[l];
  const float* W = layers[l].W;
  const int64_t n = ms.P * ms.Q;
  unsigned m = 0;
  const int64_t stride = (int64_t)nb * blockDim.x;
  for (int64_t i0 = (int64_t)b * blockDim.x + threadIdx.x; i0 < n; i0 += 8 * stride) {
    unsigned v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t i = i0 + j * stride;
      v[j] = i < n ? __float_as_uint(fabsf(W[i])) : 0u;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) m = max(m, v[j]);
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) atomicMax(&out[0], max(max(wm[0], wm[1]), max(wm[2], wm[3])));
}

__global__ void k_fill_u32(unsigned* p, int64_t n, unsigned v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

}  // namespace

hipError_t launch_absmax(const float* W, int64_t n, unsigned* out, hipStream_t s) {
  hipLaunchKernelGGL(k_absmax, dim3((unsigned)absmax_blocks(n)), dim3(256), 0, s, W, n, out);
  return hipGetLastError();
}

int absmax_blocks(int64_t n) {
  int64_t blocks = (n + 2047) / 2048;   // at least 8 elements per thread
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  return (int)blocks;
}

hipError_t launch_absmax_batch(const NdBatchLayer* layers, const int* start, int n_layers,
                               int total_blocks, hipStream_t s) {
  hipLaunchKernelGGL(k_wmax_init, dim3((unsigned)((n_layers + 255) / 256)), dim3(256), 0, s, layers,
                     n_layers);
  hipLaunchKernelGGL(k_absmax_batch, dim3((unsigned)total_blocks), dim3(256), 0, s, layers, start,
                     n_layers);
  return hipGetLastError();
}

hipError_t launch_fill_u32(unsigned* p, int64_t n, unsigned v, hipStream_t s) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_gprime_build(const MapScalars& ms, const float* W, float* gpt, hipStream_t s) {
  const int side = ms.M > ms.N ? ms.M : ms.N;
  const int64_t n_arrays = (int64_t)ms.R * ms.C * ms.A;
  const int64_t chunk = 1 << 20;
  for (int64_t a0 = 0; a0 < n_arrays; a0 += chunk) {
    const unsigned nb = (unsigned)((n_arrays - a0) < chunk ? (n_arrays - a0) : chunk);
    if (side <= 16)
      hipLaunchKernelGGL(k_gprime_build<16>, dim3(nb), dim3(TG * TG), 0, s, ms, W, gpt, a0);
    else if (side <= 32)
      hipLaunchKernelGGL(k_gprime_build<32>, dim3(nb), dim3(TG * TG), 0, s, ms, W, gpt, a0);
    else
      hipLaunchKernelGGL(k_gprime_build<64>, dim3(nb), dim3(TG * TG), 0, s, ms, W, gpt, a0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace rxnn
