// Calibration from weights (Sec. 3.1, Eqs. gweighted and gsvd; App. B): the
// second moment E[k^T k] = W^T G W and mean E[k] = hbar W of the keys (or values)
// k = h W a projection W [d_model][d] produces (one KV head, d = 128, or a layer's
// KV heads side by side, d = d_kv) from layer inputs h with
// second moment G = E[h^T h] and mean hbar. Both are fp64 on the GPU; the
// eigenbasis, variances and widths follow on the host as for a data fit.
//
// Batched tiled fp64 products C_b = A_b B_b (64 x 64 output tiles, k-steps of
// 16 staged in LDS, 4 x 4 outputs per thread) with element strides, so the same
// kernel forms P_s = G_l W_s (A = G of the stream's layer, row-major) and then
// S_s = W_s^T P_s (A = W_s read transposed).
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace spectra_dev {

constexpr int WT = 64;   // output tile edge
constexpr int WKS = 16;  // k-step

template <typename TA, typename TB>
__global__ __launch_bounds__(256) void wgemm_kernel(WgemmArgs g) {
  __shared__ double As[WKS][WT + 1];  // [k][m]
  __shared__ double Bs[WKS][WT + 1];  // [k][n]
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.x * WT, n0 = blockIdx.y * WT, bt = blockIdx.z;
  const TA* A = reinterpret_cast<const TA*>(g.A) + (int64_t)(bt / g.a_div) * g.a_bs;
  const TB* B = reinterpret_cast<const TB*>(g.B) + (int64_t)bt * g.b_bs;
  double* C = g.C + (int64_t)bt * g.c_bs;
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  // element e of a 64 x 16 operand tile: the contiguous index runs fastest across
  // consecutive threads (k when the column stride is 1, else the row index)
  const bool a_k_fast = g.a_cs == 1, b_n_fast = g.b_cs == 1;
  for (int k0 = 0; k0 < g.K; k0 += WKS) {
#pragma unroll
    for (int r = 0; r < (WT * WKS) / 256; ++r) {
      const int e = tid + 256 * r;
      const int k = a_k_fast ? (e & (WKS - 1)) : (e >> 6);
      const int m = a_k_fast ? (e >> 4) : (e & (WT - 1));
      As[k][m] = (double)A[(int64_t)(m0 + m) * g.a_rs + (int64_t)(k0 + k) * g.a_cs];
    }
#pragma unroll
    for (int r = 0; r < (WT * WKS) / 256; ++r) {
      const int e = tid + 256 * r;
      const int n = b_n_fast ? (e & (WT - 1)) : (e >> 4);
      const int k = b_n_fast ? (e >> 6) : (e & (WKS - 1));
      Bs[k][n] = (double)B[(int64_t)(k0 + k) * g.b_rs + (int64_t)(n0 + n) * g.b_cs];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < WKS; ++k) {
      double a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[k][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[k][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fma(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) C[(int64_t)(m0 + ty + 16 * i) * g.c_rs + (n0 + tx + 16 * j)] = acc[i][j];
}

// mu_s[j] = sum_a hbar_l[a] W_s[a][j] (zero when hbar is null): one workgroup of
// 128 threads per stream, output columns j = tid, tid + 128, ..., ascending a.
__global__ __launch_bounds__(128) void wmean_kernel(const float* W, const double* hbar, int32_t d_model, int32_t d,
                                                    int32_t streams_per_layer, double* moments, int64_t mom_stride) {
  const int s = blockIdx.x;
  const float* Ws = W + (int64_t)s * d_model * d;
  const double* h = hbar ? hbar + (int64_t)(s / streams_per_layer) * d_model : nullptr;
  for (int j = threadIdx.x; j < d; j += 128) {
    double acc = 0.0;
    if (h)
      for (int a = 0; a < d_model; ++a) acc = __builtin_fma(h[a], (double)Ws[(int64_t)a * d + j], acc);
    moments[(int64_t)s * mom_stride + (int64_t)d * d + j] = acc;
  }
}

}  // namespace spectra_dev

namespace spectra {
using namespace spectra_dev;

// moments[s] = [W_s^T G W_s (d x d, row-major), hbar W_s (d)]; scratch holds
// P_s = G W_s for every stream ([n_streams][d_model][d] fp64). d a multiple of 64.
hipError_t launch_weights_moments(const float* W, const double* G, const double* hbar, int32_t d_model, int32_t d,
                                  int32_t n_streams, int32_t streams_per_layer, double* scratch, double* moments,
                                  int64_t mom_stride, hipStream_t st) {
  WgemmArgs p{};
  p.A = G;
  p.B = W;
  p.C = scratch;
  p.M = d_model;
  p.N = d;
  p.K = d_model;
  p.a_rs = d_model;
  p.a_cs = 1;
  p.a_bs = (int64_t)d_model * d_model;
  p.a_div = streams_per_layer;
  p.b_rs = d;
  p.b_cs = 1;
  p.b_bs = (int64_t)d_model * d;
  p.c_rs = d;
  p.c_bs = (int64_t)d_model * d;
  hipLaunchKernelGGL((wgemm_kernel<double, float>), dim3(d_model / WT, d / WT, n_streams), dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  WgemmArgs q{};
  q.A = W;  // A(i, k) = W_s[k][i]
  q.B = scratch;
  q.C = moments;
  q.M = d;
  q.N = d;
  q.K = d_model;
  q.a_rs = 1;
  q.a_cs = d;
  q.a_bs = (int64_t)d_model * d;
  q.a_div = 1;
  q.b_rs = d;
  q.b_cs = 1;
  q.b_bs = (int64_t)d_model * d;
  q.c_rs = d;
  q.c_bs = mom_stride;
  hipLaunchKernelGGL((wgemm_kernel<float, double>), dim3(d / WT, d / WT, n_streams), dim3(256), 0, st, q);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(wmean_kernel, dim3(n_streams), dim3(128), 0, st, W, hbar, d_model, d, streams_per_layer, moments,
                     mom_stride);
  return hipGetLastError();
}

}  // namespace spectra
