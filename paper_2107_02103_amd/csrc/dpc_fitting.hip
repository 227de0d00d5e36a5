// Fitting net: descriptor D_i -> atomic energy E_i and dE/dD_i (DP Compress,
// Sec. II: a fully connected network maps the descriptor to E^i; Sec. III:
// widths (240, 240, 240)).  Read as
//   h_1 = tanh(x W_1 + b_1),  h_l = h_{l-1} + tanh(h_{l-1} W_l + b_l) (l = 2, 3),
//   E = h_3 . w_out + b_out,
// with x = D_i flattened row-major.  Backward (delta_l = dE/dh_l):
//   delta_3 = w_out,  delta_{l-1} = delta_l + W_l ((1 - t_l^2) delta_l),
//   dE/dx = W_1 ((1 - t_1^2) delta_1).
//
// The layer products are plain GEMMs with atoms as the long dimension
// (N x 1600 by 1600 x 240 and 240 x 240, float64) and go to rocBLAS on the
// caller's handle; bias, tanh, residual, the energy dot product and the
// backward's (1 - t^2) scaling are the kernels below, each one pass over the
// activations.  Row-major X [N][c] is column-major [c][N], so
// Z^T = W^T H^T is dgemm(N, N, out, N, in, W, ld out, H, ld in) and
// dH^T = W dZ^T is dgemm(T, N, in, N, out, W, ld out, dZ, ld out).
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <cstdint>

#include "dpc.h"
#include "dpc_internal.h"

namespace {

// t = tanh(z + b) over [n][w]; h = t (first layer) or h += t (residual)
__global__ __launch_bounds__(256) void bias_tanh_kernel(int64_t n, int w, const double* __restrict__ z,
                                                        const double* __restrict__ b,
                                                        double* __restrict__ t, double* __restrict__ h,
                                                        int residual) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n * w; e += stride) {
    const double v = tanh(z[e] + b[e % w]);
    t[e] = v;
    h[e] = residual ? h[e] + v : v;
  }
}

// E[i] = h[i] . w_out + b_out, one wavefront per atom, fixed-order sum
__global__ __launch_bounds__(256) void energy_kernel(int n, int w, const double* __restrict__ h,
                                                     const double* __restrict__ wout, double bout,
                                                     double* __restrict__ E) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (i >= n) return;
  double acc = 0.0;
  for (int c = lane; c < w; c += 64) acc = fma(h[(size_t)i * w + c], wout[c], acc);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t u = __builtin_bit_cast(uint64_t, acc);
    const int lo = __builtin_amdgcn_ds_bpermute(((lane ^ off) & 63) << 2, (int)(uint32_t)u);
    const int hi = __builtin_amdgcn_ds_bpermute(((lane ^ off) & 63) << 2, (int)(uint32_t)(u >> 32));
    acc += __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
  }
  if (lane == 0) E[i] = acc + bout;
}

// delta[i][c] = w_out[c]
__global__ __launch_bounds__(256) void delta_init_kernel(int64_t n, int w, const double* __restrict__ wout,
                                                         double* __restrict__ delta) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n * w; e += stride)
    delta[e] = wout[e % w];
}

// dz = (1 - t^2) delta
__global__ __launch_bounds__(256) void tanh_grad_kernel(int64_t n, const double* __restrict__ t,
                                                        const double* __restrict__ delta,
                                                        double* __restrict__ dz) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride)
    dz[e] = (1.0 - t[e] * t[e]) * delta[e];
}

dim3 stream_grid(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return dim3((unsigned)(b < 8192 ? (b > 0 ? b : 1) : 8192));
}

}  // namespace

extern "C" size_t dpc_fitting_workspace_bytes(int nloc, int width) {
  if (nloc < 0 || width < 1) return 0;
  return (size_t)6 * nloc * width * sizeof(double);
}

extern "C" int dpc_fitting_fwd_bwd(void* stream, void* blas, int nloc, const dpc_fitting_net* net,
                                   const double* D, void* workspace, size_t workspace_bytes,
                                   double* E, double* dE_dD) {
  if (!net || nloc < 0) return DPC_EINVAL;
  const int nin = net->n_in, w = net->width;
  if (nin < 1 || w < 1) return DPC_EINVAL;
  for (int l = 0; l < 3; ++l)
    if (!net->W[l] || !net->b[l]) return DPC_EINVAL;
  if (!net->w_out) return DPC_EINVAL;
  if (nloc == 0) return DPC_OK;
  if (!blas || !D || !workspace || !E) return DPC_EINVAL;
  if (workspace_bytes < dpc_fitting_workspace_bytes(nloc, w)) return DPC_EINVAL;
  if ((uintptr_t)workspace % 16) return DPC_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  rocblas_handle hb = static_cast<rocblas_handle>(blas);
  if (rocblas_set_stream(hb, s) != rocblas_status_success) return DPC_EHIP;
  const int64_t nw = (int64_t)nloc * w;
  double* ws = static_cast<double*>(workspace);
  double* t[3] = {ws, ws + nw, ws + 2 * nw};   // tanh outputs of the three layers
  double* h = ws + 3 * nw;                      // h_2, then h_3
  double* z = ws + 4 * nw;                      // pre-activations, then dz
  double* delta = ws + 5 * nw;
  const double one = 1.0, zero = 0.0;
  (void)hipGetLastError();
  auto gemm_fwd = [&](const double* W, int in, const double* H) {
    return rocblas_dgemm(hb, rocblas_operation_none, rocblas_operation_none, w, nloc, in, &one, W, w,
                         H, in, &zero, z, w) == rocblas_status_success;
  };
  // layer 1: t_1 = h_1
  if (!gemm_fwd(net->W[0], nin, D)) return DPC_EHIP;
  hipLaunchKernelGGL(bias_tanh_kernel, stream_grid(nw), dim3(256), 0, s, (int64_t)nloc, w, z, net->b[0],
                     t[0], t[0], 0);
  // layer 2: h_2 = h_1 + t_2 (h_1 = t_1 copied into h by the first residual step)
  if (!gemm_fwd(net->W[1], w, t[0])) return DPC_EHIP;
  if (hipMemcpyAsync(h, t[0], nw * sizeof(double), hipMemcpyDeviceToDevice, s) != hipSuccess)
    return DPC_EHIP;
  hipLaunchKernelGGL(bias_tanh_kernel, stream_grid(nw), dim3(256), 0, s, (int64_t)nloc, w, z, net->b[1],
                     t[1], h, 1);
  // layer 3: h_3 = h_2 + t_3
  if (!gemm_fwd(net->W[2], w, h)) return DPC_EHIP;
  hipLaunchKernelGGL(bias_tanh_kernel, stream_grid(nw), dim3(256), 0, s, (int64_t)nloc, w, z, net->b[2],
                     t[2], h, 1);
  hipLaunchKernelGGL(energy_kernel, dim3((nloc + 3) / 4), dim3(256), 0, s, nloc, w, h, net->w_out,
                     net->b_out, E);
  if (dE_dD) {
    hipLaunchKernelGGL(delta_init_kernel, stream_grid(nw), dim3(256), 0, s, (int64_t)nloc, w, net->w_out,
                       delta);
    for (int l = 2; l >= 1; --l) {   // delta_{l-1} = delta_l + W_l dz_l
      hipLaunchKernelGGL(tanh_grad_kernel, stream_grid(nw), dim3(256), 0, s, nw, t[l], delta, z);
      if (rocblas_dgemm(hb, rocblas_operation_transpose, rocblas_operation_none, w, nloc, w, &one,
                        net->W[l], w, z, w, &one, delta, w) != rocblas_status_success)
        return DPC_EHIP;
    }
    hipLaunchKernelGGL(tanh_grad_kernel, stream_grid(nw), dim3(256), 0, s, nw, t[0], delta, z);
    if (rocblas_dgemm(hb, rocblas_operation_transpose, rocblas_operation_none, nin, nloc, w, &one,
                      net->W[0], w, z, w, &zero, dE_dD, nin) != rocblas_status_success)
      return DPC_EHIP;
  }
  return dpc_internal_launch_status();
}
