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
// caller's handle.  Everything else is four streaming kernels, one pass over
// the activations each: bias + tanh (layer 1), bias + tanh + residual
// (layer 2), layer 3 fused with the energy dot product and the first
// backward scaling (h_3 is never stored), and (1 - t^2) (w_out + e) for the
// two remaining layers, where e = delta - w_out accumulates in the backward
// GEMMs so that the constant delta_3 = w_out is never materialised.  Row-major X [N][c] is column-major [c][N], so
// Z^T = W^T H^T is dgemm(N, N, out, N, in, W, ld out, H, ld in) and
// dH^T = W dZ^T is dgemm(T, N, in, N, out, W, ld out, dZ, ld out).
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <cstdint>

#include "dpc.h"
#include "dpc_internal.h"

namespace {

// tanh(x) = expm1(2x) / (expm1(2x) + 2): expm1 keeps its relative accuracy
// near 0, so the quotient does too, and it costs about two thirds of the
// library tanh here.  |x| is capped at 20, where tanh(x) rounds to +-1 in
// float64 and expm1(2x) is still finite; NaN passes through.
__device__ inline double tanh_e(double x) {
  const double c = x > 20.0 ? 20.0 : (x < -20.0 ? -20.0 : x);
  const double y = expm1(2.0 * c);
  return y / (y + 2.0);
}


// Grid-stride walk over the element pairs (e, e + 1), e = 0, 2, 4, ... of a
// row-major [n][w] array, tracking the column of e without a division per
// step.  nw = n * w may be odd: the last element then goes alone.
struct PairWalk {
  int64_t e, step, nw;
  int col, w, step_col;
  __device__ PairWalk(int64_t nw_, int w_) : nw(nw_), w(w_) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    step = 2 * (int64_t)gridDim.x * blockDim.x;
    e = 2 * t;
    col = (int)(e % w);
    step_col = (int)(step % w);
  }
  __device__ bool ok() const { return e < nw; }
  __device__ bool pair() const { return e + 1 < nw; }
  __device__ int col1() const { return col + 1 == w ? 0 : col + 1; }
  __device__ void next() {
    e += step;
    col += step_col;
    if (col >= w) col -= w;
  }
};

__device__ inline double2 ld2(const double* p) { return *reinterpret_cast<const double2*>(p); }
__device__ inline void st2(double* p, double a, double b) { *reinterpret_cast<double2*>(p) = make_double2(a, b); }

// layer 1: t1 = tanh(z + b1)
__global__ __launch_bounds__(256) void layer1_kernel(int64_t nw, int w, const double* __restrict__ z,
                                                     const double* __restrict__ b, double* __restrict__ t1) {
  for (PairWalk it(nw, w); it.ok(); it.next()) {
    if (it.pair()) {
      const double2 v = ld2(z + it.e);
      st2(t1 + it.e, tanh_e(v.x + b[it.col]), tanh_e(v.y + b[it.col1()]));
    } else {
      t1[it.e] = tanh_e(z[it.e] + b[it.col]);
    }
  }
}

// layer 2: t2 = tanh(z + b2), h2 = t1 + t2
__global__ __launch_bounds__(256) void layer2_kernel(int64_t nw, int w, const double* __restrict__ z,
                                                     const double* __restrict__ b,
                                                     const double* __restrict__ t1, double* __restrict__ t2,
                                                     double* __restrict__ h2) {
  for (PairWalk it(nw, w); it.ok(); it.next()) {
    if (it.pair()) {
      const double2 v = ld2(z + it.e), u = ld2(t1 + it.e);
      const double a = tanh_e(v.x + b[it.col]), c = tanh_e(v.y + b[it.col1()]);
      st2(t2 + it.e, a, c);
      st2(h2 + it.e, u.x + a, u.y + c);
    } else {
      const double a = tanh_e(z[it.e] + b[it.col]);
      t2[it.e] = a;
      h2[it.e] = t1[it.e] + a;
    }
  }
}

// layer 3 and the energy, one wavefront per atom:
//   t3 = tanh(z + b3), E = (h2 + t3) . w_out + b_out (fixed-order sum),
//   and, when dz is given, dz = (1 - t3^2) w_out (dz may alias z)
__global__ __launch_bounds__(256) void layer3_energy_kernel(int n, int w, const double* z,
                                                            const double* __restrict__ b,
                                                            const double* __restrict__ h2,
                                                            const double* __restrict__ wout, double bout,
                                                            double* __restrict__ E, double* dz) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (i >= n) return;
  const size_t row = (size_t)i * w;
  double acc = 0.0;
  for (int c = lane; c < w; c += 64) {
    const double t = tanh_e(z[row + c] + b[c]);
    acc = fma(h2[row + c] + t, wout[c], acc);
    if (dz) dz[row + c] = (1.0 - t * t) * wout[c];
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t u = __builtin_bit_cast(uint64_t, acc);
    const int lo = __builtin_amdgcn_ds_bpermute(((lane ^ off) & 63) << 2, (int)(uint32_t)u);
    const int hi = __builtin_amdgcn_ds_bpermute(((lane ^ off) & 63) << 2, (int)(uint32_t)(u >> 32));
    acc += __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
  }
  if (lane == 0) E[i] = acc + bout;
}

// dz = (1 - t^2) (w_out + e), where e = delta - w_out
__global__ __launch_bounds__(256) void tanh_grad_kernel(int64_t nw, int w, const double* __restrict__ t,
                                                        const double* __restrict__ wout,
                                                        const double* __restrict__ e,
                                                        double* __restrict__ dz) {
  for (PairWalk it(nw, w); it.ok(); it.next()) {
    if (it.pair()) {
      const double2 tv = ld2(t + it.e), ev = ld2(e + it.e);
      st2(dz + it.e, (1.0 - tv.x * tv.x) * (wout[it.col] + ev.x),
          (1.0 - tv.y * tv.y) * (wout[it.col1()] + ev.y));
    } else {
      dz[it.e] = (1.0 - t[it.e] * t[it.e]) * (wout[it.col] + e[it.e]);
    }
  }
}

dim3 stream_grid(int64_t nw) {
  const int64_t b = (nw / 2 + 255) / 256;
  return dim3((unsigned)(b < 8192 ? (b > 0 ? b : 1) : 8192));
}

}  // namespace

extern "C" size_t dpc_fitting_workspace_bytes(int nloc, int width) {
  if (nloc < 0 || width < 1) return 0;
  const size_t nw = (size_t)nloc * width;
  return 5 * (nw + (nw & 1)) * sizeof(double);   // each array 16-byte aligned
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
  // alpha and beta live on the host: host pointer mode for this call, the
  // caller's mode restored on every return
  struct ModeGuard {
    rocblas_handle h;
    rocblas_pointer_mode old = rocblas_pointer_mode_host;
    bool set = false;
    ~ModeGuard() {
      if (set) rocblas_set_pointer_mode(h, old);
    }
  } mode{hb};
  if (rocblas_get_pointer_mode(hb, &mode.old) != rocblas_status_success ||
      rocblas_set_pointer_mode(hb, rocblas_pointer_mode_host) != rocblas_status_success)
    return DPC_EHIP;
  mode.set = true;
  const int64_t nw = (int64_t)nloc * w;
  double* ws = static_cast<double*>(workspace);
  const int64_t np = nw + (nw & 1);   // array pitch: keeps every array 16-byte aligned
  double* t1 = ws;            // tanh outputs of layers 1 and 2
  double* t2 = ws + np;
  double* h2 = ws + 2 * np;   // h_2 = t_1 + t_2
  double* z = ws + 3 * np;    // pre-activations, then dz
  double* e = ws + 4 * np;    // delta_l - w_out in the backward pass
  const double one = 1.0, zero = 0.0;
  (void)hipGetLastError();
  auto gemm_fwd = [&](const double* W, int in, const double* H) {
    return rocblas_dgemm(hb, rocblas_operation_none, rocblas_operation_none, w, nloc, in, &one, W, w,
                         H, in, &zero, z, w) == rocblas_status_success;
  };
  // dH^T = W dZ^T (+ beta C): the data gradient of one layer
  auto gemm_bwd = [&](const double* W, int in, const double* beta, double* C) {
    return rocblas_dgemm(hb, rocblas_operation_transpose, rocblas_operation_none, in, nloc, w, &one, W,
                         w, z, w, beta, C, in) == rocblas_status_success;
  };
  if (!gemm_fwd(net->W[0], nin, D)) return DPC_EHIP;
  hipLaunchKernelGGL(layer1_kernel, stream_grid(nw), dim3(256), 0, s, nw, w, z, net->b[0], t1);
  if (!gemm_fwd(net->W[1], w, t1)) return DPC_EHIP;
  hipLaunchKernelGGL(layer2_kernel, stream_grid(nw), dim3(256), 0, s, nw, w, z, net->b[1], t1, t2, h2);
  if (!gemm_fwd(net->W[2], w, h2)) return DPC_EHIP;
  // h_3 is used only by the energy: it is never stored; dz_3 replaces z_3
  hipLaunchKernelGGL(layer3_energy_kernel, dim3((nloc + 3) / 4), dim3(256), 0, s, nloc, w, z, net->b[2],
                     h2, net->w_out, net->b_out, E, dE_dD ? z : nullptr);
  if (dE_dD) {
    // delta_2 = w_out + W_3 dz_3; e holds delta - w_out so that the constant
    // delta_3 = w_out is never stored
    if (!gemm_bwd(net->W[2], w, &zero, e)) return DPC_EHIP;
    hipLaunchKernelGGL(tanh_grad_kernel, stream_grid(nw), dim3(256), 0, s, nw, w, t2, net->w_out, e, z);
    if (!gemm_bwd(net->W[1], w, &one, e)) return DPC_EHIP;   // delta_1 - w_out
    hipLaunchKernelGGL(tanh_grad_kernel, stream_grid(nw), dim3(256), 0, s, nw, w, t1, net->w_out, e, z);
    if (!gemm_bwd(net->W[0], nin, &zero, dE_dD)) return DPC_EHIP;
  }
  return dpc_internal_launch_status();
}
