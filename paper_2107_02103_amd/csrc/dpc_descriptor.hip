// Backward of the descriptor D = T (T<)^T (DP Compress, Sec. II; the
// descriptor of the se_a model: D_i[m][n] = sum_k T_i[m][k] T_i[n][k] with
// n < M', T_i< the first M' rows of T_i).  Given dE/dD,
//
//   dE/dT[m][k] = sum_{n < M'} dE/dD[m][n] T[n][k]
//               + (m < M') sum_{m'} dE/dD[m'][m] T[m'][k].
//
// The kernels move 8 (4 M + M M' + 4 M) bytes per atom in float64 and do
// 2 M M' 4 FMA, far below the HBM ridge: they are bound by HBM bandwidth.
// descriptor_bwd_m16_kernel (float64 inputs, M' = 16, M <= 128, 16-byte
// aligned buffers) streams atoms through each wavefront with the next atom's
// loads in flight; descriptor_bwd_kernel serves every other shape.
//
// General kernel: one wavefront per atom.  The atom's T and dE/dD are read
// once, coalesced, into LDS (dE/dD rows padded to M' + 1 elements, so that
// the 16 rows read by one instruction fall into different banks); lane o of a
// pass then forms output element o = 4 m + k of the atom, and the outputs are
// written in flat order.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dpc.h"
#include "dpc_internal.h"

namespace {

constexpr int kLanes = 64;
constexpr size_t kMaxLds = 65536;   // LDS a workgroup may take without opting in

// LDS of one wavefront: T [m1][4] and dE/dD [m1][m2 + 1], in the compute type
template <typename TC>
constexpr size_t wave_bytes(int m1, int m2) {
  return ((size_t)m1 * 4 + (size_t)m1 * (m2 + 1)) * sizeof(TC);
}

// TT: type of T and dE/dD, TO: type of dE/dT, TC: arithmetic
template <typename TT, typename TO, typename TC>
__global__ __launch_bounds__(256) void descriptor_bwd_kernel(int nloc, int m1, int m2,
                                                             const TT* __restrict__ T,
                                                             const TT* __restrict__ dD,
                                                             TO* __restrict__ dT) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x >> 6) + wave);
  if (i >= nloc) return;
  TC* sT = reinterpret_cast<TC*>(smem + wave * wave_bytes<TC>(m1, m2));
  TC* sD = sT + m1 * 4;
  const int ldd = m2 + 1;
  const TT* Ti = T + (size_t)i * m1 * 4;
  const TT* Di = dD + (size_t)i * m1 * m2;
  for (int e = lane; e < m1 * 4; e += kLanes) sT[e] = (TC)__builtin_nontemporal_load(Ti + e);
  {
    // element e = m * m2 + n of dE/dD goes to row m, column n
    const int m_step = kLanes / m2, n_step = kLanes % m2;
    int m = lane / m2, n = lane % m2;
    for (int e = lane; e < m1 * m2; e += kLanes) {
      sD[m * ldd + n] = (TC)__builtin_nontemporal_load(Di + e);
      m += m_step;
      n += n_step;
      if (n >= m2) {
        n -= m2;
        ++m;
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  TO* dTi = dT + (size_t)i * m1 * 4;
  for (int o = lane; o < m1 * 4; o += kLanes) {
    const int m = o >> 2, k = o & 3;
    TC acc = (TC)0;
    for (int n = 0; n < m2; ++n) acc = fma(sD[m * ldd + n], sT[n * 4 + k], acc);
    if (m < m2) {
      for (int q = 0; q < m1; ++q) acc = fma(sD[q * ldd + m], sT[q * 4 + k], acc);
    }
    __builtin_nontemporal_store((TO)acc, dTi + o);
  }
}

// float64 inputs, M' = 16, M <= 128 (the workloads' descriptor): each
// wavefront walks atoms i, i + W, ... (W wavefronts in the grid) and loads
// the next atom's T and dE/dD into registers (16-byte loads, 16 or fewer per
// lane) while it computes the current one from LDS, so that HBM latency
// overlaps the arithmetic.  LDS per wavefront: T [M][4], dE/dD [M][18]
// (rows 144 bytes apart: the 16 rows read by 16 lanes start in different
// bank groups) and the partial sums of the second term [64][4].
constexpr int kFastM2 = 16, kFastMaxM1 = 128;
constexpr int kRowD = 18;                        // doubles per dE/dD row in LDS
constexpr int kLoadsT = 2 * kFastMaxM1 / 64;     // 16-byte chunks of T per lane
constexpr int kLoadsD = kFastMaxM1 * kFastM2 / 2 / 64;
__host__ __device__ constexpr size_t fast_wave_bytes(int m1) {
  return ((size_t)m1 * 4 + (size_t)m1 * kRowD + 64 * 4) * sizeof(double);
}

typedef double d2 __attribute__((ext_vector_type(2)));

template <typename TO>
__global__ __launch_bounds__(128) void descriptor_bwd_m16_kernel(int nloc, int m1,
                                                                 const double* __restrict__ T,
                                                                 const double* __restrict__ dD,
                                                                 TO* __restrict__ dT) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wpb = blockDim.x >> 6;
  double* sT = reinterpret_cast<double*>(smem + wave * fast_wave_bytes(m1));
  double* sD = sT + m1 * 4;
  double* sP = sD + m1 * kRowD;
  const int nT = 2 * m1, nD = m1 * kFastM2 / 2;   // 16-byte chunks per atom
  d2 rT[kLoadsT], rD[kLoadsD];
  auto fetch = [&](int i) __attribute__((always_inline)) {
    const d2* pT = reinterpret_cast<const d2*>(T + (size_t)i * m1 * 4);
    const d2* pD = reinterpret_cast<const d2*>(dD + (size_t)i * m1 * kFastM2);
#pragma unroll
    for (int c = 0; c < kLoadsT; ++c)
      if (lane + 64 * c < nT) rT[c] = __builtin_nontemporal_load(pT + lane + 64 * c);
#pragma unroll
    for (int c = 0; c < kLoadsD; ++c)
      if (lane + 64 * c < nD) rD[c] = __builtin_nontemporal_load(pD + lane + 64 * c);
  };
  const int stride = gridDim.x * wpb;
  int i = __builtin_amdgcn_readfirstlane(blockIdx.x * wpb + wave);
  if (i < nloc) fetch(i);
  for (; i < nloc; i += stride) {
    // this atom's registers into LDS, then the next atom's loads
#pragma unroll
    for (int c = 0; c < kLoadsT; ++c)
      if (lane + 64 * c < nT) *reinterpret_cast<d2*>(sT + 2 * (lane + 64 * c)) = rT[c];
#pragma unroll
    for (int c = 0; c < kLoadsD; ++c) {
      const int u = lane + 64 * c;                 // chunk u: row u / 8, columns 2 (u % 8) + 0, 1
      if (u < nD) *reinterpret_cast<d2*>(sD + (u >> 3) * kRowD + 2 * (u & 7)) = rD[c];
    }
    if (i + stride < nloc) fetch(i + stride);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // second term: lane (m = lane % 16, quarter q = lane / 16) sums rows
    // m' = q, q + 4, ... of dE/dD[m'][m] T[m'][k]; the quarters' sums are
    // added in the first pass below
    {
      const int m = lane & 15, q = lane >> 4;
      double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
      for (int r = q; r < m1; r += 4) {
        const double w = sD[r * kRowD + m];
        const d2 t01 = *reinterpret_cast<const d2*>(sT + 4 * r);
        const d2 t23 = *reinterpret_cast<const d2*>(sT + 4 * r + 2);
        a0 = fma(w, t01.x, a0);
        a1 = fma(w, t01.y, a1);
        a2 = fma(w, t23.x, a2);
        a3 = fma(w, t23.y, a3);
      }
      *reinterpret_cast<d2*>(sP + 4 * lane) = d2{a0, a1};
      *reinterpret_cast<d2*>(sP + 4 * lane + 2) = d2{a2, a3};
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // first term: lane m forms row m of dE/dT, all four k
    TO* dTi = dT + (size_t)i * m1 * 4;
    for (int m = lane; m < m1; m += 64) {
      double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
#pragma unroll
      for (int n = 0; n < kFastM2; n += 2) {
        const d2 w = *reinterpret_cast<const d2*>(sD + m * kRowD + n);
        const d2 t01 = *reinterpret_cast<const d2*>(sT + 4 * n);
        const d2 t23 = *reinterpret_cast<const d2*>(sT + 4 * n + 2);
        const d2 u01 = *reinterpret_cast<const d2*>(sT + 4 * n + 4);
        const d2 u23 = *reinterpret_cast<const d2*>(sT + 4 * n + 6);
        a0 = fma(w.x, t01.x, a0);
        a1 = fma(w.x, t01.y, a1);
        a2 = fma(w.x, t23.x, a2);
        a3 = fma(w.x, t23.y, a3);
        a0 = fma(w.y, u01.x, a0);
        a1 = fma(w.y, u01.y, a1);
        a2 = fma(w.y, u23.x, a2);
        a3 = fma(w.y, u23.y, a3);
      }
      if (m < kFastM2) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const d2 p01 = *reinterpret_cast<const d2*>(sP + 4 * (m + 16 * q));
          const d2 p23 = *reinterpret_cast<const d2*>(sP + 4 * (m + 16 * q) + 2);
          a0 += p01.x;
          a1 += p01.y;
          a2 += p23.x;
          a3 += p23.y;
        }
      }
      if constexpr (sizeof(TO) == 8) {
        __builtin_nontemporal_store(d2{a0, a1}, reinterpret_cast<d2*>(dTi + 4 * m));
        __builtin_nontemporal_store(d2{a2, a3}, reinterpret_cast<d2*>(dTi + 4 * m) + 1);
      } else {
        typedef float f4 __attribute__((ext_vector_type(4)));
        __builtin_nontemporal_store(f4{(float)a0, (float)a1, (float)a2, (float)a3},
                                    reinterpret_cast<f4*>(dTi + 4 * m));
      }
    }
    // the LDS of this atom is rewritten in the next iteration
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

template <typename TO>
int launch_m16(hipStream_t s, int nloc, int m1, const void* T, const void* dD, void* dT) {
  const size_t wb = fast_wave_bytes(m1);
  const int waves = 2;
  int dev = 0, ncu = 256;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  // workgroups that fit in LDS at once, a few rounds of them
  const int per_cu = (int)(160 * 1024 / (waves * wb));
  const int blocks = (nloc + waves - 1) / waves;
  const int grid = blocks < ncu * per_cu ? blocks : ncu * per_cu;
  (void)hipGetLastError();  // report only what this launch raises
  hipLaunchKernelGGL((descriptor_bwd_m16_kernel<TO>), dim3(grid), dim3(64 * waves), waves * wb, s,
                     nloc, m1, (const double*)T, (const double*)dD, (TO*)dT);
  return dpc_internal_launch_status();
}

template <typename TT, typename TO, typename TC>
int launch(hipStream_t s, int nloc, int m1, int m2, const void* T, const void* dD, void* dT) {
  const size_t wb = wave_bytes<TC>(m1, m2);
  if (wb > kMaxLds) return DPC_ENOTSUP;
  const int waves = wb * 4 <= kMaxLds ? 4 : (wb * 2 <= kMaxLds ? 2 : 1);
  const dim3 grid((nloc + waves - 1) / waves), block(kLanes * waves);
  (void)hipGetLastError();  // report only what this launch raises
  hipLaunchKernelGGL((descriptor_bwd_kernel<TT, TO, TC>), grid, block, waves * wb, s, nloc, m1, m2,
                     (const TT*)T, (const TT*)dD, (TO*)dT);
  return dpc_internal_launch_status();
}

}  // namespace

extern "C" int dpc_descriptor_bwd(void* stream, dpc_dtype dtype, int nloc, int m1, int m2,
                                  const void* T, const void* dE_dD, void* dE_dT) {
  if (dtype != DPC_F64 && dtype != DPC_F32 && dtype != DPC_F32_ACC64) return DPC_EINVAL;
  if (nloc < 0 || m1 < 1 || m2 < 1 || m2 > m1) return DPC_EINVAL;
  if (m1 > DPC_MAX_M1) return DPC_ENOTSUP;
  if (nloc == 0) return DPC_OK;
  if (!T || !dE_dD || !dE_dT) return DPC_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // 16-byte loads and stores of T, dE/dD and dE/dT need 16-byte alignment
  const bool fast = dtype != DPC_F32 && m2 == kFastM2 && m1 <= kFastMaxM1 &&
                    reinterpret_cast<uintptr_t>(T) % 16 == 0 &&
                    reinterpret_cast<uintptr_t>(dE_dD) % 16 == 0 &&
                    reinterpret_cast<uintptr_t>(dE_dT) % 16 == 0;
  if (fast && dtype == DPC_F64) return launch_m16<double>(s, nloc, m1, T, dE_dD, dE_dT);
  if (fast) return launch_m16<float>(s, nloc, m1, T, dE_dD, dE_dT);
  switch (dtype) {
    case DPC_F64: return launch<double, double, double>(s, nloc, m1, m2, T, dE_dD, dE_dT);
    case DPC_F32: return launch<float, float, float>(s, nloc, m1, m2, T, dE_dD, dE_dT);
    default: return launch<double, float, double>(s, nloc, m1, m2, T, dE_dD, dE_dT);
  }
}
