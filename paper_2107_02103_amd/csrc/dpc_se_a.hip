// Compressed se_a descriptor kernels for CDNA4 (gfx950).
//
// DP Compress (arXiv:2107.02103), Sec. II: the embedding net is replaced by a
// table of quintic Hermite pieces and fused with S = G^T R~ (here T), which is
// evaluated only over valid neighbours; D = T (T<)^T.  The backward kernel
// maps dE/dT to dE/dR~ through the polynomial and its derivative.
//
// Forward mapping: one wavefront per atom, lanes = channels (channel m is
// handled by lane m % 64).  The neighbour list is scanned 64 slots at a time:
// each lane locates the interval of its slot, a ballot gives the valid slots,
// and the wave then walks the valid slots in order with the slot's row of R~
// and its interval offset uniform across the wave.  Coefficients of the
// current interval stay in registers until the interval changes (neighbours
// are distance-sorted, so consecutive slots often share an interval).
//
// Backward mapping: one wavefront per atom, lanes = neighbour slots, a loop
// over the channels with dE/dT_i[m][:] uniform across the wave.  Each lane
// keeps v_k = sum_m dT[m][k] g_m and u_k = sum_m dT[m][k] g'_m, then
// dE/dR~[k] = v_k + (k == 0) sum_k' u_k' R~[k'], which regroups
// sum_m g'_m sum_k' dT[m][k'] R~[k'] without changing its value.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "dpc.h"

namespace {

constexpr int kWaves = 4;  // wavefronts per workgroup

struct PairRange {          // one ordered type pair's table, as the kernels see it
  double lo, d1, d2;
  int L1, L2;
  int offset;               // element offset of the pair's coefficients
  int pad;
};

struct Geo {
  int nloc, nnei, ntypes, m1, m2;
  int blk_end[DPC_MAX_TYPES];   // slot index one past the end of each sel block
  PairRange pr[DPC_MAX_TYPES * DPC_MAX_TYPES];
};

__device__ __forceinline__ int block_of(const Geo& g, int j) {
  int b = 0;
#pragma unroll
  for (int k = 0; k < DPC_MAX_TYPES - 1; ++k) b += (k < g.ntypes - 1 && j >= g.blk_end[k]) ? 1 : 0;
  return b;
}

// Interval of x in one pair's table (see dpc_range in dpc.h).  Always float64.
__device__ __forceinline__ void locate(const PairRange& P, double x, int& l, double& t,
                                       bool& clamped) {
  const double x_up = P.lo + (double)P.L1 * P.d1;
  const double x_end = x_up + (double)P.L2 * P.d2;
  clamped = false;
  if (x < x_up) {
    double q = floor((x - P.lo) / P.d1);
    q = fmin(fmax(q, 0.0), (double)(P.L1 - 1));
    l = (int)q;
    t = x - (P.lo + q * P.d1);
  } else if (x < x_end) {
    double q = floor((x - x_up) / P.d2);
    q = fmin(fmax(q, 0.0), (double)(P.L2 - 1));
    l = P.L1 + (int)q;
    t = x - (x_up + q * P.d2);
  } else {
    l = P.L1 + P.L2 - 1;
    t = P.d2;
    clamped = true;
  }
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <typename TA, typename TI>
__device__ __forceinline__ TA fma_acc(TI a, TI b, TA c) {
  return fma((TA)a, (TA)b, c);
}

// ---------------------------------------------------------------------------
// forward: T and D
// ---------------------------------------------------------------------------
template <typename TI, typename TA, int CPL>
__global__ __launch_bounds__(64 * kWaves) void se_a_fwd_kernel(
    const Geo g, const TI* __restrict__ coeff, const int* __restrict__ atype,
    const int* __restrict__ nlist, const TI* __restrict__ em, TA* __restrict__ T,
    TA* __restrict__ D) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i = __builtin_amdgcn_readfirstlane(blockIdx.x * kWaves + wave);
  if (i >= g.nloc) return;
  const int nnei = g.nnei, m1 = g.m1, m2 = g.m2;
  TA* sT = reinterpret_cast<TA*>(smem) + wave * m2 * 4;                       // [m2][4]
  TI* st = reinterpret_cast<TI*>(reinterpret_cast<TA*>(smem) + kWaves * m2 * 4) + wave * 64;
  int* so = reinterpret_cast<int*>(reinterpret_cast<TI*>(reinterpret_cast<TA*>(smem) +
                                                          kWaves * m2 * 4) + kWaves * 64) +
            wave * 64;

  const int ai = __builtin_amdgcn_readfirstlane(atype[i]);
  if (ai < 0 || ai >= g.ntypes) {  // invalid type: the atom's outputs become NaN
    const TA nan = (TA)NAN;
    for (int e = lane; e < m1 * 4; e += 64) T[(size_t)i * m1 * 4 + e] = nan;
    for (int e = lane; e < m1 * m2; e += 64) D[(size_t)i * m1 * m2 + e] = nan;
    return;
  }
  const TI* emi = em + (size_t)i * nnei * 4;
  const int* nli = nlist + (size_t)i * nnei;

  TA acc[CPL][4];
  TI c[CPL][6];
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[h][k] = (TA)0;
#pragma unroll
    for (int q = 0; q < 6; ++q) c[h][q] = (TI)0;
  }
  int cur = -1;

  for (int base = 0; base < nnei; base += 64) {
    const int j = base + lane;
    bool valid = false;
    TI tt = (TI)0;
    int off = 0;
    if (j < nnei && nli[j] >= 0) {
      const PairRange& P = g.pr[ai * g.ntypes + block_of(g, j)];
      int l;
      double t;
      bool cl;
      locate(P, (double)emi[(size_t)j * 4], l, t, cl);
      off = P.offset + l * 6 * m1;
      tt = (TI)t;
      valid = true;
    }
    uint64_t mask = __ballot(valid);
    st[lane] = tt;
    so[lane] = off;
    wave_sync();
    while (mask) {
      const int jj = __builtin_ctzll(mask);
      mask &= mask - 1;
      const TI t = st[jj];
      const int o = __builtin_amdgcn_readfirstlane(so[jj]);
      const TI* r = emi + (size_t)(base + jj) * 4;
      const TI r0 = r[0], r1 = r[1], r2 = r[2], r3 = r[3];
      if (o != cur) {
        cur = o;
#pragma unroll
        for (int h = 0; h < CPL; ++h) {
          const int m = lane + 64 * h;
#pragma unroll
          for (int q = 0; q < 6; ++q) c[h][q] = (m < m1) ? coeff[o + q * m1 + m] : (TI)0;
        }
      }
#pragma unroll
      for (int h = 0; h < CPL; ++h) {
        TI gv = c[h][5];
        gv = fma(gv, t, c[h][4]);
        gv = fma(gv, t, c[h][3]);
        gv = fma(gv, t, c[h][2]);
        gv = fma(gv, t, c[h][1]);
        gv = fma(gv, t, c[h][0]);
        acc[h][0] = fma_acc<TA>(gv, r0, acc[h][0]);
        acc[h][1] = fma_acc<TA>(gv, r1, acc[h][1]);
        acc[h][2] = fma_acc<TA>(gv, r2, acc[h][2]);
        acc[h][3] = fma_acc<TA>(gv, r3, acc[h][3]);
      }
    }
    wave_sync();
  }

  // T rows and the first m2 rows for D
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
    const int m = lane + 64 * h;
    if (m < m1) {
      TA* Tm = T + ((size_t)i * m1 + m) * 4;
#pragma unroll
      for (int k = 0; k < 4; ++k) Tm[k] = acc[h][k];
    }
    if (m < m2) {
#pragma unroll
      for (int k = 0; k < 4; ++k) sT[m * 4 + k] = acc[h][k];
    }
  }
  wave_sync();
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
    const int m = lane + 64 * h;
    if (m < m1) {
      TA* Dm = D + ((size_t)i * m1 + m) * m2;
      for (int n = 0; n < m2; ++n) {
        TA s = acc[h][0] * sT[n * 4 + 0];
        s = fma(acc[h][1], sT[n * 4 + 1], s);
        s = fma(acc[h][2], sT[n * 4 + 2], s);
        s = fma(acc[h][3], sT[n * 4 + 3], s);
        Dm[n] = s;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// backward: dE/dR~
// ---------------------------------------------------------------------------
template <typename TI, typename TA>
__global__ __launch_bounds__(64 * kWaves) void se_a_bwd_kernel(
    const Geo g, const TI* __restrict__ coeff, const int* __restrict__ atype,
    const int* __restrict__ nlist, const TI* __restrict__ em, const TI* __restrict__ dT,
    TA* __restrict__ dR) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i = __builtin_amdgcn_readfirstlane(blockIdx.x * kWaves + wave);
  if (i >= g.nloc) return;
  const int nnei = g.nnei, m1 = g.m1;
  const int ai = __builtin_amdgcn_readfirstlane(atype[i]);
  TA* dRi = dR + (size_t)i * nnei * 4;
  if (ai < 0 || ai >= g.ntypes) {  // invalid type: the atom's outputs become NaN
    for (int e = lane; e < nnei * 4; e += 64) dRi[e] = (TA)NAN;
    return;
  }
  const TI* emi = em + (size_t)i * nnei * 4;
  const int* nli = nlist + (size_t)i * nnei;
  const TI* dTi = dT + (size_t)i * m1 * 4;

  for (int base = 0; base < nnei; base += 64) {
    const int j = base + lane;
    TA o0 = 0, o1 = 0, o2 = 0, o3 = 0;
    if (j < nnei && nli[j] >= 0) {
      const TI r0 = emi[(size_t)j * 4 + 0], r1 = emi[(size_t)j * 4 + 1];
      const TI r2 = emi[(size_t)j * 4 + 2], r3 = emi[(size_t)j * 4 + 3];
      const PairRange& P = g.pr[ai * g.ntypes + block_of(g, j)];
      int l;
      double td;
      bool cl;
      locate(P, (double)r0, l, td, cl);
      const TI t = (TI)td;
      const TI* c = coeff + P.offset + l * 6 * m1;
      TA v0 = 0, v1 = 0, v2 = 0, v3 = 0, u0 = 0, u1 = 0, u2 = 0, u3 = 0;
      for (int m = 0; m < m1; ++m) {
        const TI c0 = c[m], c1 = c[m1 + m], c2 = c[2 * m1 + m];
        const TI c3 = c[3 * m1 + m], c4 = c[4 * m1 + m], c5 = c[5 * m1 + m];
        // value and derivative of the quintic by a joint Horner scheme
        TI p = c5, d = c5;
        p = fma(p, t, c4);
        d = fma(d, t, p);
        p = fma(p, t, c3);
        d = fma(d, t, p);
        p = fma(p, t, c2);
        d = fma(d, t, p);
        p = fma(p, t, c1);
        d = fma(d, t, p);
        p = fma(p, t, c0);
        const TI* dm = dTi + m * 4;
        const TI a0 = dm[0], a1 = dm[1], a2 = dm[2], a3 = dm[3];
        v0 = fma_acc<TA>(a0, p, v0);
        v1 = fma_acc<TA>(a1, p, v1);
        v2 = fma_acc<TA>(a2, p, v2);
        v3 = fma_acc<TA>(a3, p, v3);
        u0 = fma_acc<TA>(a0, d, u0);
        u1 = fma_acc<TA>(a1, d, u1);
        u2 = fma_acc<TA>(a2, d, u2);
        u3 = fma_acc<TA>(a3, d, u3);
      }
      if (cl) u0 = u1 = u2 = u3 = 0;
      o0 = v0 + (u0 * (TA)r0 + u1 * (TA)r1 + u2 * (TA)r2 + u3 * (TA)r3);
      o1 = v1;
      o2 = v2;
      o3 = v3;
    }
    if (j < nnei) {
      TA* out = dRi + (size_t)j * 4;
      out[0] = o0;
      out[1] = o1;
      out[2] = o2;
      out[3] = o3;
    }
  }
}

thread_local hipError_t g_last_hip = hipSuccess;

int launch_status() {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return DPC_OK;
  g_last_hip = e;
  return DPC_EHIP;
}

bool dtype_ok(int dt) { return dt == DPC_F64 || dt == DPC_F32 || dt == DPC_F32_ACC64; }

// Host-side validation shared by both passes; fills the kernel geometry.
int make_geo(int nloc, int ntypes, const int* sel, int m1, int m2, const dpc_range* ranges,
             Geo* g) {
  if (nloc < 0 || ntypes < 1 || !sel || !ranges || m1 < 1 || m2 < 1 || m2 > m1)
    return DPC_EINVAL;
  if (ntypes > DPC_MAX_TYPES || m1 > DPC_MAX_M1) return DPC_ENOTSUP;
  int64_t nnei = 0;
  for (int b = 0; b < ntypes; ++b) {
    if (sel[b] < 0) return DPC_EINVAL;
    nnei += sel[b];
    g->blk_end[b] = (int)nnei;
  }
  if (nnei < 1 || nnei > (1 << 20)) return DPC_EINVAL;
  for (int b = ntypes; b < DPC_MAX_TYPES; ++b) g->blk_end[b] = (int)nnei;
  for (int p = 0; p < ntypes * ntypes; ++p) {
    const dpc_range& r = ranges[p];
    if (!(std::isfinite(r.lo) && std::isfinite(r.d1) && std::isfinite(r.d2) && r.d1 > 0 &&
          r.d2 > 0 && r.L1 >= 1 && r.L2 >= 1 && r.offset >= 0))
      return DPC_ERANGE;
    if (r.offset + (r.L1 + r.L2) * 6 * (int64_t)m1 >= (int64_t(1) << 31)) return DPC_ENOTSUP;
    PairRange& q = g->pr[p];
    q.lo = r.lo;
    q.d1 = r.d1;
    q.d2 = r.d2;
    q.L1 = (int)r.L1;
    q.L2 = (int)r.L2;
    q.offset = (int)r.offset;
    q.pad = 0;
  }
  g->nloc = nloc;
  g->nnei = (int)nnei;
  g->ntypes = ntypes;
  g->m1 = m1;
  g->m2 = m2;
  return DPC_OK;
}

template <typename TI, typename TA>
int launch_fwd(hipStream_t s, const Geo& g, const void* coeff, const int* atype, const int* nlist,
               const void* em, void* T, void* D) {
  const dim3 grid((g.nloc + kWaves - 1) / kWaves), block(64 * kWaves);
  const size_t shm = (size_t)kWaves * g.m2 * 4 * sizeof(TA) + kWaves * 64 * (sizeof(TI) + 4);
  const int cpl = (g.m1 + 63) / 64;
  (void)hipGetLastError();  // report only what this launch raises
  auto args = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, block, shm, s, g, (const TI*)coeff, atype, nlist,
                       (const TI*)em, (TA*)T, (TA*)D);
  };
  switch (cpl) {
    case 1: args(se_a_fwd_kernel<TI, TA, 1>); break;
    case 2: args(se_a_fwd_kernel<TI, TA, 2>); break;
    case 3: args(se_a_fwd_kernel<TI, TA, 3>); break;
    default: args(se_a_fwd_kernel<TI, TA, 4>); break;
  }
  return launch_status();
}

template <typename TI, typename TA>
int launch_bwd(hipStream_t s, const Geo& g, const void* coeff, const int* atype, const int* nlist,
               const void* em, const void* dT, void* dR) {
  const dim3 grid((g.nloc + kWaves - 1) / kWaves), block(64 * kWaves);
  (void)hipGetLastError();  // report only what this launch raises
  hipLaunchKernelGGL((se_a_bwd_kernel<TI, TA>), grid, block, 0, s, g, (const TI*)coeff, atype,
                     nlist, (const TI*)em, (const TI*)dT, (TA*)dR);
  return launch_status();
}

}  // namespace

extern "C" const char* dpc_last_hip_error(void) { return hipGetErrorString(g_last_hip); }

extern "C" int dpc_se_a_tab_fwd(void* stream, dpc_dtype dtype, int nloc, int ntypes,
                                const int* sel, int m1, int m2, const dpc_range* ranges,
                                const void* coeff, const int* atype, const int* nlist,
                                const void* em, void* T, void* D) {
  if (!dtype_ok(dtype)) return DPC_EINVAL;
  Geo g;
  const int st = make_geo(nloc, ntypes, sel, m1, m2, ranges, &g);
  if (st != DPC_OK) return st;
  if (nloc == 0) return DPC_OK;
  if (!coeff || !atype || !nlist || !em || !T || !D) return DPC_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (dtype) {
    case DPC_F64: return launch_fwd<double, double>(s, g, coeff, atype, nlist, em, T, D);
    case DPC_F32: return launch_fwd<float, float>(s, g, coeff, atype, nlist, em, T, D);
    default: return launch_fwd<float, double>(s, g, coeff, atype, nlist, em, T, D);
  }
}

extern "C" int dpc_se_a_tab_bwd(void* stream, dpc_dtype dtype, int nloc, int ntypes,
                                const int* sel, int m1, const dpc_range* ranges,
                                const void* coeff, const int* atype, const int* nlist,
                                const void* em, const void* dE_dT, void* dE_dem) {
  if (!dtype_ok(dtype)) return DPC_EINVAL;
  Geo g;
  const int st = make_geo(nloc, ntypes, sel, m1, 1, ranges, &g);
  if (st != DPC_OK) return st;
  if (nloc == 0) return DPC_OK;
  if (!coeff || !atype || !nlist || !em || !dE_dT || !dE_dem) return DPC_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (dtype) {
    case DPC_F64: return launch_bwd<double, double>(s, g, coeff, atype, nlist, em, dE_dT, dE_dem);
    case DPC_F32: return launch_bwd<float, float>(s, g, coeff, atype, nlist, em, dE_dT, dE_dem);
    default: return launch_bwd<float, double>(s, g, coeff, atype, nlist, em, dE_dT, dE_dem);
  }
}
