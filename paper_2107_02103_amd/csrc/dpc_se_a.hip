// Compressed se_a descriptor kernels for CDNA4 (gfx950).
//
// DP Compress (arXiv:2107.02103), Sec. II: the embedding net is replaced by a
// table of quintic Hermite pieces and fused with S = G^T R~ (here T), which is
// evaluated only over valid neighbours; D = T (T<)^T.  The backward kernel
// maps dE/dT to dE/dR~ through the polynomial and its derivative.
//
// Both kernels: one wavefront per atom, lanes = channels.  Lane l owns the
// CPL consecutive channels CPL*l .. CPL*l + CPL - 1, so that one 16-byte load
// brings the coefficient of t^q for all of them (table rows are padded to a
// multiple of 4 channels).  The neighbour list is first compacted, 64 slots
// at a time, into per-wave records {t, interval offset, slot} in LDS; the wave
// then walks the records with the record, the R~ row (scalar loads) and the
// interval uniform across the wave.  The coefficients of the current interval
// stay in registers until the interval changes: neighbours are distance
// sorted, so consecutive records often share an interval.
//
// Forward: acc[k] += g_m(t) * R~[k] per channel, then T and D = T (T<)^T.
// Backward: for every record each lane forms its share of
//   dE/dR~[k] = sum_m dT[m][k] g_m + (k == 0) sum_m g'_m sum_k' dT[m][k'] R~[k']
// over its channels; the shares of a batch of records are summed across
// lanes through LDS (a transpose: each lane adds up a strip of the batch).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "dpc.h"

namespace {

constexpr int kWaves = 4;      // wavefronts per workgroup (one atom each)
constexpr int kSeg = 128;      // neighbour slots compacted per segment
constexpr int kBatch = 8;      // records per cross-lane reduction in the backward pass

struct PairRange {             // one ordered type pair's table, as the kernels see it
  double lo, d1, d2;
  int L1, L2;
  int offset;                  // element offset of the pair's coefficients
  int pad;
};

struct Geo {
  int nloc, nnei, ntypes, m1, m2, ld;
  int blk_end[DPC_MAX_TYPES];  // slot index one past the end of each sel block
  PairRange pr[DPC_MAX_TYPES * DPC_MAX_TYPES];
};

struct Rec {                   // one valid neighbour, as staged in LDS
  double t;                    // offset from the left node of its interval
  int off;                     // element offset of the interval's coefficient rows
  int slot;                    // neighbour slot; bit 30 set = beyond the table (clamped)
};
constexpr int kClamped = 1 << 30;

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

__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

// Compact the valid slots [s0, s1) of atom i into records; returns their count.
// Invalid slots get a zero row in `zero_out` when it is non-null.
template <typename TI, typename TA>
__device__ __forceinline__ int compact(const Geo& g, int ai, const int* nli, const TI* emi,
                                       int s0, int s1, Rec* rec, TA* zero_out, int lane) {
  int n = 0;
  for (int base = s0; base < s1; base += 64) {
    const int j = base + lane;
    bool valid = false;
    Rec r;
    if (j < s1) {
      valid = nli[j] >= 0;
      if (valid) {
        const PairRange& P = g.pr[ai * g.ntypes + block_of(g, j)];
        int l;
        bool cl;
        locate(P, (double)emi[(size_t)j * 4], l, r.t, cl);
        r.off = P.offset + l * 6 * g.ld;
        r.slot = j | (cl ? kClamped : 0);
      } else if (zero_out) {
        TA* o = zero_out + (size_t)j * 4;
        o[0] = o[1] = o[2] = o[3] = (TA)0;
      }
    }
    const uint64_t mask = __ballot(valid);
    if (valid) rec[n + lanes_below(mask)] = r;
    n += __popcll(mask);
  }
  return n;
}

// Coefficients of t^q (q = 0..5) for the lane's CPL channels of one interval.
template <typename TI, int CPL>
__device__ __forceinline__ void load_coef(const TI* __restrict__ rows, int ld, int c0,
                                          TI (&cf)[6][CPL]) {
#pragma unroll
  for (int q = 0; q < 6; ++q) {
#pragma unroll
    for (int h = 0; h < CPL; ++h) cf[q][h] = rows[q * ld + c0 + h];
  }
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
  const int nnei = g.nnei, m1 = g.m1, m2 = g.m2, ld = g.ld;
  Rec* rec = reinterpret_cast<Rec*>(smem) + wave * kSeg;
  TA* sT = reinterpret_cast<TA*>(reinterpret_cast<Rec*>(smem) + kWaves * kSeg) + wave * m2 * 4;

  const int ai = __builtin_amdgcn_readfirstlane(atype[i]);
  if (ai < 0 || ai >= g.ntypes) {  // invalid type: the atom's outputs become NaN
    const TA nan = (TA)NAN;
    for (int e = lane; e < m1 * 4; e += 64) T[(size_t)i * m1 * 4 + e] = nan;
    for (int e = lane; e < m1 * m2; e += 64) D[(size_t)i * m1 * m2 + e] = nan;
    return;
  }
  const TI* emi = em + (size_t)i * nnei * 4;
  const int* nli = nlist + (size_t)i * nnei;
  const int c0 = min(lane * CPL, ld - CPL);   // lanes past the last channel reload a valid row

  TA acc[CPL][4];
  TI cf[6][CPL];
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[h][k] = (TA)0;
  }
#pragma unroll
  for (int q = 0; q < 6; ++q) {
#pragma unroll
    for (int h = 0; h < CPL; ++h) cf[q][h] = (TI)0;
  }
  int cur = -1;

  for (int s0 = 0; s0 < nnei; s0 += kSeg) {
    const int n = compact<TI, TA>(g, ai, nli, emi, s0, min(nnei, s0 + kSeg), rec, nullptr, lane);
    wave_sync();
    for (int e = 0; e < n; ++e) {
      const Rec r = rec[e];
      const int off = __builtin_amdgcn_readfirstlane(r.off);
      const int slot = __builtin_amdgcn_readfirstlane(r.slot) & (kClamped - 1);
      const TI* R = emi + (size_t)slot * 4;
      const TI r0 = R[0], r1 = R[1], r2 = R[2], r3 = R[3];
      if (off != cur) {
        cur = off;
        load_coef<TI, CPL>(coeff + off, ld, c0, cf);
      }
      const TI t = (TI)r.t;
#pragma unroll
      for (int h = 0; h < CPL; ++h) {
        TI gv = cf[5][h];
        gv = fma(gv, t, cf[4][h]);
        gv = fma(gv, t, cf[3][h]);
        gv = fma(gv, t, cf[2][h]);
        gv = fma(gv, t, cf[1][h]);
        gv = fma(gv, t, cf[0][h]);
        const TA ga = (TA)gv;
        acc[h][0] = fma(ga, (TA)r0, acc[h][0]);
        acc[h][1] = fma(ga, (TA)r1, acc[h][1]);
        acc[h][2] = fma(ga, (TA)r2, acc[h][2]);
        acc[h][3] = fma(ga, (TA)r3, acc[h][3]);
      }
    }
    wave_sync();
  }

  // T rows and the first m2 rows for D
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
    const int m = lane * CPL + h;
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
    const int m = lane * CPL + h;
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
// Sum over lanes of the per-lane shares of a batch of nb <= kBatch records:
// red[b][lane][k] holds lane `lane`'s share of dE/dR~[k] for record b (only
// the nl lanes that own channels).  Lane L adds up, for record b = L / 8 and
// the component pair kk = (L / 4) % 2, every fourth owning lane starting at
// L % 4; four lanes then combine their sums.
template <typename TA>
__device__ __forceinline__ void reduce_batch(const TA* red, int nl, int nb, const Rec* rec,
                                             TA* dRi, int lane) {
  const int b = lane >> 3, kk = (lane >> 2) & 1, x = lane & 3;
  TA s0 = 0, s1 = 0;
  if (b < nb) {
    const TA* base = red + (size_t)b * nl * 4 + 2 * kk;
    for (int l2 = x; l2 < nl; l2 += 4) {
      s0 += base[l2 * 4];
      s1 += base[l2 * 4 + 1];
    }
  }
  s0 += __shfl_xor(s0, 1);
  s1 += __shfl_xor(s1, 1);
  s0 += __shfl_xor(s0, 2);
  s1 += __shfl_xor(s1, 2);
  if (b < nb && x == 0) {
    const int slot = rec[b].slot & (kClamped - 1);
    TA* o = dRi + (size_t)slot * 4 + 2 * kk;
    o[0] = s0;
    o[1] = s1;
  }
}

template <typename TI, typename TA, int CPL>
__global__ __launch_bounds__(64 * kWaves) void se_a_bwd_kernel(
    const Geo g, const TI* __restrict__ coeff, const int* __restrict__ atype,
    const int* __restrict__ nlist, const TI* __restrict__ em, const TI* __restrict__ dT,
    TA* __restrict__ dR) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i = __builtin_amdgcn_readfirstlane(blockIdx.x * kWaves + wave);
  if (i >= g.nloc) return;
  const int nnei = g.nnei, m1 = g.m1, ld = g.ld;
  const int nl = (m1 + CPL - 1) / CPL;          // lanes that own channels
  Rec* rec = reinterpret_cast<Rec*>(smem) + wave * kSeg;
  TA* red = reinterpret_cast<TA*>(reinterpret_cast<Rec*>(smem) + kWaves * kSeg) +
            (size_t)wave * kBatch * nl * 4;

  const int ai = __builtin_amdgcn_readfirstlane(atype[i]);
  TA* dRi = dR + (size_t)i * nnei * 4;
  if (ai < 0 || ai >= g.ntypes) {  // invalid type: the atom's outputs become NaN
    for (int e = lane; e < nnei * 4; e += 64) dRi[e] = (TA)NAN;
    return;
  }
  const TI* emi = em + (size_t)i * nnei * 4;
  const int* nli = nlist + (size_t)i * nnei;
  const int c0 = min(lane * CPL, ld - CPL);
  const bool owner = lane < nl;

  // dE/dT of the lane's channels (zero for lanes past the last channel)
  TA dt[CPL][4];
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
    const int m = lane * CPL + h;
#pragma unroll
    for (int k = 0; k < 4; ++k) dt[h][k] = (m < m1) ? (TA)dT[((size_t)i * m1 + m) * 4 + k] : (TA)0;
  }
  TI cf[6][CPL];
#pragma unroll
  for (int q = 0; q < 6; ++q) {
#pragma unroll
    for (int h = 0; h < CPL; ++h) cf[q][h] = (TI)0;
  }
  int cur = -1;

  for (int s0 = 0; s0 < nnei; s0 += kSeg) {
    const int n = compact<TI, TA>(g, ai, nli, emi, s0, min(nnei, s0 + kSeg), rec, dRi, lane);
    wave_sync();
    for (int e0 = 0; e0 < n; e0 += kBatch) {
      const int nb = min(kBatch, n - e0);
      for (int b = 0; b < nb; ++b) {
        const Rec r = rec[e0 + b];
        const int off = __builtin_amdgcn_readfirstlane(r.off);
        const int sf = __builtin_amdgcn_readfirstlane(r.slot);
        const TI* R = emi + (size_t)(sf & (kClamped - 1)) * 4;
        const TI r0 = R[0], r1 = R[1], r2 = R[2], r3 = R[3];
        if (off != cur) {
          cur = off;
          load_coef<TI, CPL>(coeff + off, ld, c0, cf);
        }
        const TI t = (TI)r.t;
        TA p0 = 0, p1 = 0, p2 = 0, p3 = 0;
        const bool clamped = (sf & kClamped) != 0;
#pragma unroll
        for (int h = 0; h < CPL; ++h) {
          // value and derivative of the quintic by a joint Horner scheme
          TI v = cf[5][h], d = cf[5][h];
          v = fma(v, t, cf[4][h]);
          d = fma(d, t, v);
          v = fma(v, t, cf[3][h]);
          d = fma(d, t, v);
          v = fma(v, t, cf[2][h]);
          d = fma(d, t, v);
          v = fma(v, t, cf[1][h]);
          d = fma(d, t, v);
          v = fma(v, t, cf[0][h]);
          const TA gv = (TA)v;
          const TA gd = clamped ? (TA)0 : (TA)d;
          TA w = dt[h][0] * (TA)r0;
          w = fma(dt[h][1], (TA)r1, w);
          w = fma(dt[h][2], (TA)r2, w);
          w = fma(dt[h][3], (TA)r3, w);
          p0 = fma(dt[h][0], gv, fma(gd, w, p0));
          p1 = fma(dt[h][1], gv, p1);
          p2 = fma(dt[h][2], gv, p2);
          p3 = fma(dt[h][3], gv, p3);
        }
        if (owner) {
          TA* o = red + ((size_t)b * nl + lane) * 4;
          o[0] = p0;
          o[1] = p1;
          o[2] = p2;
          o[3] = p3;
        }
      }
      wave_sync();
      reduce_batch<TA>(red, nl, nb, rec + e0, dRi, lane);
      wave_sync();
    }
  }
}

bool dtype_ok(int dt) { return dt == DPC_F64 || dt == DPC_F32 || dt == DPC_F32_ACC64; }

thread_local hipError_t g_last_hip = hipSuccess;

int launch_status() {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return DPC_OK;
  g_last_hip = e;
  return DPC_EHIP;
}

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
  const int ld = DPC_TABLE_LD(m1);
  for (int p = 0; p < ntypes * ntypes; ++p) {
    const dpc_range& r = ranges[p];
    if (!(std::isfinite(r.lo) && std::isfinite(r.d1) && std::isfinite(r.d2) && r.d1 > 0 &&
          r.d2 > 0 && r.L1 >= 1 && r.L2 >= 1 && r.offset >= 0))
      return DPC_ERANGE;
    if (r.offset + (r.L1 + r.L2) * 6 * (int64_t)ld >= (int64_t(1) << 31)) return DPC_ENOTSUP;
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
  g->ld = ld;
  return DPC_OK;
}

// Channels per lane: 1 (m1 <= 64), 2 (m1 <= 128) or 4 (m1 <= 256).
int channels_per_lane(int m1) { return m1 <= 64 ? 1 : (m1 <= 128 ? 2 : 4); }

template <typename TI, typename TA>
int launch_fwd(hipStream_t s, const Geo& g, const void* coeff, const int* atype, const int* nlist,
               const void* em, void* T, void* D) {
  const dim3 grid((g.nloc + kWaves - 1) / kWaves), block(64 * kWaves);
  const size_t shm = (size_t)kWaves * kSeg * sizeof(Rec) + (size_t)kWaves * g.m2 * 4 * sizeof(TA);
  (void)hipGetLastError();  // report only what this launch raises
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, block, shm, s, g, (const TI*)coeff, atype, nlist,
                       (const TI*)em, (TA*)T, (TA*)D);
  };
  switch (channels_per_lane(g.m1)) {
    case 1: go(se_a_fwd_kernel<TI, TA, 1>); break;
    case 2: go(se_a_fwd_kernel<TI, TA, 2>); break;
    default: go(se_a_fwd_kernel<TI, TA, 4>); break;
  }
  return launch_status();
}

template <typename TI, typename TA>
int launch_bwd(hipStream_t s, const Geo& g, const void* coeff, const int* atype, const int* nlist,
               const void* em, const void* dT, void* dR) {
  const dim3 grid((g.nloc + kWaves - 1) / kWaves), block(64 * kWaves);
  const int cpl = channels_per_lane(g.m1);
  const int nl = (g.m1 + cpl - 1) / cpl;
  const size_t shm =
      (size_t)kWaves * kSeg * sizeof(Rec) + (size_t)kWaves * kBatch * nl * 4 * sizeof(TA);
  (void)hipGetLastError();  // report only what this launch raises
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, block, shm, s, g, (const TI*)coeff, atype, nlist,
                       (const TI*)em, (const TI*)dT, (TA*)dR);
  };
  switch (cpl) {
    case 1: go(se_a_bwd_kernel<TI, TA, 1>); break;
    case 2: go(se_a_bwd_kernel<TI, TA, 2>); break;
    default: go(se_a_bwd_kernel<TI, TA, 4>); break;
  }
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
