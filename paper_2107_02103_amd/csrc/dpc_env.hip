// Environment matrix R~ from positions, and forces / virials from dE/dR~
// (DP Compress, Sec. II: the weighting function of Eq. (1), the per-type
// normalisation after it, and F = -dE/dr).
//
// For neighbour slot s of atom i with j = nlist[i][s] >= 0, r_ij = r_j - r_i
// is the minimum image in a cubic periodic box of edge L (L > 2 r_c), r =
// |r_ij|, and the row of R~ is
//   ((s(r) - mean_t) / sigma_t, s(r) x / sigma_all_t, s(r) y / ..., s(r) z / ...)
// with t the type of atom i; padding rows are zero.
//
// Forces: g_is = dE/dr_ij = sum_c dE/dR~_is[c] dR~_is[c]/dr_ij, which is
//   g = (s'(r) / r) (lam_0 / sigma_t + <lam_xyz, r_ij> / sigma_all_t) r_ij
//       + (s(r) / sigma_all_t) lam_xyz          (lam = dE/dR~_is).
// F_i = sum_s g_is - sum over the rows (j, s') in which i is the neighbour of
// g_js'.  Those rows are found once per neighbour list (dpc_nlist_reverse),
// so that each atom gathers its force in a fixed order: no atomics, and the
// result is bitwise reproducible.  The derivative dR~/dr (12 numbers per
// slot) is recomputed from the positions, not stored.  The per-atom virial
// is V_i = -sum_s r_is (x) g_is.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "dpc.h"
#include "dpc_internal.h"

namespace {

struct EnvGeo {
  int nloc, nnei, ntypes;
  double box, rc, rcs;
  double inv_box, inv_w;            // 1 / box, 1 / (rc - rcs)
  double mean[DPC_MAX_TYPES], inv_sigma[DPC_MAX_TYPES], inv_sigma_all[DPC_MAX_TYPES];
  int blk[DPC_MAX_TYPES + 1];       // sel block boundaries (slot offsets)
};

// minimum image of b - a in the cubic box
__device__ __forceinline__ void min_image(const EnvGeo& g, const double* a, const double* b,
                                          double (&d)[3]) {
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    const double x = b[c] - a[c];
    d[c] = x - g.box * round(x * g.inv_box);
  }
}

// s(r) and ds/dr of Eq. (1)
__device__ __forceinline__ void weight(const EnvGeo& g, double r, double& s, double& ds) {
  const double ir = 1.0 / r;
  if (r < g.rcs) {
    s = ir;
    ds = -ir * ir;
  } else if (r < g.rc) {
    const double u = (r - g.rcs) * g.inv_w;
    const double u2 = u * u, u3 = u2 * u;
    const double sw = u3 * (-6.0 * u2 + 15.0 * u - 10.0) + 1.0;
    const double dsw = (-30.0 * u2 * (u - 1.0) * (u - 1.0)) * g.inv_w;
    s = sw * ir;
    ds = (dsw - sw * ir) * ir;
  } else {
    s = 0.0;
    ds = 0.0;
  }
}

// workgroup b covers slots 256 c .. 256 c + 255 of atom b / chunks (c = b mod
// chunks), so that the atom index is uniform; rows are written 16 bytes at a
// time when the output is 16-byte aligned (kPair), float64 rows of whole
// wavefronts in contiguous 1 KB stores
template <typename TO, bool kPair>
__global__ __launch_bounds__(256) void env_mat_kernel(const EnvGeo g, int chunks,
                                                      const double* __restrict__ coord,
                                                      const int* __restrict__ atype,
                                                      const int* __restrict__ nlist,
                                                      TO* __restrict__ em) {
  const int i = __builtin_amdgcn_readfirstlane((int)(blockIdx.x / (unsigned)chunks));
  const int s = (int)(blockIdx.x - (unsigned)i * chunks) * 256 + threadIdx.x;
  if (s >= g.nnei) return;
  const size_t e = (size_t)i * g.nnei + s;
  const int j = __builtin_nontemporal_load(nlist + e);
  double row[4] = {0.0, 0.0, 0.0, 0.0};
  const int t = atype[i];
  if (j >= 0 && j < g.nloc && t >= 0 && t < g.ntypes) {
    double d[3];
    min_image(g, coord + 3 * (size_t)i, coord + 3 * (size_t)j, d);
    const double r = sqrt(d[0] * d[0] + d[1] * d[1] + d[2] * d[2]);
    double sv, ds;
    weight(g, r, sv, ds);
    row[0] = (sv - g.mean[t]) * g.inv_sigma[t];
    const double f = sv * g.inv_sigma_all[t];
    row[1] = f * d[0];
    row[2] = f * d[1];
    row[3] = f * d[2];
  } else if (j >= 0) {   // neighbour or centre out of range: the row is NaN
    row[0] = row[1] = row[2] = row[3] = (double)NAN;
  }
  TO* o = em + 4 * e;
  if constexpr (kPair && sizeof(TO) == 8) {
    typedef double D2 __attribute__((ext_vector_type(2)));
    // a wavefront whose 64 slots are all in the list writes its 2 KB of rows
    // as two fully contiguous 1 KB stores, transposed through LDS (each lane
    // storing its own 32-byte row leaves every store instruction with gaps)
    __shared__ __align__(16) D2 stage[4][128];
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int sw = __builtin_amdgcn_readfirstlane(s - l);
    if (sw + 64 <= g.nnei) {
      stage[w][2 * l] = D2{row[0], row[1]};
      stage[w][2 * l + 1] = D2{row[2], row[3]};
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      D2* ow = reinterpret_cast<D2*>(em + 4 * ((size_t)i * g.nnei + sw));
      __builtin_nontemporal_store(stage[w][l], ow + l);
      __builtin_nontemporal_store(stage[w][l + 64], ow + l + 64);
      return;
    }
    __builtin_nontemporal_store(D2{row[0], row[1]}, reinterpret_cast<D2*>(o));
    __builtin_nontemporal_store(D2{row[2], row[3]}, reinterpret_cast<D2*>(o) + 1);
  } else if constexpr (kPair) {
    typedef float F4 __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(F4{(float)row[0], (float)row[1], (float)row[2], (float)row[3]},
                                reinterpret_cast<F4*>(o));
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) __builtin_nontemporal_store((TO)row[c], o + c);
  }
}

// rev[i][s] = slot of i in the list of j = nlist[i][s], in the sel block of
// i's type, or -1.  rev starts as -1 everywhere (fill_kernel).  A pair found
// in both lists gives both entries, rev[i][s] = k and rev[j][k] = s, so each
// pair is searched once, by the wavefront of its smaller atom i < j (the
// other one skips it; a pair that only one list holds is searched by that
// list's atom when it is the smaller one, and else stays -1, which is then
// right).  The wavefront takes its pairs eight at a time, and for each the
// whole wavefront reads the two 128-byte lines of j's block around where i
// is expected (i's rank in j's list is close to j's rank in i's list: the
// same distance orders both) and looks for i with one ballot; the eight
// window reads are issued together.  A miss (lists in another order, ranks
// further apart) scans j's whole block.
constexpr int kRevGroup = 8;
__global__ void fill_kernel(int64_t n, int v, int* __restrict__ p) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < n) p[e] = v;
}

__global__ __launch_bounds__(256) void reverse_kernel(const EnvGeo g, const int* __restrict__ atype,
                                                      const int* __restrict__ nlist,
                                                      int* __restrict__ rev) {
  const int lane = threadIdx.x & 63;
  const int i = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6));
  if (i >= g.nloc) return;
  const int t = __builtin_amdgcn_readfirstlane(atype[i]);
  if (t < 0 || t >= g.ntypes) return;       // its slots stay -1
  const int b0 = g.blk[t], b1 = g.blk[t + 1];
  const int wlo = b0, whi = b1 - 32 > b0 ? b1 - 32 : b0;     // window centres start here
  const int* li = nlist + (size_t)i * g.nnei;
  int* ri = rev + (size_t)i * g.nnei;
  int jn = lane < g.nnei ? li[lane] : -1;      // the next batch's slots, loaded ahead
  for (int s0 = 0; s0 < g.nnei; s0 += 64) {
    const int s = s0 + lane;
    const int j = jn;
    jn = s + 64 < g.nnei ? li[s + 64] : -1;
    const bool mine = j > i && j < g.nloc;
    int found = -1, tmine = -1;       // this lane's pair: slot of i in j's list, j's type
    uint64_t todo = __ballot(mine);
    while (todo) {
      int src[kRevGroup], jj[kRevGroup], tj[kRevGroup], w0[kRevGroup], v[kRevGroup];
#pragma unroll
      for (int q = 0; q < kRevGroup; ++q) {
        src[q] = todo ? (int)__builtin_ctzll(todo) : -1;
        todo &= todo ? todo - 1 : 0;
        jj[q] = src[q] >= 0 ? __builtin_amdgcn_readlane(j, src[q]) : 0;
        tj[q] = atype[jj[q]];          // uniform: a scalar load beside the window's
        // j's place in i's list, relative to the start of its block there
        const int sj = s0 + (src[q] >= 0 ? src[q] : 0);
        int bs = 0;
#pragma unroll
        for (int u = 1; u < DPC_MAX_TYPES; ++u) bs = (u < g.ntypes && sj >= g.blk[u]) ? g.blk[u] : bs;
        // 32 slots centred where i is expected, clamped into the block, read
        // as the two 32-entry groups of the row that hold them
        const int c = b0 + (sj - bs) - 16;
        const int ca = c < wlo ? wlo : (c > whi ? whi : c);
        w0[q] = ca & ~31;
        // every lane reads an entry inside j's row; those outside the block are masked
        const int k = w0[q] + lane;
        v[q] = nlist[(size_t)jj[q] * g.nnei + (k < g.nnei ? k : g.nnei - 1)];
        v[q] = k >= b0 && k < b1 ? v[q] : -1;
      }
#pragma unroll
      for (int q = 0; q < kRevGroup; ++q) {
        if (src[q] < 0) break;
        const uint64_t hit = __ballot(v[q] == i);
        int kk = hit ? w0[q] + (int)__builtin_ctzll(hit) : -1;
        for (int c0 = b0; kk < 0 && c0 < b1; c0 += 64) {   // not in the window: the whole block
          const int k = c0 + lane;
          const int e = k < b1 ? nlist[(size_t)jj[q] * g.nnei + k] : -1;
          const uint64_t h = __ballot(e == i);
          kk = h ? c0 + (int)__builtin_ctzll(h) : -1;
        }
        if (lane == src[q]) {
          found = kk;
          tmine = tj[q];
        }
      }
    }
    // one store instruction each per batch: the found slots, and their
    // reverses, j's slot in i's list, where it lies in the block of j's
    // type (where that search would look)
    if (found >= 0) {
      ri[s] = found;
      if (tmine >= 0 && tmine < g.ntypes && s >= g.blk[tmine] && s < g.blk[tmine + 1])
        rev[(size_t)j * g.nnei + found] = s;
    }
  }
}

// one wavefront per atom; lane l takes slots l, l + 64, ...
template <typename TI>
__global__ __launch_bounds__(256) void force_kernel(const EnvGeo g, const double* __restrict__ coord,
                                                    const int* __restrict__ atype,
                                                    const int* __restrict__ nlist,
                                                    const int* __restrict__ rev,
                                                    const TI* __restrict__ dem,
                                                    double* __restrict__ force,
                                                    double* __restrict__ virial) {
  const int lane = threadIdx.x & 63;
  const int i = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6));
  if (i >= g.nloc) return;
  const int ti = atype[i];
  const bool ok_i = ti >= 0 && ti < g.ntypes;
  double acc[12];                          // F (3), then V row-major (9)
#pragma unroll
  for (int c = 0; c < 12; ++c) acc[c] = 0.0;
  const double* ci = coord + 3 * (size_t)i;
  // g for a pair vector d of a row with dE/dR~ lam, centre type t
  auto pair_grad = [&](const double (&d)[3], const TI* lam_p, int t, double (&gv)[3]) {
    const double r = sqrt(d[0] * d[0] + d[1] * d[1] + d[2] * d[2]);
    double s, ds;
    weight(g, r, s, ds);
    const double l0 = (double)lam_p[0], l1 = (double)lam_p[1], l2 = (double)lam_p[2],
                 l3 = (double)lam_p[3];
    const double c1 = (ds / r) * (l0 * g.inv_sigma[t] + (l1 * d[0] + l2 * d[1] + l3 * d[2]) * g.inv_sigma_all[t]);
    const double c2 = s * g.inv_sigma_all[t];
    gv[0] = c1 * d[0] + c2 * l1;
    gv[1] = c1 * d[1] + c2 * l2;
    gv[2] = c1 * d[2] + c2 * l3;
  };
  for (int s0 = 0; s0 < g.nnei; s0 += 64) {
    const int s = s0 + lane;
    if (s >= g.nnei || !ok_i) continue;
    const size_t e = (size_t)i * g.nnei + s;
    const int j = nlist[e];
    if (j < 0 || j >= g.nloc) continue;
    double d[3];
    min_image(g, ci, coord + 3 * (size_t)j, d);
    double go[3];
    pair_grad(d, dem + 4 * e, ti, go);
    acc[0] += go[0];
    acc[1] += go[1];
    acc[2] += go[2];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
#pragma unroll
      for (int b = 0; b < 3; ++b) acc[3 + 3 * a + b] -= d[a] * go[b];
    }
    const int rs = rev[e];
    const int tj = atype[j];
    if (rs >= 0 && rs < g.nnei && tj >= 0 && tj < g.ntypes) {
      // the row of j in which i is the neighbour: pair vector r_ji
      const double dr[3] = {-d[0], -d[1], -d[2]};
      double gr[3];
      pair_grad(dr, dem + 4 * ((size_t)j * g.nnei + rs), tj, gr);
      acc[0] -= gr[0];
      acc[1] -= gr[1];
      acc[2] -= gr[2];
    }
  }
  // sum over the wavefront in a fixed order
#pragma unroll
  for (int c = 0; c < 12; ++c) {
    double v = acc[c];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const int lo = __builtin_amdgcn_ds_bpermute(((lane ^ off) & 63) << 2,
                                                  (int)(uint32_t)__builtin_bit_cast(uint64_t, v));
      const int hi = __builtin_amdgcn_ds_bpermute(((lane ^ off) & 63) << 2,
                                                  (int)(uint32_t)(__builtin_bit_cast(uint64_t, v) >> 32));
      const double w = __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
      v = lane < (lane ^ off) ? v + w : w + v;
    }
    acc[c] = v;
  }
  if (lane == 0) {
    const double nan = ok_i ? 0.0 : (double)NAN;
    for (int c = 0; c < 3; ++c) force[3 * (size_t)i + c] = acc[c] + nan;
    if (virial)
      for (int c = 0; c < 9; ++c) virial[9 * (size_t)i + c] = acc[3 + c] + nan;
  }
}

int make_env_geo(int nloc, int ntypes, int nnei, double box, double rc, double rcs,
                 const double* mean, const double* sigma, const double* sigma_all, EnvGeo* g) {
  if (nloc < 0 || nnei < 1 || ntypes < 1) return DPC_EINVAL;
  if (ntypes > DPC_MAX_TYPES) return DPC_ENOTSUP;
  if (!(std::isfinite(box) && std::isfinite(rc) && std::isfinite(rcs) && rc > 0 && rcs >= 0 &&
        rcs < rc && box > 2 * rc))
    return DPC_ERANGE;
  if ((int64_t)nloc * nnei >= (int64_t(1) << 40)) return DPC_ENOTSUP;
  g->nloc = nloc;
  g->nnei = nnei;
  g->ntypes = ntypes;
  g->box = box;
  g->rc = rc;
  g->rcs = rcs;
  g->inv_box = 1.0 / box;
  g->inv_w = 1.0 / (rc - rcs);
  for (int t = 0; t < DPC_MAX_TYPES; ++t) {
    g->mean[t] = 0.0;
    g->inv_sigma[t] = g->inv_sigma_all[t] = 0.0;
    g->blk[t] = 0;
  }
  g->blk[DPC_MAX_TYPES] = 0;
  for (int t = 0; t < ntypes; ++t) {
    if (mean) {
      if (!std::isfinite(mean[t])) return DPC_ERANGE;
      g->mean[t] = mean[t];
    }
    if (sigma) {
      if (!(sigma[t] > 0 && std::isfinite(sigma[t]))) return DPC_ERANGE;
      g->inv_sigma[t] = 1.0 / sigma[t];
    }
    if (sigma_all) {
      if (!(sigma_all[t] > 0 && std::isfinite(sigma_all[t]))) return DPC_ERANGE;
      g->inv_sigma_all[t] = 1.0 / sigma_all[t];
    }
  }
  return DPC_OK;
}

}  // namespace

extern "C" int dpc_env_mat_a(void* stream, dpc_dtype dtype, int nloc, int ntypes, int nnei,
                             double box, double rc, double rcs, const double* mean,
                             const double* sigma, const double* sigma_all, const double* coord,
                             const int* atype, const int* nlist, void* em) {
  if (dtype != DPC_F64 && dtype != DPC_F32 && dtype != DPC_F32_ACC64) return DPC_EINVAL;
  if (!mean || !sigma || !sigma_all) return DPC_EINVAL;
  EnvGeo g;
  const int st = make_env_geo(nloc, ntypes, nnei, box, rc, rcs, mean, sigma, sigma_all, &g);
  if (st != DPC_OK) return st;
  if (nloc == 0) return DPC_OK;
  if (!coord || !atype || !nlist || !em) return DPC_EINVAL;
  const int chunks = (nnei + 255) / 256;
  if ((int64_t)nloc * chunks >= (int64_t(1) << 31)) return DPC_ENOTSUP;
  const dim3 grid((unsigned)(nloc * chunks));
  const bool pair = reinterpret_cast<uintptr_t>(em) % 16 == 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();  // report only what this launch raises
  auto go = [&](auto kern, auto* out) {
    hipLaunchKernelGGL(kern, grid, dim3(256), 0, s, g, chunks, coord, atype, nlist, out);
  };
  if (dtype == DPC_F64) {
    if (pair) go(env_mat_kernel<double, true>, (double*)em);
    else go(env_mat_kernel<double, false>, (double*)em);
  } else {
    if (pair) go(env_mat_kernel<float, true>, (float*)em);
    else go(env_mat_kernel<float, false>, (float*)em);
  }
  return dpc_internal_launch_status();
}

extern "C" int dpc_nlist_reverse(void* stream, int nloc, int ntypes, const int* sel, double box,
                                 const double* coord, const int* atype, const int* nlist,
                                 int* rev) {
  if (!sel) return DPC_EINVAL;
  if (ntypes < 1) return DPC_EINVAL;
  if (ntypes > DPC_MAX_TYPES) return DPC_ENOTSUP;
  int64_t nnei = 0;
  for (int t = 0; t < ntypes; ++t) {
    if (sel[t] < 0) return DPC_EINVAL;
    nnei += sel[t];
  }
  if (nnei < 1 || nnei > (1 << 20)) return DPC_EINVAL;
  EnvGeo g;
  // rc only bounds the box check here: any cutoff below half the box
  const int st = make_env_geo(nloc, ntypes, (int)nnei, box, 0.5 * box * 0.999, 0.0, nullptr,
                              nullptr, nullptr, &g);
  if (st != DPC_OK) return st;
  int off = 0;
  for (int t = 0; t < ntypes; ++t) {
    g.blk[t] = off;
    off += sel[t];
  }
  for (int t = ntypes; t <= DPC_MAX_TYPES; ++t) g.blk[t] = off;
  if (nloc == 0) return DPC_OK;
  if (!coord || !atype || !nlist || !rev) return DPC_EINVAL;
  const int64_t nslot = (int64_t)nloc * nnei;
  if ((nslot + 255) / 256 >= (int64_t(1) << 31)) return DPC_ENOTSUP;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((nslot + 255) / 256)), dim3(256), 0, s, nslot, -1, rev);
  hipLaunchKernelGGL(reverse_kernel, dim3((nloc + 3) / 4), dim3(256), 0, s, g, atype, nlist, rev);
  return dpc_internal_launch_status();
}

extern "C" int dpc_force_a(void* stream, dpc_dtype dtype, int nloc, int ntypes, int nnei,
                           double box, double rc, double rcs, const double* sigma,
                           const double* sigma_all, const double* coord, const int* atype,
                           const int* nlist, const int* rev, const void* dE_dem, double* force,
                           double* virial) {
  if (dtype != DPC_F64 && dtype != DPC_F32 && dtype != DPC_F32_ACC64) return DPC_EINVAL;
  if (!sigma || !sigma_all) return DPC_EINVAL;
  EnvGeo g;
  const int st = make_env_geo(nloc, ntypes, nnei, box, rc, rcs, nullptr, sigma, sigma_all, &g);
  if (st != DPC_OK) return st;
  if (nloc == 0) return DPC_OK;
  if (!coord || !atype || !nlist || !rev || !dE_dem || !force) return DPC_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid((nloc + 3) / 4), block(256);
  (void)hipGetLastError();
  if (dtype == DPC_F32)
    hipLaunchKernelGGL(force_kernel<float>, grid, block, 0, s, g, coord, atype, nlist, rev,
                       (const float*)dE_dem, force, virial);
  else
    hipLaunchKernelGGL(force_kernel<double>, grid, block, 0, s, g, coord, atype, nlist, rev,
                       (const double*)dE_dem, force, virial);
  return dpc_internal_launch_status();
}
