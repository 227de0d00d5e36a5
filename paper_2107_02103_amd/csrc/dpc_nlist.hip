// Neighbour list of a periodic cubic box (DP Compress, Sec. II: the rows of
// the environment matrix are the neighbours within r_c, grouped by type into
// sel_beta rows each, sorted by distance inside a group, unused rows empty).
//
// Definition (the same as the plain oracle's): minimum image per component,
// d = x_j - x_i - box rint((x_j - x_i) / box); r2 = dx dx + dy dy + dz dz,
// every operation rounded on its own; j != i is a neighbour when
// r2 < rc * rc; neighbours are ordered by (type, r2, j) and the first
// sel[beta] of type beta fill block beta; empty slots hold -1.
//
// Cell list: cells of edge box / nc >= r_c (slightly more, so that rounding
// at a cell face cannot put two atoms closer than r_c two cells apart).
//   1. zero the counters;  2. cell of each atom, counted with atomics;
//   3. exclusive scan (one workgroup);  4. scatter the atoms into cell order
//   with their coordinates, index and type packed in 32 bytes;
//   5. one wavefront per atom walks the (up to) 27 cells around its own as
//   column spans of the cell-ordered array, 64 candidates at a time with
//   the next batch in flight, keeps those within r_c in LDS, ranks each of
//   them among the neighbours of its type and writes its slot.
// The order inside a cell depends on the atomics, but the ranking is a total
// order, so the list does not.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "dpc.h"
#include "dpc_internal.h"

namespace {

constexpr int kNlWaves = 4;      // wavefronts (atoms) per workgroup of the list kernel
constexpr int kNlCap = 1024;     // neighbours within rc one wavefront keeps (12 KB of LDS)
constexpr int kScanThreads = 1024;

struct alignas(16) NlAtom {      // an atom in cell order
  double x, y, z;
  int j, type;
};

// A neighbour within r_c as kept in LDS: the bits of r2 (>= 0: ordered like
// the value) in one array, type and index packed as type << 28 | j in another
// (12 bytes per neighbour, so that three workgroups share a CU).
constexpr int kJBits = 28;
constexpr uint32_t kJMask = (1u << kJBits) - 1;

struct NlGeo {
  int nloc, ntypes, nnei, nc, ncell;
  int lo_off, n_off;             // stencil offsets per axis: lo_off .. lo_off + n_off - 1
  double box, rc2, inv_cs, inv_box;
  int sel[DPC_MAX_TYPES];
  int blk[DPC_MAX_TYPES + 1];    // first slot of each type block
};

// d - box rint(d / box) with the quotient correctly rounded, as defined.
// rint(d / box) is taken from d (1 / box) instead of a division whenever that
// product lies more than 1e-6 away from a half-integer (and |q| < 2^20): the
// two quotients differ by a few units in the last place (< 1e-9 there), so
// both round to the same integer.  Otherwise (rare; NaN and infinities too)
// the division decides.
__device__ __forceinline__ double min_image(double d, const NlGeo& g) {
#pragma clang fp contract(off)
  const double q = d * g.inv_box;
  double n = rint(q);
  if (!(fabs(q - n) < 0.499999 && fabs(q) < 1048576.0)) n = rint(d / g.box);
  return d - g.box * n;
}

__device__ __forceinline__ int cell_axis(double x, const NlGeo& g) {
#pragma clang fp contract(off)
  const double w = x - g.box * floor(x / g.box);       // into [0, box]
  // clamped as a double first: NaN and infinite positions land in cell 0
  return (int)fmin(fmax(w * g.inv_cs, 0.0), (double)(g.nc - 1));
}

__global__ void nl_zero_kernel(int n, int* __restrict__ p) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

__global__ void nl_cell_kernel(const NlGeo g, const double* __restrict__ coord,
                               int* __restrict__ count, int* __restrict__ cell_of) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= g.nloc) return;
  const double* p = coord + 3 * (size_t)i;
  const int c = (cell_axis(p[0], g) * g.nc + cell_axis(p[1], g)) * g.nc + cell_axis(p[2], g);
  cell_of[i] = c;
  atomicAdd(count + c, 1);
}

// exclusive scan of count[0..ncell) into start[0..ncell] and cursor[0..ncell)
__global__ __launch_bounds__(kScanThreads) void nl_scan_kernel(int ncell,
                                                               const int* __restrict__ count,
                                                               int* __restrict__ start,
                                                               int* __restrict__ cursor) {
  __shared__ int part[kScanThreads];
  const int t = threadIdx.x;
  const int per = (ncell + kScanThreads - 1) / kScanThreads;
  const int c0 = min(ncell, t * per), c1 = min(ncell, c0 + per);
  int sum = 0;
  for (int c = c0; c < c1; ++c) sum += count[c];
  part[t] = sum;
  __syncthreads();
  for (int off = 1; off < kScanThreads; off <<= 1) {   // inclusive scan of the parts
    const int v = t >= off ? part[t - off] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int run = part[t] - sum;
  for (int c = c0; c < c1; ++c) {
    start[c] = run;
    cursor[c] = run;
    run += count[c];
  }
  if (t == kScanThreads - 1) start[ncell] = part[t];
}

__global__ void nl_scatter_kernel(const NlGeo g, const double* __restrict__ coord,
                                  const int* __restrict__ atype,
                                  const int* __restrict__ cell_of, int* __restrict__ cursor,
                                  NlAtom* __restrict__ sorted) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= g.nloc) return;
  const int p = atomicAdd(cursor + cell_of[i], 1);
  const double* c = coord + 3 * (size_t)i;
  NlAtom a;
  a.x = c[0];
  a.y = c[1];
  a.z = c[2];
  a.j = i;
  a.type = atype[i];
  sorted[p] = a;
}

__device__ __forceinline__ uint64_t ballot(bool b) { return __ballot(b); }

// rank + 1 if (type, r2, j) of the packed neighbour (or2, ojt) is below
// (t, r2, j) as unsigned words (the borrow
// of the four-word subtraction), else rank.  r2 >= 0, so its bits order like
// its value.  A subtraction chain keeps the whole comparison in the vector
// unit; compares combined with mask logic would go through scalar registers.
__device__ __forceinline__ unsigned count_before(uint64_t or2, uint32_t ojt, uint32_t j, uint32_t r2lo,
                                                 uint32_t r2hi, uint32_t t, unsigned rank) {
  uint32_t d;
  asm("v_sub_co_u32 %0, vcc, %2, %3\n\t"
      "v_subb_co_u32 %0, vcc, %4, %5, vcc\n\t"
      "v_subb_co_u32 %0, vcc, %6, %7, vcc\n\t"
      "v_subb_co_u32 %0, vcc, %8, %9, vcc\n\t"
      "v_addc_co_u32 %1, vcc, 0, %1, vcc"
      : "=&v"(d), "+v"(rank)
      : "v"(ojt & kJMask), "v"(j), "v"((uint32_t)or2), "v"(r2lo), "v"((uint32_t)(or2 >> 32)),
        "v"(r2hi), "v"(ojt >> kJBits), "v"(t)
      : "vcc");
  return rank;
}

__device__ __forceinline__ int lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

// one wavefront per atom
__global__ __launch_bounds__(64 * kNlWaves) void nl_list_kernel(
    const NlGeo g, const double* __restrict__ coord, const int* __restrict__ cell_of,
    const int* __restrict__ start, const NlAtom* __restrict__ sorted, int* __restrict__ nlist,
    int* __restrict__ status) {
#pragma clang fp contract(off)
  __shared__ uint64_t cand_r2[kNlWaves][kNlCap + 4];
  __shared__ uint32_t cand_jt[kNlWaves][kNlCap + 4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * kNlWaves + wave));
  if (i >= g.nloc) return;
  uint64_t* my_r2 = cand_r2[wave];
  uint32_t* my_jt = cand_jt[wave];
  const double xi = coord[3 * (size_t)i], yi = coord[3 * (size_t)i + 1], zi = coord[3 * (size_t)i + 2];
  const int ci = __builtin_amdgcn_readfirstlane(cell_of[i]);
  const int cx = ci / (g.nc * g.nc), cy = (ci / g.nc) % g.nc, cz = ci % g.nc;

  // candidates within rc, in the order they are met (n may pass kNlCap:
  // the extra ones are counted, not kept).  The stencil's cells are read as
  // spans of `sorted`: the cells of one (x, y) column that are consecutive
  // in z are consecutive there too, so a column is one span, or two where
  // it wraps around the box.  Lane k < 2 n_off^2 holds span k (column k / 2,
  // part k % 2, possibly empty); the loop walks the spans 64 atoms at a time
  // and loads the next batch before it works on the current one.
  const int nsp = 2 * g.n_off * g.n_off;
  int sp0 = 0, sp1 = 0;
  if (lane < nsp) {
    const int col = lane >> 1, part = lane & 1;
    const int ax = (cx + g.lo_off + col / g.n_off + g.nc) % g.nc;
    const int ay = (cy + g.lo_off + col % g.n_off + g.nc) % g.nc;
    const int base = (ax * g.nc + ay) * g.nc;
    int c0 = 0, c1 = 0;                 // cells [c0, c1) of this column
    if (g.nc < 3) {
      if (part == 0) c1 = g.nc;
    } else if (cz > 0 && cz < g.nc - 1) {
      if (part == 0) { c0 = cz - 1; c1 = cz + 2; }
    } else if (cz == 0) {
      if (part == 0) { c0 = g.nc - 1; c1 = g.nc; } else { c0 = 0; c1 = 2; }
    } else {
      if (part == 0) { c0 = g.nc - 2; c1 = g.nc; } else { c0 = 0; c1 = 1; }
    }
    sp0 = start[base + c0];
    sp1 = start[base + c1];
  }
  // the first batch at or after (span s, atom b) that holds atoms
  auto advance = [&](int& s, int& b, int& e) __attribute__((always_inline)) {
    while (b >= e && ++s < nsp) {
      b = __builtin_amdgcn_readlane(sp0, s);
      e = __builtin_amdgcn_readlane(sp1, s);
    }
  };
  int n = 0;
  int s = 0, b = __builtin_amdgcn_readlane(sp0, 0), e = __builtin_amdgcn_readlane(sp1, 0);
  advance(s, b, e);
  NlAtom cur = sorted[s < nsp ? min(b + lane, g.nloc - 1) : 0];
  while (s < nsp) {
    int s2 = s, b2 = b + 64, e2 = e;
    advance(s2, b2, e2);
    // every lane loads (an index inside the array), so that no load is conditional
    const NlAtom nxt = sorted[s2 < nsp ? min(b2 + lane, g.nloc - 1) : 0];
    bool ok = false;
    uint64_t kr2 = 0;
    uint32_t kjt = 0;
    if (b + lane < e) {
      const double dx = min_image(cur.x - xi, g);
      const double dy = min_image(cur.y - yi, g);
      const double dz = min_image(cur.z - zi, g);
      const double r2 = dx * dx + dy * dy + dz * dz;
      ok = r2 < g.rc2 && cur.j != i && cur.type >= 0 && cur.type < g.ntypes;
      kr2 = __builtin_bit_cast(uint64_t, r2);
      kjt = (uint32_t)cur.type << kJBits | (uint32_t)cur.j;
    }
    const uint64_t msk = ballot(ok);
    const int pos = n + lanes_below(msk);
    if (ok && pos < kNlCap) {
      my_r2[pos] = kr2;
      my_jt[pos] = kjt;
    }
    n += __popcll(msk);
    cur = nxt;
    s = s2;
    b = b2;
    e = e2;
  }
  const int m = n < kNlCap ? n : kNlCap;
  // four entries that rank after every neighbour (type field 15) after the
  // kept ones, so that the ranking below reads the list four at a time
  if (lane < 4) {
    my_r2[m + lane] = ~0ull;
    my_jt[m + lane] = ~0u;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  // neighbours of each type (all of them, before truncation)
  int cnt[DPC_MAX_TYPES];
#pragma unroll
  for (int t = 0; t < DPC_MAX_TYPES; ++t) cnt[t] = 0;
  for (int b = 0; b < m; b += 64) {
    const int q = b + lane;
    const int ty = q < m ? (int)(my_jt[q] >> kJBits) : -1;
#pragma unroll
    for (int t = 0; t < DPC_MAX_TYPES; ++t) cnt[t] += __popcll(ballot(ty == t));
  }

  // slot of each kept neighbour: its rank among the neighbours of its type
  // by (r2, j), i.e. its rank among all of them by (type, r2, j) less the
  // number of neighbours of smaller types; up to four candidates per lane
  // per pass over all m, four list entries per step
  int* row = nlist + (size_t)i * g.nnei;
  for (int b = 0; b < m; b += 256) {
    uint64_t own_r2[4];
    uint32_t own_jt[4];
    unsigned rank[4];
    const int nu = min(4, (m - b + 63) / 64);   // candidate sets of this pass
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int q = b + 64 * u + lane;
      own_r2[u] = q < m ? my_r2[q] : ~0ull;
      own_jt[u] = q < m ? my_jt[q] : ~0u;
      rank[u] = 0;
#pragma unroll
      for (int t = 0; t < DPC_MAX_TYPES; ++t)
        rank[u] -= (uint32_t)t < (own_jt[u] >> kJBits) ? (unsigned)cnt[t] : 0u;
    }
    for (int e = 0; e < m; e += 4) {
      uint64_t o_r2[4];
      uint32_t o_jt[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        o_r2[v] = my_r2[e + v];
        o_jt[v] = my_jt[e + v];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (u >= nu) break;
#pragma unroll
        for (int v = 0; v < 4; ++v)
          rank[u] = count_before(o_r2[v], o_jt[v], own_jt[u] & kJMask, (uint32_t)own_r2[u],
                                 (uint32_t)(own_r2[u] >> 32), own_jt[u] >> kJBits, rank[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int q = b + 64 * u + lane;
      const int t = (int)(own_jt[u] >> kJBits);
      if (q < m && (int)rank[u] < g.sel[t]) row[g.blk[t] + (int)rank[u]] = (int)(own_jt[u] & kJMask);
    }
  }
  // empty slots of each block
  for (int s = lane; s < g.nnei; s += 64) {
    int t = 0;
#pragma unroll
    for (int u = 1; u < DPC_MAX_TYPES; ++u) t += (u < g.ntypes && s >= g.blk[u]) ? 1 : 0;
    int c = 0;
#pragma unroll
    for (int u = 0; u < DPC_MAX_TYPES; ++u) c = u == t ? cnt[u] : c;
    if (s - g.blk[t] >= c) row[s] = -1;
  }
  if (lane == 0) {
    bool trunc = false;
#pragma unroll
    for (int t = 0; t < DPC_MAX_TYPES; ++t) trunc |= t < g.ntypes && cnt[t] > g.sel[t];
    if (trunc) atomicAdd(status, 1);
    if (n > kNlCap) atomicAdd(status + 1, 1);
  }
}

constexpr size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// cells per axis: edge >= rc (1 + 1e-9); at most 1024 per axis and one cell per atom
int cells_per_axis(int nloc, double box, double rc) {
  double n = std::floor(box / (rc * (1.0 + 1e-9)));
  if (!(n >= 1.0)) n = 1.0;
  if (n > 1024.0) n = 1024.0;
  const double cap = std::max(64.0, (double)nloc);
  while (n > 1.0 && n * n * n > cap) n -= 1.0;
  return (int)n;
}

struct NlLayout {
  size_t status, count, start, cursor, cell_of, sorted, total;
};

constexpr NlLayout layout(int nloc, int ncell) {
  NlLayout L{};
  size_t o = 0;
  L.status = o; o += align256(2 * sizeof(int));
  L.count = o; o += align256((size_t)ncell * sizeof(int));
  L.start = o; o += align256(((size_t)ncell + 1) * sizeof(int));
  L.cursor = o; o += align256((size_t)ncell * sizeof(int));
  L.cell_of = o; o += align256((size_t)nloc * sizeof(int));
  L.sorted = o; o += align256((size_t)nloc * sizeof(NlAtom));
  L.total = o;
  return L;
}

int make_geo(int nloc, int ntypes, const int* sel, double box, double rc, NlGeo* g) {
#pragma clang fp contract(off)
  if (nloc < 0 || ntypes < 1 || !sel) return DPC_EINVAL;
  // neighbour indices are kept in kJBits bits
  if (ntypes > DPC_MAX_TYPES || nloc > (1 << kJBits)) return DPC_ENOTSUP;
  if (!(std::isfinite(box) && std::isfinite(rc) && rc > 0.0 && box > 2.0 * rc)) return DPC_ERANGE;
  int64_t nnei = 0;
  for (int t = 0; t < ntypes; ++t) {
    if (sel[t] < 0) return DPC_EINVAL;
    g->blk[t] = (int)nnei;
    g->sel[t] = sel[t];
    nnei += sel[t];
  }
  if (nnei < 1 || nnei > (1 << 20)) return DPC_EINVAL;
  for (int t = ntypes; t < DPC_MAX_TYPES; ++t) g->sel[t] = 0;
  for (int t = ntypes; t <= DPC_MAX_TYPES; ++t) g->blk[t] = (int)nnei;
  g->nloc = nloc;
  g->ntypes = ntypes;
  g->nnei = (int)nnei;
  g->nc = cells_per_axis(nloc, box, rc);
  g->ncell = g->nc * g->nc * g->nc;
  g->lo_off = g->nc >= 3 ? -1 : 0;
  g->n_off = g->nc >= 3 ? 3 : g->nc;
  g->box = box;
  g->rc2 = rc * rc;
  g->inv_cs = g->nc / box;
  g->inv_box = 1.0 / box;
  return DPC_OK;
}

}  // namespace

static size_t dpc_nlist_scratch_bytes(int nloc, double box, double rc) {
  if (nloc < 0 || !(std::isfinite(box) && std::isfinite(rc) && rc > 0.0 && box > 2.0 * rc)) return 0;
  const int nc = cells_per_axis(nloc, box, rc);
  return layout(nloc, nc * nc * nc).total;
}

// status_dev: device int[2] for the two counters (NULL: the first 8 bytes of
// the workspace); status_host: host int[2] to wait for and copy them to, or NULL
static int dpc_nlist_launch(void* stream, int nloc, int ntypes, const int* sel, double box, double rc,
                            const double* coord, const int* atype, void* workspace,
                            size_t workspace_bytes, int* nlist, int* status_dev,
                            int* status_host) {
  NlGeo g;
  const int st = make_geo(nloc, ntypes, sel, box, rc, &g);
  if (st != DPC_OK) return st;
  if (nloc == 0) {
    if (status_host) status_host[0] = status_host[1] = 0;
    return DPC_OK;
  }
  if (!coord || !atype || !workspace || !nlist) return DPC_EINVAL;
  const NlLayout L = layout(nloc, g.ncell);
  if (workspace_bytes < L.total || reinterpret_cast<uintptr_t>(workspace) % 256) return DPC_EINVAL;
  unsigned char* w = static_cast<unsigned char*>(workspace);
  int* status = status_dev ? status_dev : reinterpret_cast<int*>(w + L.status);
  int* count = reinterpret_cast<int*>(w + L.count);
  int* start = reinterpret_cast<int*>(w + L.start);
  int* cursor = reinterpret_cast<int*>(w + L.cursor);
  int* cell_of = reinterpret_cast<int*>(w + L.cell_of);
  NlAtom* sorted = reinterpret_cast<NlAtom*>(w + L.sorted);
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();  // report only what these launches raise
  // the counters and the status words start at zero (a fill kernel, not a memset)
  hipLaunchKernelGGL(nl_zero_kernel, dim3(1), dim3(64), 0, s, 2, status);
  hipLaunchKernelGGL(nl_zero_kernel, dim3((g.ncell + 255) / 256), dim3(256), 0, s, g.ncell, count);
  const dim3 ga((nloc + 255) / 256), b256(256);
  hipLaunchKernelGGL(nl_cell_kernel, ga, b256, 0, s, g, coord, count, cell_of);
  hipLaunchKernelGGL(nl_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, g.ncell, count, start, cursor);
  hipLaunchKernelGGL(nl_scatter_kernel, ga, b256, 0, s, g, coord, atype, cell_of, cursor, sorted);
  hipLaunchKernelGGL(nl_list_kernel, dim3((nloc + kNlWaves - 1) / kNlWaves), dim3(64 * kNlWaves), 0, s,
                     g, coord, cell_of, start, sorted, nlist, status);
  const int ls = dpc_internal_launch_status();
  if (ls != DPC_OK || !status_host) return ls;
  int h[2] = {0, 0};
  if (hipMemcpyAsync(h, status, sizeof h, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess) {
    const int e = dpc_internal_launch_status();   // keeps the HIP error for dpc_last_hip_error
    return e == DPC_OK ? DPC_EHIP : e;
  }
  status_host[0] = h[0];
  status_host[1] = h[1];
  if (h[1] > 0) return DPC_ENOTSUP;
  if (h[0] > 0) return DPC_EOVERFLOW;
  return DPC_OK;
}

// ---------------------------------------------------------------------------
// The same list with the cell list in a static device array of the library,
// for callers that cannot allocate device memory.  Each GPU that runs it
// holds one copy of the array until the process ends; host code reaches it
// only through the device address hipGetSymbolAddress gives for that GPU.
// ---------------------------------------------------------------------------
// the cell count is capped at max(64, nloc): the largest layout is that of
// DPC_NLIST_NOALLOC_MAX_ATOMS atoms and as many cells
static constexpr size_t kScratchBytes =
    layout(DPC_NLIST_NOALLOC_MAX_ATOMS, DPC_NLIST_NOALLOC_MAX_ATOMS).total;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// device address of this GPU's copy of `scratch`, looked up once per device
// with that device current
int scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return DPC_ENOTSUP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      const int e = dpc_internal_launch_status();
      return e == DPC_OK ? DPC_EHIP : e;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DPC_OK;
}

}  // namespace

extern "C" int dpc_nlist_build_noalloc(void* stream, int nloc, int ntypes, const int* sel,
                                       double box, double rc, const double* coord,
                                       const int* atype, int* nlist, int* status) {
  NlGeo g;
  const int st = make_geo(nloc, ntypes, sel, box, rc, &g);
  if (st != DPC_OK) return st;
  if (nloc > DPC_NLIST_NOALLOC_MAX_ATOMS || layout(nloc, g.ncell).total > kScratchBytes)
    return DPC_ENOTSUP;
  if (nloc == 0) return DPC_OK;
  if (!coord || !atype || !nlist) return DPC_EINVAL;
  // the array of the GPU the stream runs on, which must be the current one
  int cur = -1;
  hipDevice_t sdev = -1;
  if (hipGetDevice(&cur) != hipSuccess ||
      hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev) != hipSuccess) {
    const int e = dpc_internal_launch_status();
    return e == DPC_OK ? DPC_EHIP : e;
  }
  if (sdev != cur) return DPC_EINVAL;
  void* ws = nullptr;
  const int sa = scratch_address(cur, &ws);
  if (sa != DPC_OK) return sa;
  return dpc_nlist_launch(stream, nloc, ntypes, sel, box, rc, coord, atype, ws, kScratchBytes,
                          nlist, status, nullptr);
}

extern "C" size_t dpc_nlist_workspace_bytes(int nloc, double box, double rc) {
  return dpc_nlist_scratch_bytes(nloc, box, rc);
}

extern "C" int dpc_nlist_build(void* stream, int nloc, int ntypes, const int* sel, double box,
                               double rc, const double* coord, const int* atype, void* workspace,
                               size_t workspace_bytes, int* nlist, int* status_host) {
  return dpc_nlist_launch(stream, nloc, ntypes, sel, box, rc, coord, atype, workspace,
                          workspace_bytes, nlist, nullptr, status_host);
}
