// Compressed se_a descriptor kernels for CDNA4 (gfx950).
//
// DP Compress (arXiv:2107.02103), Sec. II: the embedding net is replaced by a
// table of quintic Hermite pieces and fused with S = G^T R~ (here T), which is
// evaluated only over valid neighbours; D = T (T<)^T.  The backward kernel
// maps dE/dT to dE/dR~ through the polynomial and its derivative.
//
// Mapping (both kernels): lanes = channels.  Lane l owns the CPL consecutive
// channels CPL*l .. CPL*l + CPL - 1, so one 16-byte buffer load brings the
// coefficient of t^q for all of them (table rows are padded to a multiple of
// 4 channels).  A coefficient load costs the vector memory path the same time
// however many lanes use it, so a wavefront serves NB atoms at once and lets
// all their neighbours that fall into one interval share the load.
//
// Chunk sets: the neighbour lists of the NB atoms are walked in lockstep,
// 64 / NB slots per atom at a time, so that one pass of 64 lanes covers a
// chunk set.  Valid slots become records {R~ row, t} plus a key that orders
// intervals by (neighbour block, decreasing coefficient offset); lists sorted
// by distance are sorted by key.  The NB sorted lists are merged into one LDS
// array (rank = own position + binary-search counts in the other lists), in
// which equal keys form runs and, inside a run, records are grouped by atom;
// lists that are not sorted are concatenated instead, which is correct but
// shares less.  Each lane r holds the key, start and per-atom split points of
// run r; the wave fetches them with v_readlane.
//
// The wave walks the runs.  At the start of a run it issues the loads of the
// next run's coefficients into the second register set (always, so that the
// wait for the current set is a fixed count), then runs one loop per atom
// over that atom's records of the run, so accumulators and dE/dT are indexed
// statically.  Records are read from LDS two at a time.
//
// Forward: acc[a][k] += g_m(t) * R~[k] per channel, then T and D = T (T<)^T.
// Backward: for every record each lane forms its share of
//   dE/dR~[k] = sum_m dT[m][k] g_m + (k == 0) sum_m g'_m sum_k' dT[m][k'] R~[k']
// over its channels; the shares of a batch of 4 records are summed across
// lanes through LDS.  Beyond the table g is constant; the record then carries
// a zero row for the w term, which removes the derivative term.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <type_traits>

#include "dpc.h"
#include "dpc_internal.h"

#ifndef DPC_FWD_ATOMS_PER_WAVE
#define DPC_FWD_ATOMS_PER_WAVE 4
#endif
#ifndef DPC_BWD_ATOMS_PER_WAVE
#define DPC_BWD_ATOMS_PER_WAVE 2
#endif

namespace {

constexpr int kWaves = 4;      // wavefronts per workgroup
constexpr int kLanes = 64;
constexpr int kBatch = 4;      // records per cross-lane reduction in the backward pass
constexpr int kOffBits = 28;   // keys: (block << 28) | (2^28 - 1 - coefficient offset)
constexpr int kOffMask = (1 << kOffBits) - 1;
constexpr size_t kMaxLds = 65536;    // LDS a workgroup may take without opting in

struct PairRange {             // one ordered type pair's table, as the kernels see it
  double lo, d1, d2;
  double x_up, x_end;          // ends of the main range and of the band (formed on the host)
  int L1, L2;
  int offset;                  // element offset of the pair's coefficients
  int pad;
};

struct Geo {
  int nloc, nnei, ntypes, m1, m2, ld;
  int coeff_bytes;             // size of the coefficient buffer (bounds the buffer loads)
  int pair_out;                // forward: T and D may be written 16 bytes at a time
  int blk_end[DPC_MAX_TYPES];  // slot index one past the end of each sel block
  PairRange pr[DPC_MAX_TYPES * DPC_MAX_TYPES];
};

template <typename TI>
struct alignas(16) Rec {       // one valid neighbour, as staged in LDS
  double t;                    // offset from the left node of its interval (read first:
  double pad;                  //   the polynomial needs it before the row)
  TI r[4];                     // its row of R~ (zero in the backward pass when clamped)
};

// A chunk set's keys and run tables in LDS (dead while its runs are walked).
struct ChunkScratch {
  int mk[kLanes];              // keys in merged order
  int mi[kLanes];              // slot | atom << 20 in merged order
  int rk[kLanes + 2];          // run keys (before that: keys of the compacted per-atom lists)
  int rs[kLanes + 2];          // run starts, then the record count
};

// LDS of one wavefront for one chunk set.
template <typename TI>
struct WaveLds {
  Rec<TI> z[kLanes];           // merged records
  ChunkScratch s;
};

__host__ __device__ constexpr size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

// Record e of a wave's merged list, the list starting `zoff` bytes into the
// workgroup's LDS.  The offset is formed in 32 bits (indexing through a
// generic pointer costs a 64-bit multiply-add per read).
template <typename TI>
__device__ __forceinline__ const Rec<TI>& zrec(const unsigned char* lds, uint32_t zoff, int e) {
  return *reinterpret_cast<const Rec<TI>*>(
      __builtin_assume_aligned(lds + zoff + (uint32_t)e * (uint32_t)sizeof(Rec<TI>), 16));
}

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int block_of(const Geo& g, int j) {
  int b = 0;
#pragma unroll
  for (int k = 0; k < DPC_MAX_TYPES - 1; ++k) b += (k < g.ntypes - 1 && j >= g.blk_end[k]) ? 1 : 0;
  return b;
}

__device__ __forceinline__ int key_offset(int key) { return kOffMask - (key & kOffMask); }

// Interval of x in one pair's table (see dpc_range in dpc.h).  Always float64.
// The range ends come from the host and the node is rounded on its own (no
// fused multiply-add), so every x gets the interval and offset that a plain
// evaluation of the same formulas gives.  NaN takes the clamped branch.
__device__ __forceinline__ void locate(const PairRange& P, double x, int& l, double& t,
                                       bool& clamped) {
#pragma clang fp contract(off)
  // one division: origin, stride and last index of the part (main range or
  // band) that x falls in are selected first, so lanes do not diverge
  const bool main = x < P.x_up;
  const double org = main ? P.lo : P.x_up, d = main ? P.d1 : P.d2;
  double q = floor((x - org) / d);
  q = fmin(fmax(q, 0.0), (double)((main ? P.L1 : P.L2) - 1));
  l = (main ? 0 : P.L1) + (int)q;
  const double node = org + q * d;
  t = x - node;
  clamped = !(x < P.x_end);
  if (clamped) {
    l = P.L1 + P.L2 - 1;
    t = P.d2;
  }
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The NB atoms of a wavefront.  A workgroup takes kWaves * NB consecutive
// atoms.  With several types it hands them to its wavefronts grouped by type
// (atoms of an invalid type after the others, index order inside a group),
// so that the atoms of one wavefront share their tables as often as
// possible: more records per interval.  An atom's records and sums do not
// depend on which atoms share its wavefront; only the chunk set its sums
// start from does (the start rotates with the wavefront), i.e. the order of
// rounding.  idx[a] is the atom's index, -1 past
// nloc (those come last); lane a < NB of `lanes` holds idx[a] as well, for
// lookups with an index known only at run time (a register array indexed so
// would go to scratch memory).
template <int NB>
struct WaveAtoms {
  int idx[NB];
  int lanes;
};

template <int NB, bool kOne>
__device__ __forceinline__ WaveAtoms<NB> wave_atoms(const Geo& g, const int* __restrict__ atype,
                                                    int lane, int wave) {
  constexpr int kG = kWaves * NB;
  static_assert(kG <= kLanes, "one lane per atom of the workgroup");
  WaveAtoms<NB> w;
  const int base = (int)blockIdx.x * kG;
  if (kOne || g.ntypes == 1) {
#pragma unroll
    for (int a = 0; a < NB; ++a) {
      const int i = base + wave * NB + a;
      w.idx[a] = __builtin_amdgcn_readfirstlane(i < g.nloc ? i : -1);
    }
    const int il = base + wave * NB + lane;
    w.lanes = lane < NB && il < g.nloc ? il : -1;
    return w;
  }
  const int at = base + lane;
  const bool in = lane < kG && at < g.nloc;
  int key = 0;
  if (in) {
    const int t = atype[at];
    key = t >= 0 && t < g.ntypes ? t : g.ntypes;
  }
  // position of this lane's atom in the order (key, index)
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  int pos = 0;
#pragma unroll
  for (int v = 0; v <= DPC_MAX_TYPES; ++v) {
    const uint64_t m = __ballot(in && key == v);
    pos += v < key ? __popcll(m) : (v == key ? __popcll(m & below) : 0);
  }
  w.lanes = -1;
#pragma unroll
  for (int a = 0; a < NB; ++a) {
    const uint64_t hit = __ballot(in && pos == wave * NB + a);
    w.idx[a] = __builtin_amdgcn_readfirstlane(hit ? base + (int)__builtin_ctzll(hit) : -1);
    w.lanes = lane == a ? w.idx[a] : w.lanes;
  }
  return w;
}

// idx[a] for an index a in [0, NB) that is the same in every lane
template <int NB>
__device__ __forceinline__ int atom_of(const WaveAtoms<NB>& w, int a) {
  return __builtin_amdgcn_readlane(w.lanes, a);
}

// idx[a] for a per-lane index a in [0, NB)
template <int NB>
__device__ __forceinline__ int lane_atom_of(const WaveAtoms<NB>& w, int a) {
  return __builtin_amdgcn_ds_bpermute(a << 2, w.lanes);
}

__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

__device__ __forceinline__ int readlane(int v, int lane) {
  return __builtin_amdgcn_readlane(v, lane);
}

template <typename TI>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const TI* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, bytes, 0x00020000);
}

// Coefficients of t^q (q = 0..5) of the lane's CPL channels of the interval
// whose coefficients start at element `off`; voff = byte offset of the lane's
// first channel inside a power pair (see DPC_TABLE_AT: power pair j holds
// (t^2j, t^(2j+1)) per channel, so the lane reads 2 * CPL consecutive
// elements per pair).  Every lane loads (lanes without channels read the
// last entries again), so the number of loads in flight is fixed.
template <typename TI, int CPL>
__device__ __forceinline__ void load_coef(__amdgpu_buffer_rsrc_t rs, int off, int ld, int voff,
                                          TI (&cf)[6][CPL]) {
  constexpr int kBytes = 2 * CPL * (int)sizeof(TI);     // per power pair
  constexpr int kLoads = kBytes >= 16 ? kBytes / 16 : 1;
  constexpr int kPer = kBytes >= 16 ? 16 / (int)sizeof(TI) : 2 * CPL;   // elements per load
  const int soff = off * (int)sizeof(TI);
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const int vo = voff + j * 2 * ld * (int)sizeof(TI);
    TI e[2 * CPL];
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      if constexpr (kBytes >= 16) {
        const v4i a = __builtin_amdgcn_raw_buffer_load_b128(rs, vo + 16 * i, soff, 0);
        __builtin_memcpy(e + kPer * i, &a, 16);
      } else {
        const v2i a = __builtin_amdgcn_raw_buffer_load_b64(rs, vo, soff, 0);
        __builtin_memcpy(e, &a, 8);
      }
    }
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      cf[2 * j][h] = e[2 * h];
      cf[2 * j + 1][h] = e[2 * h + 1];
    }
  }
}

// ---------------------------------------------------------------------------
// Chunk sets (shared by both passes)
// ---------------------------------------------------------------------------
struct Tables {
  int n, nruns;                // records and runs of the chunk set
  int rank;                    // this lane's slot: merged position, -1 padding, -2 no row
  int vs;                      // lane r: start of run r (n for r >= nruns)
  int vk;                      // lane r: key of run min(r, nruns - 1)
  int vp[2];                   // lane r: first record of atoms 1..NB-1 in run r, 8 bits each
};

// First record of atom b (0 < b < NB) in a run, from its packed split points.
template <int NB>
__device__ __forceinline__ int split_at(const int (&p)[2], int b) {
  return (p[(b - 1) >> 2] >> (8 * ((b - 1) & 3))) & 255;
}

// Validity of the slots of one window: kWindow / NB slots per atom starting
// at wbase, i.e. 32 slots per lane.  Bit k of lane l covers window index
// l + 64 k = a * (kWindow / NB) + (j - wbase) (atom a, slot j).  Only the
// sign of nlist is used, so one round trip to memory serves 32 chunk sets.
constexpr int kWindow = 32 * kLanes;

template <int NB>
__device__ __forceinline__ uint32_t valid_window(const Geo& g, const WaveAtoms<NB>& wa, int wbase,
                                                 const int* __restrict__ nlist, int lane) {
  constexpr int W = kWindow / NB;
  constexpr int kGroup = 8;   // loads in flight at once
  uint32_t vm = 0;
#pragma unroll 1
  for (int k0 = 0; k0 < 32; k0 += kGroup) {
    int v[kGroup];
    bool in[kGroup];
#pragma unroll
    for (int q = 0; q < kGroup; ++q) {
      const int il = lane + kLanes * (k0 + q);
      // W is a multiple of 64: the atom slot is the same in every lane
      const int ia = atom_of<NB>(wa, kLanes * (k0 + q) / W), j = wbase + il % W;
      in[q] = ia >= 0 && j < g.nnei;
      // out-of-range entries read slot 0 of atom idx[0] (always present) and are masked below
      v[q] = __builtin_nontemporal_load(nlist + (in[q] ? (size_t)ia * g.nnei + j
                                                       : (size_t)wa.idx[0] * g.nnei));
    }
#pragma unroll
    for (int q = 0; q < kGroup; ++q) vm |= (in[q] && v[q] >= 0 ? 1u : 0u) << (k0 + q);
  }
  return vm;
}

// Chunk sets of a window that hold at least one valid slot (bit c: chunk set
// c of the window's 32).  Bit k of lane l covers window index l + 64 k, i.e.
// atom k / (32 / NB) and chunk set NB (k mod 32 / NB) + l / (64 / NB); the
// atoms are folded first, then one ballot per remaining bit.
template <int NB>
__device__ __forceinline__ uint32_t occupied_chunks(uint32_t vm) {
  constexpr int B = 32 / NB, kC = kLanes / NB;
  constexpr uint64_t seg = kC == 64 ? ~0ull : ((1ull << kC) - 1);
  uint32_t v = 0;
#pragma unroll
  for (int a = 0; a < NB; ++a) v |= vm >> (a * B);
  uint32_t occ = 0;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    const uint64_t bal = __ballot((v >> b) & 1);
#pragma unroll
    for (int c = 0; c < NB; ++c) occ |= ((bal >> (c * kC)) & seg) != 0 ? 1u << (NB * b + c) : 0u;
  }
  return occ;
}

// One R~ row (16-byte aligned: checked on the host).
template <typename TI>
__device__ __forceinline__ void load_row(const TI* p, TI (&r)[4]) {
  if constexpr (sizeof(TI) == 8) {
    typedef TI V2 __attribute__((ext_vector_type(2)));
    const V2 a = __builtin_nontemporal_load(reinterpret_cast<const V2*>(p));
    const V2 b = __builtin_nontemporal_load(reinterpret_cast<const V2*>(p) + 1);
    r[0] = a.x; r[1] = a.y; r[2] = b.x; r[3] = b.y;
  } else {
    typedef TI V4 __attribute__((ext_vector_type(4)));
    const V4 a = __builtin_nontemporal_load(reinterpret_cast<const V4*>(p));
    r[0] = a.x; r[1] = a.y; r[2] = a.z; r[3] = a.w;
  }
}

// One dE/dR~ row (16-byte aligned: checked on the host).
template <typename TA>
__device__ __forceinline__ void store_row(TA* p, const TA (&v)[4]) {
  if constexpr (sizeof(TA) == 8) {
    typedef TA V2 __attribute__((ext_vector_type(2)));
    __builtin_nontemporal_store(V2{v[0], v[1]}, reinterpret_cast<V2*>(p));
    __builtin_nontemporal_store(V2{v[2], v[3]}, reinterpret_cast<V2*>(p) + 1);
  } else {
    typedef TA V4 __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(V4{v[0], v[1], v[2], v[3]}, reinterpret_cast<V4*>(p));
  }
}

// Zero dE/dR~ rows of a chunk set without valid slots (slots s0 + lane % kC
// of atom `atom`, the wavefront's atom lane / kC; atoms past nloc or of an
// invalid type are skipped).
template <typename TA, int NB>
__device__ __forceinline__ void zero_rows(const Geo& g, const int (&ai)[NB], int atom, int s0,
                                          TA* __restrict__ dR, int lane) {
  constexpr int kC = kLanes / NB;
  const int a = lane / kC, j = s0 + lane % kC;
  int at = -1;
#pragma unroll
  for (int b = 0; b < NB; ++b)
    if (b == a) at = ai[b];
  if (at >= 0 && j < g.nnei) {
    const TA z[4] = {(TA)0, (TA)0, (TA)0, (TA)0};
    store_row(dR + ((size_t)atom * g.nnei + j) * 4, z);
  }
}

// Merge slots [s0, s0 + 64/NB) of the wave's NB atoms into W and build the
// run tables.  Lane l covers slot s0 + l % (64/NB) of the wavefront's atom
// l / (64/NB), whose index is `atom`.  In
// the backward pass (kBwd) clamped records get a zero R~ row.  With kPairs
// the lane also gets the index of its record's (interval, atom) pair among
// the chunk set's pairs in merged order (`pair`, -1 without a record), a
// pair being a maximal group of records with equal key and atom, and keeps
// its record in registers (`mine`) instead of writing it to z.
template <typename TI, typename TA, int NB, bool kBwd, bool kOne, bool kPairs = false>
__device__ __forceinline__ Tables build_chunk_set(const Geo& g, const int (&ai)[NB], int atom,
                                                  int s0, int wbase, uint32_t vm,
                                                  const TI* __restrict__ em, Rec<TI>* z,
                                                  ChunkScratch& W, int lane,
                                                  int* pair = nullptr, Rec<TI>* mine = nullptr,
                                                  bool use_pre = false, const TI* pre = nullptr) {
  constexpr int kC = kLanes / NB;
  const int a = lane / kC, sl = lane % kC, j = s0 + sl;
  int at = -1;
#pragma unroll
  for (int b = 0; b < NB; ++b)
    if (b == a) at = ai[b];
  // the lane of the window masks that holds this slot's bit
  const int il = a * (kWindow / NB) + (s0 - wbase) + sl;
  const int holder = __builtin_amdgcn_ds_bpermute((il & 63) << 2, (int)vm);
  bool valid = false;
  Rec<TI> rec;
  if constexpr (kPairs) rec = Rec<TI>{0.0, 0.0, {(TI)0, (TI)0, (TI)0, (TI)0}};
  int key = 0;
  if (at >= 0 && j < g.nnei) {
    const size_t row = (size_t)atom * g.nnei + j;
    valid = (holder >> (il >> 6)) & 1;
    if (valid) {
      if (use_pre) {    // the caller has loaded the row already
#pragma unroll
        for (int k = 0; k < 4; ++k) rec.r[k] = pre[k];
      } else {
        load_row(em + row * 4, rec.r);
      }
      // one type (kOne): the pair range is uniform (scalar loads); else per lane
      int blk = 0;
      PairRange P;
      if constexpr (kOne) {
        P = g.pr[0];
      } else {
        blk = block_of(g, j);
        P = g.pr[at * g.ntypes + blk];
      }
      int l;
      bool cl;
      locate(P, (double)rec.r[0], l, rec.t, cl);
      rec.pad = 0.0;
      key = (blk << kOffBits) | (kOffMask - (P.offset + l * 6 * g.ld));
      // beyond the table the derivative term vanishes: a zero row removes it
      // (a NaN or infinite x keeps its row, so that it propagates)
      if (kBwd && cl && isfinite(rec.r[0])) {
#pragma unroll
        for (int k = 0; k < 4; ++k) rec.r[k] = (TI)0;
      }
    }
  }
  const int has_row = at >= 0 && j < g.nnei;
  const uint64_t m = __ballot(valid);
  if constexpr (kPairs) *pair = -1;
  if (m == 0) return Tables{0, 0, has_row ? -1 : -2, 0, 0, {0, 0}};
  const uint64_t seg = kC == 64 ? ~0ull : ((1ull << kC) - 1);
  const uint64_t before_seg = a == 0 ? 0ull : ((1ull << (a * kC)) - 1);
  const int pos = lanes_below(m) - __popcll(m & before_seg);
  int r = pos;
  if constexpr (NB > 1) {
    // Each atom's list of keys, padded to kC entries with 0xFFFFFFFF (above
    // every key): every lane writes one entry, and the searches below need
    // no bounds.  Keys are below 2^31 (block < 8), so key + 1 cannot wrap.
    uint32_t* lk = reinterpret_cast<uint32_t*>(W.rk);  // free until the run tables are written
    const int cnt_a = __popcll((m >> (a * kC)) & seg);
    lk[a * kC + (valid ? pos : cnt_a + sl - pos)] = valid ? (uint32_t)key : 0xFFFFFFFFu;
    wave_sync();
    const bool bad = sl + 1 < kC && lk[lane] > lk[lane + 1];
    const bool sorted = __ballot(bad) == 0;
    if (sorted) {
      // Records of list b that come first: smaller key, or equal key of a
      // lower atom, i.e. keys below thr[b].  The NB lower-bound searches run
      // side by side, one round trip to LDS per step for all lists.
      uint32_t thr[NB];
      int c[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        thr[b] = (uint32_t)key + (b < a ? 1u : 0u);
        c[b] = 0;
      }
#pragma unroll
      for (int step = kC / 2; step > 0; step >>= 1) {
        uint32_t kk[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) kk[b] = lk[b * kC + c[b] + step - 1];
#pragma unroll
        for (int b = 0; b < NB; ++b) c[b] += kk[b] < thr[b] ? step : 0;
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const uint32_t kk = lk[b * kC + c[b]];
        r += b == a ? 0 : c[b] + (kk < thr[b] ? 1 : 0);
      }
    } else {
#pragma unroll
      for (int b = 0; b < NB; ++b) r += b < a ? __popcll((m >> (b * kC)) & seg) : 0;
    }
  }
  if constexpr (kPairs) *mine = rec;
  if (valid) {
    if constexpr (!kPairs) z[r] = rec;
    W.mk[r] = key;
    W.mi[r] = j | (a << 20);
  }
  wave_sync();

  Tables T;
  T.rank = valid ? r : (has_row ? -1 : -2);
  T.n = __popcll(m);
  const bool in = lane < T.n;
  const int ke = W.mk[lane], ae = (W.mi[lane] >> 20) & 7;
  const int kp = W.mk[lane > 0 ? lane - 1 : 0];
  const bool f = in && (lane == 0 || ke != kp);
  const uint64_t F = __ballot(f);
  T.nruns = __popcll(F);
  if (f) {
    const int rr = lanes_below(F);
    W.rk[rr] = ke;
    W.rs[rr] = lane;
  }
  if (lane == 0) W.rs[T.nruns] = T.n;
  if constexpr (kPairs) {
    const int ap = (W.mi[lane > 0 ? lane - 1 : 0] >> 20) & 7;
    const uint64_t F2 = __ballot(in && (lane == 0 || ke != kp || ae != ap));
    wave_sync();              // every lane has read mk: it now takes the pair indices
    W.mk[lane] = lanes_below(F2) + (int)((F2 >> lane) & 1) - 1;
  }
  wave_sync();
  if constexpr (kPairs) *pair = valid ? W.mk[r] : -1;
  const int S = W.rs[min(lane, T.nruns)], E = W.rs[min(lane + 1, T.nruns)];
  T.vs = S;
  T.vk = W.rk[min(lane, max(T.nruns - 1, 0))];
  // records of run r are [S, E); inside it atoms come in increasing order
  const uint64_t run_mask = (E >= 64 ? ~0ull : ((1ull << E) - 1)) & ~(S >= 64 ? ~0ull : ((1ull << S) - 1));
  T.vp[0] = T.vp[1] = 0;
#pragma unroll
  for (int b = 1; b < NB; ++b) {
    const uint64_t below = __ballot(in && ae < b);
    const int p = S + __popcll(below & run_mask);
    T.vp[(b - 1) >> 2] |= p << (8 * ((b - 1) & 3));
  }
  wave_sync();
  return T;
}

// ---------------------------------------------------------------------------
// forward: T and D
// ---------------------------------------------------------------------------
// The epilogue reuses the chunk-set LDS of the wave for the atom's T rows.
template <typename TI, typename TA>
__host__ __device__ constexpr size_t fwd_wave_bytes(int m1) {
  return align16(sizeof(WaveLds<TI>)) > align16((size_t)m1 * 4 * sizeof(TA))
             ? align16(sizeof(WaveLds<TI>))
             : align16((size_t)m1 * 4 * sizeof(TA));
}

template <typename TA>
using Pair = TA __attribute__((ext_vector_type(2)));

// kOne: all atoms and neighbours have one type (one table, no blocks)
template <typename TI, typename TA, int CPL, int NB, bool kOne>
// up to 128 channels: registers capped so that 3 wavefronts fit on a SIMD
__global__ __launch_bounds__(64 * kWaves)
__attribute__((amdgpu_waves_per_eu(CPL <= 2 ? 3 : 1))) void se_a_fwd_kernel(
    const Geo g, const TI* __restrict__ coeff, const int* __restrict__ atype,
    const int* __restrict__ nlist, const TI* __restrict__ em, TA* __restrict__ T,
    TA* __restrict__ D) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int kC = kLanes / NB;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const WaveAtoms<NB> wa = wave_atoms<NB, kOne>(g, atype, lane, wave);
  if (wa.idx[0] < 0) return;
  const int my_atom = lane_atom_of<NB>(wa, lane / kC);   // the atom of this lane's chunk-set slots
  const int nnei = g.nnei, m1 = g.m1, m2 = g.m2, ld = g.ld;
  const uint32_t zoff = __builtin_amdgcn_readfirstlane(wave * (uint32_t)fwd_wave_bytes<TI, TA>(m1));
  unsigned char* wb = smem + zoff;
  WaveLds<TI>& W = *reinterpret_cast<WaveLds<TI>*>(wb);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(coeff, g.coeff_bytes);
  const int voff = 2 * min(lane * CPL, ld - CPL) * (int)sizeof(TI);

  int ai[NB];
#pragma unroll
  for (int a = 0; a < NB; ++a) {
    const int i = wa.idx[a];
    ai[a] = -1;
    if (i >= 0) {
      const int t = __builtin_amdgcn_readfirstlane(atype[i]);
      if (t < 0 || t >= g.ntypes) {  // invalid type: the atom's outputs become NaN
        const TA nan = (TA)NAN;
        for (int e = lane; e < m1 * 4; e += 64) T[(size_t)i * m1 * 4 + e] = nan;
        for (int e = lane; e < m1 * m2; e += 64) D[(size_t)i * m1 * m2 + e] = nan;
      } else {
        ai[a] = t;
      }
    }
  }
  TA acc[NB][CPL][4];
#pragma unroll
  for (int a = 0; a < NB; ++a) {
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[a][h][k] = (TA)0;
    }
  }
  TI cfA[6][CPL], cfB[6][CPL];
  // lanes without channels (lane * CPL >= m1) load coefficients like the
  // others, so that every load stays unconditional, but skip the arithmetic:
  // idle float64 FMAs still draw power, and this kernel runs at a lower
  // clock than the rest
  const bool active = lane * CPL < m1;

  // Chunk sets are visited cyclically from a start that differs between
  // wavefronts, so that waves sharing a SIMD are not all building (a
  // latency-bound phase) at the same time.
  const int nch = (nnei + kC - 1) / kC;
  int s0 = ((int)(blockIdx.x * 5 + wave * 3) % nch) * kC;
  uint32_t vm = 0, occ = 0;
  for (int cc = 0, wbase = -1; cc < nch; ++cc, s0 = s0 + kC < nnei ? s0 + kC : 0) {
    if (s0 - s0 % (kWindow / NB) != wbase) {  // window of nlist signs holding s0
      wbase = s0 - s0 % (kWindow / NB);
      vm = valid_window<NB>(g, wa, wbase, nlist, lane);
      occ = occupied_chunks<NB>(vm);
    }
    if (!((occ >> ((s0 - wbase) / kC)) & 1)) continue;   // padding only
    const Tables tb = build_chunk_set<TI, TA, NB, false, kOne>(g, ai, my_atom, s0, wbase, vm, em, W.z, W.s, lane);
    if (tb.n == 0) continue;
    load_coef<TI, CPL>(rs, key_offset(readlane(tb.vk, 0)), ld, voff, cfA);
    int r = 0;
    // run r with `cur` loaded; the next run's coefficients go to `nxt`
    auto run = [&](TI (&cur)[6][CPL], TI (&nxt)[6][CPL]) __attribute__((always_inline)) {
      load_coef<TI, CPL>(rs, key_offset(readlane(tb.vk, min(r + 1, kLanes - 1))), ld, voff,
                         nxt);
      const int S = readlane(tb.vs, r);
      const int E = r + 1 < kLanes ? readlane(tb.vs, r + 1) : tb.n;
      int p[2] = {0, 0};
      if constexpr (NB > 1) p[0] = readlane(tb.vp[0], r);
      if constexpr (NB > 5) p[1] = readlane(tb.vp[1], r);
      auto one = [&](const Rec<TI>& c, auto& ac) __attribute__((always_inline)) {
        const TI t = (TI)c.t;
#pragma unroll
        for (int h = 0; h < CPL; ++h) {
          TI v = cur[5][h];
          v = fma(v, t, cur[4][h]);
          v = fma(v, t, cur[3][h]);
          v = fma(v, t, cur[2][h]);
          v = fma(v, t, cur[1][h]);
          v = fma(v, t, cur[0][h]);
#pragma unroll
          for (int k = 0; k < 4; ++k) ac[h][k] = fma((TA)v, (TA)c.r[k], ac[h][k]);
        }
      };
      if (!active) return;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int lo = b == 0 ? S : split_at<NB>(p, b);
        const int hi = b == NB - 1 ? E : split_at<NB>(p, b + 1);
        int e = lo;
        for (; e + 1 < hi; e += 2) {
          const Rec<TI> c0 = zrec<TI>(smem, zoff, e), c1 = zrec<TI>(smem, zoff, e + 1);
          one(c0, acc[b]);
          one(c1, acc[b]);
        }
        if (e < hi) {
          const Rec<TI> c0 = zrec<TI>(smem, zoff, e);
          one(c0, acc[b]);
        }
      }
    };
    for (;;) {
      run(cfA, cfB);
      if (++r == tb.nruns) break;
      run(cfB, cfA);
      if (++r == tb.nruns) break;
    }
    wave_sync();
  }

  // T and D = T (T<)^T of each atom.  The rows go through LDS so that both
  // outputs are written in flat order, consecutive lanes to consecutive
  // addresses; lane f of a D pass computes element f = m * m2 + n.
  TA* sT = reinterpret_cast<TA*>(wb);
  const int m_step = 64 / m2, n_step = 64 % m2;
#pragma unroll
  for (int a = 0; a < NB; ++a) {
    const int i = wa.idx[a];
    if (ai[a] < 0) continue;
    wave_sync();
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int m = lane * CPL + h;
      if (m < m1) {
        Pair<TA>* d = reinterpret_cast<Pair<TA>*>(sT + m * 4);
        d[0] = Pair<TA>{acc[a][h][0], acc[a][h][1]};
        d[1] = Pair<TA>{acc[a][h][2], acc[a][h][3]};
      }
    }
    wave_sync();
    TA* Ti = T + (size_t)i * m1 * 4;
    TA* Di = D + (size_t)i * m1 * m2;
    auto dot = [&](int m, int n) __attribute__((always_inline)) -> TA {
      const Pair<TA>* pm = reinterpret_cast<const Pair<TA>*>(sT + m * 4);
      const Pair<TA>* pn = reinterpret_cast<const Pair<TA>*>(sT + n * 4);
      const Pair<TA> a0 = pm[0], a1 = pm[1], b0 = pn[0], b1 = pn[1];
      TA v = a0.x * b0.x;
      v = fma(a0.y, b0.y, v);
      v = fma(a1.x, b1.x, v);
      return (TA)fma(a1.y, b1.y, v);
    };
    if (g.pair_out) {
      // two elements per lane and store
      for (int e = lane; e < m1 * 2; e += 64)
        __builtin_nontemporal_store(reinterpret_cast<const Pair<TA>*>(sT)[e],
                                    reinterpret_cast<Pair<TA>*>(Ti) + e);
      const int ms = 128 / m2, ns = 128 % m2;
      int m = (2 * lane) / m2, n = (2 * lane) % m2;
      for (int f2 = lane; f2 < m1 * m2 / 2; f2 += 64) {
        int mb = m, nb = n + 1;
        if (nb == m2) {
          nb = 0;
          ++mb;
        }
        __builtin_nontemporal_store(Pair<TA>{dot(m, n), dot(mb, nb)},
                                    reinterpret_cast<Pair<TA>*>(Di) + f2);
        m += ms;
        n += ns;
        if (n >= m2) {
          n -= m2;
          ++m;
        }
      }
    } else {
      for (int e = lane; e < m1 * 4; e += 64) __builtin_nontemporal_store(sT[e], Ti + e);
      int m = lane / m2, n = lane % m2;
      for (int f = lane; f < m1 * m2; f += 64) {
        __builtin_nontemporal_store(dot(m, n), Di + f);
        m += m_step;
        n += n_step;
        if (n >= m2) {
          n -= m2;
          ++m;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// backward: dE/dR~
// ---------------------------------------------------------------------------
// Cross-lane sums.  Record b of a batch writes (share[0], share[1]) of every
// lane to block 2b and (share[2], share[3]) to block 2b + 1, 16 bytes per
// lane, 64 lanes per block.  Blocks are kRedBlock = 1152 bytes apart (128 past
// a multiple of 256), so that the 16 lanes of two neighbouring blocks reading
// 16 bytes each touch every bank once.  Lanes without channels hold zeros
// (their dE/dT is zero), or NaN when the record is NaN, which then is NaN
// anyway.  Step 1: lane (G, x) = (lane / 8, lane % 8) adds strip x (lanes x,
// x + 8, ...) of block G; step 2: the 8 strips of each of the 16 sums are
// added by lane s = 4b + k, reading a row padded to 16 bytes past a multiple
// of 64 (no bank repeats).  The step 2 rows reuse the start of the blocks.
constexpr int kRedBlock = 1152;
template <typename TA>
__host__ __device__ constexpr int part_stride() {  // row of step 2, in TA units
  return 8 + 16 / (int)sizeof(TA);
}
template <typename TI>
__host__ __device__ constexpr size_t bwd_wave_bytes() {
  return align16(sizeof(WaveLds<TI>)) + (size_t)2 * kBatch * kRedBlock;
}

template <typename TI, typename TA, int CPL, int NB, bool kOne>
// up to 128 channels: registers capped so that 3 wavefronts fit on a SIMD
__global__ __launch_bounds__(64 * kWaves)
__attribute__((amdgpu_waves_per_eu(CPL <= 2 ? 3 : 1))) void se_a_bwd_kernel(
    const Geo g, const TI* __restrict__ coeff, const int* __restrict__ atype,
    const int* __restrict__ nlist, const TI* __restrict__ em, const TI* __restrict__ dT,
    TA* __restrict__ dR) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int kC = kLanes / NB;
  constexpr int PS = part_stride<TA>();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const WaveAtoms<NB> wa = wave_atoms<NB, kOne>(g, atype, lane, wave);
  if (wa.idx[0] < 0) return;
  const int my_atom = lane_atom_of<NB>(wa, lane / kC);   // the atom of this lane's chunk-set slots
  const int nnei = g.nnei, m1 = g.m1, ld = g.ld;
  static_assert(16 * part_stride<TA>() * sizeof(TA) <= 2 * kBatch * kRedBlock, "step 2 rows");
  const uint32_t zoff = __builtin_amdgcn_readfirstlane(wave * (uint32_t)bwd_wave_bytes<TI>());
  unsigned char* wb = smem + zoff;
  WaveLds<TI>& W = *reinterpret_cast<WaveLds<TI>*>(wb);
  unsigned char* red = wb + align16(sizeof(WaveLds<TI>));
  TA* part = reinterpret_cast<TA*>(red);
  unsigned char* const wlane = red + lane * 16;                          // record writes
  const unsigned char* const rlane =
      red + (lane >> 4) * 2 * kRedBlock + ((lane >> 3) & 1) * kRedBlock + (lane & 7) * 16;
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(coeff, g.coeff_bytes);
  const int voff = 2 * min(lane * CPL, ld - CPL) * (int)sizeof(TI);

  TA dt[NB][CPL][4];
  int ai[NB];
#pragma unroll
  for (int a = 0; a < NB; ++a) {
    const int i = wa.idx[a];
    ai[a] = -1;
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int m = lane * CPL + h;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        dt[a][h][k] = (i >= 0 && m < m1)
                          ? (TA)__builtin_nontemporal_load(dT + ((size_t)i * m1 + m) * 4 + k)
                          : (TA)0;
    }
    if (i >= 0) {
      const int t = __builtin_amdgcn_readfirstlane(atype[i]);
      if (t < 0 || t >= g.ntypes) {  // invalid type: the atom's outputs become NaN
        for (int e = lane; e < nnei * 4; e += 64) dR[(size_t)i * nnei * 4 + e] = (TA)NAN;
      } else {
        ai[a] = t;
      }
    }
  }
  TI cfA[6][CPL], cfB[6][CPL];
  int nb = 0;

  // sum the shares of the nbat records starting at merged position e0
  auto reduce = [&](int e0, int nbat) __attribute__((always_inline)) {
    wave_sync();
    Pair<TA> v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = *reinterpret_cast<const Pair<TA>*>(rlane + q * 128);
    Pair<TA> sum = v[0];
#pragma unroll
    for (int q = 1; q < 8; ++q) sum += v[q];
    wave_sync();
    const int G = lane >> 3, x = lane & 7;
    part[(2 * G) * PS + x] = sum.x;
    part[(2 * G + 1) * PS + x] = sum.y;
    wave_sync();
    if (lane < 4 * nbat) {
      // the batch's records have been read: their LDS slots take the results
      const Pair<TA>* pr = reinterpret_cast<const Pair<TA>*>(part + lane * PS);
      const Pair<TA> a = pr[0] + pr[1], b = pr[2] + pr[3];
      reinterpret_cast<TA*>(&W.z[e0 + (lane >> 2)])[lane & 3] = (a.x + a.y) + (b.x + b.y);
    }
    wave_sync();
  };
  static_assert(4 * sizeof(TA) <= sizeof(Rec<TI>), "a record slot holds one output row");

  // Chunk sets are visited cyclically from a start that differs between
  // wavefronts, so that waves sharing a SIMD are not all building (a
  // latency-bound phase) at the same time.
  const int nch = (nnei + kC - 1) / kC;
  int s0 = ((int)(blockIdx.x * 5 + wave * 3) % nch) * kC;
  uint32_t vm = 0, occ = 0;
  for (int cc = 0, wbase = -1; cc < nch; ++cc, s0 = s0 + kC < nnei ? s0 + kC : 0) {
    if (s0 - s0 % (kWindow / NB) != wbase) {  // window of nlist signs holding s0
      wbase = s0 - s0 % (kWindow / NB);
      vm = valid_window<NB>(g, wa, wbase, nlist, lane);
      occ = occupied_chunks<NB>(vm);
    }
    if (!((occ >> ((s0 - wbase) / kC)) & 1)) {   // padding only: zero rows
      zero_rows<TA, NB>(g, ai, my_atom, s0, dR, lane);
      continue;
    }
    const Tables tb = build_chunk_set<TI, TA, NB, true, kOne>(g, ai, my_atom, s0, wbase, vm, em, W.z, W.s, lane);
    // Each lane writes the dE/dR~ row of its own slot (zero for padding) after
    // the chunk set's runs: consecutive lanes, consecutive rows, and no store
    // ahead of the coefficient loads whose waits would then include it.
    auto write_rows = [&]() __attribute__((always_inline)) {
      if (tb.rank >= -1) {
        TA v[4] = {(TA)0, (TA)0, (TA)0, (TA)0};
        if (tb.rank >= 0) {
          const TA* src = reinterpret_cast<const TA*>(&W.z[tb.rank]);
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = src[k];
        }
        store_row(dR + ((size_t)my_atom * nnei + s0 + lane % kC) * 4, v);
      }
    };
    if (tb.n == 0) {
      write_rows();
      continue;
    }
    load_coef<TI, CPL>(rs, key_offset(readlane(tb.vk, 0)), ld, voff, cfA);
    int r = 0;
    auto run = [&](TI (&cur)[6][CPL], TI (&nxt)[6][CPL]) __attribute__((always_inline)) {
      load_coef<TI, CPL>(rs, key_offset(readlane(tb.vk, min(r + 1, kLanes - 1))), ld, voff,
                         nxt);
      const int S = readlane(tb.vs, r);
      const int E = r + 1 < kLanes ? readlane(tb.vs, r + 1) : tb.n;
      int p[2] = {0, 0};
      if constexpr (NB > 1) p[0] = readlane(tb.vp[0], r);
      if constexpr (NB > 5) p[1] = readlane(tb.vp[1], r);
      auto one = [&](const Rec<TI>& c, const auto& dtb, int e) __attribute__((always_inline)) {
        const TI t = (TI)c.t;
        TA p0 = 0, p1 = 0, p2 = 0, p3 = 0;
#pragma unroll
        for (int h = 0; h < CPL; ++h) {
          // value and derivative of the quintic by a joint Horner scheme
          TI v = cur[5][h], d = cur[5][h];
          v = fma(v, t, cur[4][h]);
          d = fma(d, t, v);
          v = fma(v, t, cur[3][h]);
          d = fma(d, t, v);
          v = fma(v, t, cur[2][h]);
          d = fma(d, t, v);
          v = fma(v, t, cur[1][h]);
          d = fma(d, t, v);
          v = fma(v, t, cur[0][h]);
          TA w = dtb[h][0] * (TA)c.r[0];
          w = fma(dtb[h][1], (TA)c.r[1], w);
          w = fma(dtb[h][2], (TA)c.r[2], w);
          w = fma(dtb[h][3], (TA)c.r[3], w);
          p0 = fma(dtb[h][0], (TA)v, fma((TA)d, w, p0));
          p1 = fma(dtb[h][1], (TA)v, p1);
          p2 = fma(dtb[h][2], (TA)v, p2);
          p3 = fma(dtb[h][3], (TA)v, p3);
        }
        unsigned char* o = wlane + nb * (2 * kRedBlock);
        *reinterpret_cast<Pair<TA>*>(o) = Pair<TA>{p0, p1};
        *reinterpret_cast<Pair<TA>*>(o + kRedBlock) = Pair<TA>{p2, p3};
        if (++nb == kBatch) {
          reduce(e + 1 - kBatch, kBatch);
          nb = 0;
        }
      };
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int lo = b == 0 ? S : split_at<NB>(p, b);
        const int hi = b == NB - 1 ? E : split_at<NB>(p, b + 1);
        int e = lo;
        for (; e + 1 < hi; e += 2) {
          const Rec<TI> c0 = zrec<TI>(smem, zoff, e), c1 = zrec<TI>(smem, zoff, e + 1);
          one(c0, dt[b], e);
          one(c1, dt[b], e + 1);
        }
        if (e < hi) {
          const Rec<TI> c0 = zrec<TI>(smem, zoff, e);
          one(c0, dt[b], e);
        }
      }
    };
    for (;;) {
      run(cfA, cfB);
      if (++r == tb.nruns) break;
      run(cfB, cfA);
      if (++r == tb.nruns) break;
    }
    if (nb > 0) {
      reduce(tb.n - nb, nb);
      nb = 0;
    }
    wave_sync();
    write_rows();
    wave_sync();
  }
}

// ---------------------------------------------------------------------------
// backward, float64, M1 <= 128: channel sums on the matrix cores
// ---------------------------------------------------------------------------
// For one interval (coefficients C[m][q], g_m(t) = sum_q C[m][q] t^q) and
// one atom (dE/dT rows dT[m][k]) both channel sums of a record factor
// through the 4 x 6 matrix P[k][q] = sum_m dT[m][k] C[m][q]:
//   sum_m dT[m][k] g_m(t)                  = sum_q t^q P[k][q]
//   sum_m g'_m(t) sum_k' dT[m][k'] R~[k']  = sum_k' R~[k'] sum_q q t^(q-1) P[k'][q].
// P of each (interval, atom) pair of a chunk set comes from two chains of
// v_mfma_f64_4x4x4f64 (even powers 0, 2, 4, 6 and odd powers 1, 3, 5, 7, of
// which 6 and 7 are not used), and each record then costs a few dozen
// operations in the lane that holds it.
//
// v_mfma_f64_4x4x4f64 computes four independent 4x4 products D_b = A_b B_b
// (+ C_b).  Lane L = 16 kk + 4 b + x holds A_b[x][kk] and B_b[kk][x]; D_b[i][j]
// sits in lane 16 i + 4 b + j (measured on gfx950).  Block b = h takes the
// channels m = h (mod 4); A_b = dT^T of those channels (rows k), B_b their
// coefficients (column x of chain c = power 2x + c).  K step s of block h
// covers the channels 16 s + 4 kk + h, and one 16-byte read of the power pair
// (2x, 2x + 1) of a channel gives a lane its B operands of both chains.  The
// four blocks' products are summed across lanes (DPP row shifts) into the
// lanes of block 3, which store P.
//
// The B operands are not loaded from the table directly (S loads per interval
// and lane, 7 for M1 = 100): an interval's coefficients are copied densely
// into a per-wavefront LDS slot by NS wave-wide 16-byte buffer loads that
// write LDS themselves (5 for M1 = 100), and read from there.  The vector
// memory address unit then does 5/7 of the work, and the copy takes neither
// registers nor LDS write instructions.  In a slot, row x (power pair x)
// starts 16 ld bytes after row x - 1; the 16 lanes of one K index kk read the
// channels 16 s + 4 kk + h of rows x = 0..2, i.e. 16-byte bank groups
// 4 x + h + const (mod 16) when ld = 4 (mod 16) (M1 = 100: ld = 100), which
// are distinct.  Reads past channel M1 (zero A operands) fall into the next
// row or past the interval, inside the slot.
constexpr int kMfmaAtoms = 4;      // atoms per wavefront in the matrix-core kernel

// 16-byte loads that copy one interval: its 6 ld elements and the reads of
// the last K step (up to channel 16 S - 1 of row 2) fit in NS KiB; a power
// pair of one channel is 2 esize bytes (16 for float64, 8 for float32).
__host__ __device__ constexpr int mfma_slot_kib(int S, int ld, int esize = 8) {
  return ((2 * ld + 16 * S) * 2 * esize + 1023) / 1024;
}

// The (interval, atom) products are stored as rows of 6 doubles, 26 doubles
// (13 bank groups) apart, so that the records of up to 16 different products
// read without conflicts; pair_slots of them are held at once.  Four
// wavefronts' LDS stays at or below 53,312 bytes, so that three workgroups
// share a CU (measured: 53,824 bytes leave room for two).
constexpr int kPairDoubles = 26;   // one product in LDS: 4 rows of 6 + 2 padding
constexpr int kMfmaWaveLds = 53312 / kWaves;
__host__ __device__ constexpr int pair_slots(int ns) {
  return ((kMfmaWaveLds - (int)align16(sizeof(ChunkScratch)) - 1024 * ns) /
              (kPairDoubles * (int)sizeof(double)) / 4 * 4 > 32
              ? 32
              : (kMfmaWaveLds - (int)align16(sizeof(ChunkScratch)) - 1024 * ns) /
                    (kPairDoubles * (int)sizeof(double)) / 4 * 4);
}
__host__ __device__ constexpr size_t bwdm_wave_bytes(int ns) {
  return align16(sizeof(ChunkScratch)) + (size_t)pair_slots(ns) * kPairDoubles * sizeof(double) +
         (size_t)1024 * ns;
}

__device__ __forceinline__ double mfma4(double a, double b, double c) {
  return __builtin_amdgcn_mfma_f64_4x4x4f64(a, b, c, 0, 0, 0);
}

// v from lane l - N of the same row of 16 lanes (0 for the first N lanes)
template <int N>
__device__ __forceinline__ double row_shr(double v) {
  const v2i a = __builtin_bit_cast(v2i, v);
  v2i r;
  r.x = __builtin_amdgcn_update_dpp(0, a.x, 0x110 | N, 0xF, 0xF, true);
  r.y = __builtin_amdgcn_update_dpp(0, a.y, 0x110 | N, 0xF, 0xF, true);
  return __builtin_bit_cast(double, r);
}

// The slot is written by buffer loads (counted in vmcnt) that the compiler
// does not order against LDS instructions it emits itself: it would wait for
// all of them before every LDS access.  Inside the run loop all LDS accesses
// are therefore written out here, each block ending in its own lgkmcnt(0),
// and the loop waits for the copy explicitly.
__device__ __forceinline__ uint32_t lds_addr(const unsigned char* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) unsigned char*)p;
}

// q[st] = 16 bytes at a + 256 st (S reads)
template <int S>
__device__ __forceinline__ void lds_read_steps(uint32_t a, v4i (&q)[S]) {
  static_assert(S >= 1 && S <= 8, "K steps");
#define DPC_R(i, off) "ds_read_b128 %" #i ", %[a] offset:" #off "\n\t"
  if constexpr (S == 1)
    asm volatile(DPC_R(0, 0) "s_waitcnt lgkmcnt(0)" : "=&v"(q[0]) : [a] "v"(a) : "memory");
  else if constexpr (S == 2)
    asm volatile(DPC_R(0, 0) DPC_R(1, 256) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]) : [a] "v"(a) : "memory");
  else if constexpr (S == 3)
    asm volatile(DPC_R(0, 0) DPC_R(1, 256) DPC_R(2, 512) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]) : [a] "v"(a) : "memory");
  else if constexpr (S == 4)
    asm volatile(DPC_R(0, 0) DPC_R(1, 256) DPC_R(2, 512) DPC_R(3, 768) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]) : [a] "v"(a) : "memory");
  else if constexpr (S == 5)
    asm volatile(DPC_R(0, 0) DPC_R(1, 256) DPC_R(2, 512) DPC_R(3, 768) DPC_R(4, 1024) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4])
                 : [a] "v"(a) : "memory");
  else if constexpr (S == 6)
    asm volatile(DPC_R(0, 0) DPC_R(1, 256) DPC_R(2, 512) DPC_R(3, 768) DPC_R(4, 1024) DPC_R(5, 1280) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4]), "=&v"(q[5])
                 : [a] "v"(a) : "memory");
  else if constexpr (S == 7)
    asm volatile(DPC_R(0, 0) DPC_R(1, 256) DPC_R(2, 512) DPC_R(3, 768) DPC_R(4, 1024) DPC_R(5, 1280) DPC_R(6, 1536)
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4]), "=&v"(q[5]),
                   "=&v"(q[6])
                 : [a] "v"(a) : "memory");
  else
    asm volatile(DPC_R(0, 0) DPC_R(1, 256) DPC_R(2, 512) DPC_R(3, 768) DPC_R(4, 1024) DPC_R(5, 1280) DPC_R(6, 1536) DPC_R(7, 1792)
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4]), "=&v"(q[5]),
                   "=&v"(q[6]), "=&v"(q[7])
                 : [a] "v"(a) : "memory");
#undef DPC_R
}

// q[st] = 8 bytes at a + 128 st (S reads): float32 power pairs
template <int S>
__device__ __forceinline__ void lds_read_steps_b64(uint32_t a, v2i (&q)[S]) {
  static_assert(S >= 1 && S <= 8, "K steps");
#define DPC_R(i, off) "ds_read_b64 %" #i ", %[a] offset:" #off "\n\t"
  if constexpr (S == 1)
    asm volatile(DPC_R(0, 0) "s_waitcnt lgkmcnt(0)" : "=&v"(q[0]) : [a] "v"(a) : "memory");
  else if constexpr (S == 2)
    asm volatile(DPC_R(0, 0) DPC_R(1, 128) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]) : [a] "v"(a) : "memory");
  else if constexpr (S == 3)
    asm volatile(DPC_R(0, 0) DPC_R(1, 128) DPC_R(2, 256) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]) : [a] "v"(a) : "memory");
  else if constexpr (S == 4)
    asm volatile(DPC_R(0, 0) DPC_R(1, 128) DPC_R(2, 256) DPC_R(3, 384) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]) : [a] "v"(a) : "memory");
  else if constexpr (S == 5)
    asm volatile(DPC_R(0, 0) DPC_R(1, 128) DPC_R(2, 256) DPC_R(3, 384) DPC_R(4, 512) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4])
                 : [a] "v"(a) : "memory");
  else if constexpr (S == 6)
    asm volatile(DPC_R(0, 0) DPC_R(1, 128) DPC_R(2, 256) DPC_R(3, 384) DPC_R(4, 512) DPC_R(5, 640) "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4]), "=&v"(q[5])
                 : [a] "v"(a) : "memory");
  else if constexpr (S == 7)
    asm volatile(DPC_R(0, 0) DPC_R(1, 128) DPC_R(2, 256) DPC_R(3, 384) DPC_R(4, 512) DPC_R(5, 640) DPC_R(6, 768)
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4]), "=&v"(q[5]),
                   "=&v"(q[6])
                 : [a] "v"(a) : "memory");
  else
    asm volatile(DPC_R(0, 0) DPC_R(1, 128) DPC_R(2, 256) DPC_R(3, 384) DPC_R(4, 512) DPC_R(5, 640) DPC_R(6, 768) DPC_R(7, 896)
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4]), "=&v"(q[5]),
                   "=&v"(q[6]), "=&v"(q[7])
                 : [a] "v"(a) : "memory");
#undef DPC_R
}

// Two rows (12 doubles) of a product at a (6 reads of 16 bytes).
__device__ __forceinline__ void lds_read_rows2(uint32_t a, v4i (&q)[6]) {
  asm volatile(
      "ds_read_b128 %0, %[a]\n\tds_read_b128 %1, %[a] offset:16\n\t"
      "ds_read_b128 %2, %[a] offset:32\n\tds_read_b128 %3, %[a] offset:48\n\t"
      "ds_read_b128 %4, %[a] offset:64\n\tds_read_b128 %5, %[a] offset:80\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(q[0]), "=&v"(q[1]), "=&v"(q[2]), "=&v"(q[3]), "=&v"(q[4]), "=&v"(q[5])
      : [a] "v"(a)
      : "memory");
}

__device__ __forceinline__ void lds_write16(uint32_t a, v4i v) {
  asm volatile("ds_write_b128 %0, %1" : : "v"(a), "v"(v) : "memory");
}

// vmcnt(0) only; the empty asm keeps memory accesses on their side of it
__device__ __forceinline__ void wait_copies() {
  __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8));
  __asm__ __volatile__("" ::: "memory");
}

// up to 128 channels: registers capped so that 3 wavefronts fit on a SIMD
// The A operands of the wavefront's NB atoms from T and dE/dD (the
// descriptor backward), on the matrix cores.  Both sums are 4 x 4 x 4
// products whose output layout is the A operand layout itself: output lane
// L = 16 i + 4 b + j of block b holds channel 16 s + 4 i + b, column j, which
// is where the A operand of K step s wants dE/dT[16 s + (L >> 2)][L & 3].
//   first sum,  K = n < M':   A_b[x][kk] = dE/dD[16 s + 4 x + b][n(kk)],  B_b[kk][x] = T[n(kk)][x]
//   second sum, K = m' < M1:  A_b[x][kk] = dE/dD[m'(kk)][4 x + b],        B_b[kk][x] = T[m'(kk)][x]
// (the second only into step s = 0, output channels 4 x + b < M' <= 16).  In
// the first sum the K steps come in pairs n = 8 q + 2 kk + {0, 1}, so one
// 16-byte load gives a lane the A operands of two steps.  Operands outside
// M1, M' are zero (loads clamped inside the atom's rows); atoms past nloc
// get zeros.  T and dE/dD are read straight from memory (the second sum
// re-reads dE/dD rows the first sum has just brought into the caches).
template <int NB, int S>
__device__ __forceinline__ void descriptor_bwd_operands(const Geo& g, const WaveAtoms<NB>& wa,
                                                        const double* __restrict__ Tin,
                                                        const double* __restrict__ dD, int lane,
                                                        double (&A)[NB][S]) {
  typedef double D2 __attribute__((ext_vector_type(2)));
  const int m1 = g.m1, m2 = g.m2;
  const int kk = lane >> 4, b = (lane >> 2) & 3, x = lane & 3;
  const int nq = (m2 + 7) >> 3;           // 16-byte K pairs of the first sum (M' <= 16: 1 or 2)
  const int np = (m1 + 3) >> 2;           // K steps of the second sum
  const int col = 4 * x + b;              // second sum: the output channel of the lane's A row
#pragma unroll
  for (int a = 0; a < NB; ++a) {
    const bool live = wa.idx[a] >= 0;
    const int i = live ? wa.idx[a] : wa.idx[0];
    const double* Ta = Tin + (size_t)i * m1 * 4;
    const double* Da = dD + (size_t)i * m1 * m2;
    double acc[S];
#pragma unroll
    for (int s = 0; s < S; ++s) acc[s] = 0.0;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      if (q >= nq) break;
      const int n = 8 * q + 2 * kk;
      const bool nv = n < m2;             // m2 even: n + 1 < m2 too
      const int nc = nv ? n : 0;
      const double b0 = nv ? Ta[nc * 4 + x] : 0.0, b1 = nv ? Ta[nc * 4 + 4 + x] : 0.0;
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const int m = 16 * s + 4 * x + b;
        const bool ok = nv && m < m1;
        const D2 v = *reinterpret_cast<const D2*>(Da + (size_t)min(m, m1 - 1) * m2 + nc);
        acc[s] = mfma4(ok ? v.x : 0.0, b0, acc[s]);
        acc[s] = mfma4(ok ? v.y : 0.0, b1, acc[s]);
      }
    }
    const bool cv = col < m2;
    const int cc = cv ? col : 0;
    for (int p0 = 0; p0 < np; p0 += 4) {   // four K steps at a time (zeros past M1)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int mp = 4 * (p0 + u) + kk;
        const bool ok = mp < m1;
        const int mc = ok ? mp : 0;
        const double bt = ok ? Ta[mc * 4 + x] : 0.0;
        const double at = ok && cv ? __builtin_nontemporal_load(Da + (size_t)mc * m2 + cc) : 0.0;
        acc[0] = mfma4(at, bt, acc[0]);
      }
    }
#pragma unroll
    for (int s = 0; s < S; ++s) A[a][s] = live && 16 * s + (lane >> 2) < m1 ? acc[s] : 0.0;
  }
}

// TI: storage of the table, R~ and dE/dT (float64, or float32 for the
// mixed mode: converted to float64 as they are read); TO: dE/dR~.  The
// products and the per-record polynomials are float64 in both.
// kFromD: dE/dT is not an input but formed in a prologue from the forward's
// T and dE/dD (float64, M' <= 16): the descriptor backward of D = T (T<)^T,
//   dE/dT[m][k] = sum_{n<M'} dE/dD[m][n] T[n][k] + (m < M') sum_m' dE/dD[m'][m] T[m'][k],
// evaluated per atom on the matrix cores straight into the A operands, so
// dE/dT never goes to memory.
template <typename TI, typename TO, int S, int NS, bool kOne, bool kFromD = false>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(3)))
void se_a_bwd_mfma_kernel(const Geo g, const TI* __restrict__ coeff,
                          const int* __restrict__ atype, const int* __restrict__ nlist,
                          const TI* __restrict__ em, const TI* __restrict__ dT,
                          TO* __restrict__ dR, const double* __restrict__ Tin = nullptr,
                          const double* __restrict__ dD = nullptr) {
  static_assert(S >= 1 && S <= 8, "K steps per channel block");
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NB = kMfmaAtoms;
  constexpr int kC = kLanes / NB;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const WaveAtoms<NB> wa = wave_atoms<NB, kOne>(g, atype, lane, wave);
  if (wa.idx[0] < 0) return;
  const int my_atom = lane_atom_of<NB>(wa, lane / kC);   // the atom of this lane's chunk-set slots
  const int nnei = g.nnei, m1 = g.m1, ld = g.ld;
  constexpr int kPairSlots = pair_slots(NS);
  const uint32_t zoff = __builtin_amdgcn_readfirstlane(wave * (uint32_t)bwdm_wave_bytes(NS));
  ChunkScratch& W = *reinterpret_cast<ChunkScratch*>(smem + zoff);
  const uint32_t store = lds_addr(smem) + zoff + (uint32_t)align16(sizeof(ChunkScratch));
  unsigned char* const slot_p =
      smem + zoff + align16(sizeof(ChunkScratch)) + (size_t)kPairSlots * kPairDoubles * sizeof(double);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(coeff, g.coeff_bytes);

  // this lane's place in the MFMA operands: K index kk, block h, column x
  const int kk = lane >> 4, h = (lane >> 2) & 3, x = lane & 3;
  // B column x of chain c is the power 2x + c, so that one 16-byte read of a
  // power pair gives a lane both chains' operands (x = 3 repeats the pair of
  // powers 4 and 5: those columns are not used)
  const uint32_t bread =
      lds_addr(slot_p) + (uint32_t)(min(x, 2) * ld + 4 * kk + h) * (uint32_t)(2 * sizeof(TI));
  auto channel = [&](int s) __attribute__((always_inline)) { return 16 * s + 4 * kk + h; };

  // A operands: dT of the wave's atoms, transposed, zero past M1
  double A[NB][S];
  int ai[NB];
  if constexpr (kFromD) descriptor_bwd_operands<NB, S>(g, wa, Tin, dD, lane, A);
#pragma unroll
  for (int a = 0; a < NB; ++a) {
    const int i = wa.idx[a];
    if constexpr (!kFromD) {
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const int m = channel(s);
        A[a][s] = (i >= 0 && m < m1)
                      ? (double)__builtin_nontemporal_load(dT + ((size_t)i * m1 + m) * 4 + x)
                      : 0.0;
      }
    }
    ai[a] = -1;
    if (i >= 0) {
      const int t = __builtin_amdgcn_readfirstlane(atype[i]);
      if (t < 0 || t >= g.ntypes) {  // invalid type: the atom's outputs become NaN
        for (int e = lane; e < nnei * 4; e += 64) dR[(size_t)i * nnei * 4 + e] = (TO)NAN;
      } else {
        ai[a] = t;
      }
    }
  }

  // copy the interval whose coefficients start at element `off` into the slot;
  // the interval's offset goes into the range-checked vector offset, so
  // that the bytes read past the last interval of the buffer come back as 0
  auto fetch = [&](int off) __attribute__((always_inline)) {
    const int voff = off * (int)sizeof(TI) + lane * 16;
#pragma unroll
    for (int i = 0; i < NS; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void*)(slot_p + 1024 * i), 16, voff + 1024 * i,
          0, 0, 0);
  };

  const int nch = (nnei + kC - 1) / kC;
  int s0 = ((int)(blockIdx.x * 5 + wave * 3) % nch) * kC;
  uint32_t vm = 0, occ = 0;
  TI pre[4];          // R~ rows of chunk set pre_s0, loaded ahead (valid slots use them)
  int pre_s0 = -1;
  for (int cc = 0, wbase = -1; cc < nch; ++cc, s0 = s0 + kC < nnei ? s0 + kC : 0) {
    if (s0 - s0 % (kWindow / NB) != wbase) {  // window of nlist signs holding s0
      wbase = s0 - s0 % (kWindow / NB);
      vm = valid_window<NB>(g, wa, wbase, nlist, lane);
      occ = occupied_chunks<NB>(vm);
    }
    if (!((occ >> ((s0 - wbase) / kC)) & 1)) {   // padding only: zero rows
      zero_rows<TO, NB>(g, ai, my_atom, s0, dR, lane);
      continue;
    }
    int pair;
    Rec<TI> mine;
    const Tables tb = build_chunk_set<TI, double, NB, true, kOne, true>(
        g, ai, my_atom, s0, wbase, vm, em, nullptr, W, lane, &pair, &mine, pre_s0 == s0, pre);
    // the rows of the next chunk set are loaded during this one's last run
    const int s0n = s0 + kC < nnei ? s0 + kC : 0;
    // (not when the window already shows that set to hold padding only)
    const bool more = cc + 1 < nch &&
                      (s0n - s0n % (kWindow / NB) != wbase || ((occ >> ((s0n - wbase) / kC)) & 1));
    double out[4] = {0.0, 0.0, 0.0, 0.0};   // this lane's dE/dR~ row
    if (tb.n > 0) {
      // the lanes whose records belong to pairs [base, base + np) read their products
      auto eval = [&](int base, int np) __attribute__((always_inline)) {
        if (pair >= base && pair < base + np) {
          const uint32_t pa = store + (uint32_t)((pair - base) * kPairDoubles * sizeof(double));
          const double t = mine.t;
          double val[4], der[4];
          v4i q[6];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            if (k % 2 == 0) lds_read_rows2(pa + 48 * k, q);   // rows k and k + 1
            const Pair<double> c01 = __builtin_bit_cast(Pair<double>, q[3 * (k % 2)]);
            const Pair<double> c23 = __builtin_bit_cast(Pair<double>, q[3 * (k % 2) + 1]);
            const Pair<double> c45 = __builtin_bit_cast(Pair<double>, q[3 * (k % 2) + 2]);
            double v = c45.y, d = c45.y;
            v = fma(v, t, c45.x);
            d = fma(d, t, v);
            v = fma(v, t, c23.y);
            d = fma(d, t, v);
            v = fma(v, t, c23.x);
            d = fma(d, t, v);
            v = fma(v, t, c01.y);
            d = fma(d, t, v);
            val[k] = fma(v, t, c01.x);
            der[k] = d;
          }
          // clamped records carry a zero row, which removes the derivative term
          double o0 = fma((double)mine.r[0], der[0], val[0]);
          o0 = fma((double)mine.r[1], der[1], o0);
          o0 = fma((double)mine.r[2], der[2], o0);
          out[0] = fma((double)mine.r[3], der[3], o0);
          out[1] = val[1];
          out[2] = val[2];
          out[3] = val[3];
        }
      };

      auto next_off = [&](int r) __attribute__((always_inline)) {
        return key_offset(readlane(tb.vk, min(r, kLanes - 1)));
      };
      fetch(next_off(0));
      int base = 0, np = 0;
      // run r: its coefficients are in the slot once the copy has landed;
      // after they are read, the slot takes the next run's (kLast: the
      // last run loads the next chunk set's rows instead)
      auto run = [&](int r, auto last) __attribute__((always_inline)) {
        constexpr bool kLast = decltype(last)::value;
        wait_copies();
        double Bc[2][S];
        if constexpr (sizeof(TI) == 8) {
          v4i q[S];
          lds_read_steps<S>(bread, q);
#pragma unroll
          for (int st = 0; st < S; ++st) {
            const Pair<double> v = __builtin_bit_cast(Pair<double>, q[st]);
            Bc[0][st] = v.x;
            Bc[1][st] = v.y;
          }
        } else {
          v2i q[S];
          lds_read_steps_b64<S>(bread, q);
#pragma unroll
          for (int st = 0; st < S; ++st) {
            const Pair<float> v = __builtin_bit_cast(Pair<float>, q[st]);
            Bc[0][st] = (double)v.x;
            Bc[1][st] = (double)v.y;
          }
        }
        if constexpr (!kLast) {
          fetch(next_off(r + 1));
        } else if (more) {
          const int ia = my_atom >= 0 ? my_atom : wa.idx[0], j = min(s0n + lane % kC, nnei - 1);
          load_row(em + ((size_t)ia * nnei + j) * 4, pre);
          pre_s0 = s0n;
        }
        const int Sr = readlane(tb.vs, r);
        const int Er = r + 1 < kLanes ? readlane(tb.vs, r + 1) : tb.n;
        int p[2] = {0, 0};
        p[0] = readlane(tb.vp[0], r);
        // one product per atom with records in the run, in atom order
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const int lo = b == 0 ? Sr : split_at<NB>(p, b);
          const int hi = b == NB - 1 ? Er : split_at<NB>(p, b + 1);
          if (lo < hi) {
            double d0 = 0.0, d1 = 0.0;
#pragma unroll
            for (int s = 0; s < S; ++s) {
              d0 = mfma4(A[b][s], Bc[0][s], d0);
              d1 = mfma4(A[b][s], Bc[1][s], d1);
            }
            // sum the four channel blocks into the lanes of block 3
            d0 += row_shr<4>(d0);
            d1 += row_shr<4>(d1);
            d0 += row_shr<8>(d0);
            d1 += row_shr<8>(d1);
            if (h == 3 && x < 3)   // P[k = kk][q = 2x + c] (row k: 6 doubles)
              lds_write16(store + (uint32_t)((np * kPairDoubles + 6 * kk + 2 * x) * sizeof(double)),
                          __builtin_bit_cast(v4i, Pair<double>{d0, d1}));
            ++np;
          }
        }
        if (kLast || np > kPairSlots - NB) {  // the next run may add NB products
          eval(base, np);
          base += np;
          np = 0;
        }
      };
      for (int r = 0; r + 1 < tb.nruns; ++r) run(r, std::false_type{});
      run(tb.nruns - 1, std::true_type{});
    }
    // each lane writes the dE/dR~ row of its own slot (zero for padding)
    if (tb.rank >= -1) {
      const TO o[4] = {(TO)out[0], (TO)out[1], (TO)out[2], (TO)out[3]};
      store_row(dR + ((size_t)my_atom * nnei + s0 + lane % kC) * 4, o);
    }
    wave_sync();
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
             size_t elem_bytes, Geo* g) {
#pragma clang fp contract(off)
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
  int64_t end = 0;
  for (int p = 0; p < ntypes * ntypes; ++p) {
    const dpc_range& r = ranges[p];
    if (!(std::isfinite(r.lo) && std::isfinite(r.d1) && std::isfinite(r.d2) && r.d1 > 0 &&
          r.d2 > 0 && r.L1 >= 1 && r.L2 >= 1 && r.offset >= 0))
      return DPC_ERANGE;
    const int64_t e = r.offset + (r.L1 + r.L2) * 6 * (int64_t)ld;
    // coefficient offsets must fit the key field; bytes must fit the buffer range
    if (e > kOffMask || e * (int64_t)elem_bytes >= (int64_t(1) << 31)) return DPC_ENOTSUP;
    end = e > end ? e : end;
    PairRange& q = g->pr[p];
    q.lo = r.lo;
    q.d1 = r.d1;
    q.d2 = r.d2;
    q.x_up = r.lo + (double)r.L1 * r.d1;
    q.x_end = q.x_up + (double)r.L2 * r.d2;
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
  g->coeff_bytes = (int)(end * (int64_t)elem_bytes);
  g->pair_out = 0;
  return DPC_OK;
}

// Channels per lane: 1 (m1 <= 64), 2 (m1 <= 128) or 4 (m1 <= 256).
int channels_per_lane(int m1) { return m1 <= 64 ? 1 : (m1 <= 128 ? 2 : 4); }

template <typename TI, typename TA>
int launch_fwd(hipStream_t s, const Geo& g, const void* coeff, const int* atype, const int* nlist,
               const void* em, void* T, void* D) {
  constexpr int NB = DPC_FWD_ATOMS_PER_WAVE;
  static_assert(NB == 1 || NB == 2 || NB == 4 || NB == 8, "atoms per wave: 1, 2, 4 or 8");
  const dim3 grid((g.nloc + kWaves * NB - 1) / (kWaves * NB)), block(64 * kWaves);
  const size_t shm = kWaves * fwd_wave_bytes<TI, TA>(g.m1);
  if (shm > kMaxLds) return DPC_ENOTSUP;
  (void)hipGetLastError();  // report only what this launch raises
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, block, shm, s, g, (const TI*)coeff, atype, nlist,
                       (const TI*)em, (TA*)T, (TA*)D);
  };
  switch (channels_per_lane(g.m1)) {
    case 1: g.ntypes == 1 ? go(se_a_fwd_kernel<TI, TA, 1, NB, true>) : go(se_a_fwd_kernel<TI, TA, 1, NB, false>); break;
    case 2: g.ntypes == 1 ? go(se_a_fwd_kernel<TI, TA, 2, NB, true>) : go(se_a_fwd_kernel<TI, TA, 2, NB, false>); break;
    default: g.ntypes == 1 ? go(se_a_fwd_kernel<TI, TA, 4, NB, true>) : go(se_a_fwd_kernel<TI, TA, 4, NB, false>); break;
  }
  return launch_status();
}

// M1 <= 128, float64 or mixed: the matrix-core kernel, ceil(M1 / 16) K steps
// per channel block, an interval copied by mfma_slot_kib(S, ld, esize) loads
// (ld lies in [16 S - 12, 16 S], so that count takes one of two values per S)
template <typename TI, typename TO, int S, bool kFromD>
void launch_mfma_s(hipStream_t s, const Geo& g, dim3 grid, dim3 block, const void* coeff,
                   const int* atype, const int* nlist, const void* em, const void* dT, void* dR,
                   const double* Tin, const double* dD) {
  constexpr int es = (int)sizeof(TI);
  const int ns = mfma_slot_kib(S, g.ld, es);
  auto go = [&](auto kern, size_t wave_bytes) {
    hipLaunchKernelGGL(kern, grid, block, kWaves * wave_bytes, s, g, (const TI*)coeff, atype,
                       nlist, (const TI*)em, (const TI*)dT, (TO*)dR, Tin, dD);
  };
  constexpr int lo = mfma_slot_kib(S, 16 * S - 12, es);
  static_assert(mfma_slot_kib(S, 16 * S, es) <= lo + 1, "two slot sizes per S");
  if (g.ntypes == 1) {
    if (ns <= lo) go(se_a_bwd_mfma_kernel<TI, TO, S, lo, true, kFromD>, bwdm_wave_bytes(lo));
    else go(se_a_bwd_mfma_kernel<TI, TO, S, lo + 1, true, kFromD>, bwdm_wave_bytes(lo + 1));
  } else {
    if (ns <= lo) go(se_a_bwd_mfma_kernel<TI, TO, S, lo, false, kFromD>, bwdm_wave_bytes(lo));
    else go(se_a_bwd_mfma_kernel<TI, TO, S, lo + 1, false, kFromD>, bwdm_wave_bytes(lo + 1));
  }
}

template <typename TI, typename TO, bool kFromD = false>
int launch_bwd_mfma(hipStream_t s, const Geo& g, const void* coeff, const int* atype,
                    const int* nlist, const void* em, const void* dT, void* dR,
                    const double* Tin = nullptr, const double* dD = nullptr) {
  const int S = (g.m1 + 15) / 16;
  constexpr int NB = kMfmaAtoms;
  const dim3 grid((g.nloc + kWaves * NB - 1) / (kWaves * NB)), block(64 * kWaves);
  (void)hipGetLastError();  // report only what this launch raises
  switch (S) {
#define DPC_CASE(n)                                                                                \
  case n:                                                                                          \
    launch_mfma_s<TI, TO, n, kFromD>(s, g, grid, block, coeff, atype, nlist, em, dT, dR, Tin, dD); \
    break;
    DPC_CASE(1) DPC_CASE(2) DPC_CASE(3) DPC_CASE(4) DPC_CASE(5) DPC_CASE(6) DPC_CASE(7)
#undef DPC_CASE
    default: launch_mfma_s<TI, TO, 8, kFromD>(s, g, grid, block, coeff, atype, nlist, em, dT, dR, Tin, dD); break;
  }
  return launch_status();
}

template <typename TI, typename TA>
int launch_bwd(hipStream_t s, const Geo& g, const void* coeff, const int* atype, const int* nlist,
               const void* em, const void* dT, void* dR) {
  // float64 and the mixed mode (float64 accumulation) on the matrix cores;
  // the float32 mode keeps float32 arithmetic on the vector ALUs
  if constexpr (sizeof(TA) == 8) {
    if (g.m1 <= 128) return launch_bwd_mfma<TI, TA>(s, g, coeff, atype, nlist, em, dT, dR);
  }
  constexpr int NB = DPC_BWD_ATOMS_PER_WAVE;
  static_assert(NB == 1 || NB == 2 || NB == 4 || NB == 8, "atoms per wave: 1, 2, 4 or 8");
  const dim3 grid((g.nloc + kWaves * NB - 1) / (kWaves * NB)), block(64 * kWaves);
  const int cpl = channels_per_lane(g.m1);
  const size_t shm = kWaves * bwd_wave_bytes<TI>();
  if (shm > kMaxLds) return DPC_ENOTSUP;
  (void)hipGetLastError();  // report only what this launch raises
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, block, shm, s, g, (const TI*)coeff, atype, nlist,
                       (const TI*)em, (const TI*)dT, (TA*)dR);
  };
  switch (cpl) {
    case 1: g.ntypes == 1 ? go(se_a_bwd_kernel<TI, TA, 1, NB, true>) : go(se_a_bwd_kernel<TI, TA, 1, NB, false>); break;
    case 2: g.ntypes == 1 ? go(se_a_bwd_kernel<TI, TA, 2, NB, true>) : go(se_a_bwd_kernel<TI, TA, 2, NB, false>); break;
    default: g.ntypes == 1 ? go(se_a_bwd_kernel<TI, TA, 4, NB, true>) : go(se_a_bwd_kernel<TI, TA, 4, NB, false>); break;
  }
  return launch_status();
}

}  // namespace

int dpc_internal_launch_status() { return launch_status(); }

extern "C" const char* dpc_last_hip_error(void) { return hipGetErrorString(g_last_hip); }

extern "C" int dpc_se_a_tab_fwd(void* stream, dpc_dtype dtype, int nloc, int ntypes,
                                const int* sel, int m1, int m2, const dpc_range* ranges,
                                const void* coeff, const int* atype, const int* nlist,
                                const void* em, void* T, void* D) {
  if (!dtype_ok(dtype)) return DPC_EINVAL;
  Geo g;
  const int st = make_geo(nloc, ntypes, sel, m1, m2, ranges, dtype == DPC_F64 ? 8 : 4, &g);
  if (st != DPC_OK) return st;
  if (nloc == 0) return DPC_OK;
  if (!coeff || !atype || !nlist || !em || !T || !D) return DPC_EINVAL;
  if (reinterpret_cast<uintptr_t>(em) % 16) return DPC_EINVAL;  // rows are read 16 bytes at a time
  g.pair_out = reinterpret_cast<uintptr_t>(T) % 16 == 0 && reinterpret_cast<uintptr_t>(D) % 16 == 0 &&
               (m1 * m2) % 2 == 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (dtype) {
    case DPC_F64: return launch_fwd<double, double>(s, g, coeff, atype, nlist, em, T, D);
    case DPC_F32: return launch_fwd<float, float>(s, g, coeff, atype, nlist, em, T, D);
    default: return launch_fwd<float, double>(s, g, coeff, atype, nlist, em, T, D);
  }
}

extern "C" int dpc_se_a_tab_bwd_from_dD(void* stream, dpc_dtype dtype, int nloc, int ntypes,
                                        const int* sel, int m1, int m2, const dpc_range* ranges,
                                        const void* coeff, const int* atype, const int* nlist,
                                        const void* em, const void* T, const void* dE_dD,
                                        void* dE_dem) {
  if (!dtype_ok(dtype)) return DPC_EINVAL;
  Geo g;
  const int st = make_geo(nloc, ntypes, sel, m1, m2, ranges, dtype == DPC_F64 ? 8 : 4, &g);
  if (st != DPC_OK) return st;
  // float64, the matrix-core backward (M1 <= 128), M' even and at most 16
  if (dtype != DPC_F64 || m1 > 128 || m2 > 16 || m2 % 2) return DPC_ENOTSUP;
  if (nloc == 0) return DPC_OK;
  if (!coeff || !atype || !nlist || !em || !T || !dE_dD || !dE_dem) return DPC_EINVAL;
  // rows of R~, dE/dR~, T and dE/dD are moved 16 bytes at a time
  if (reinterpret_cast<uintptr_t>(em) % 16 || reinterpret_cast<uintptr_t>(dE_dem) % 16 ||
      reinterpret_cast<uintptr_t>(T) % 16 || reinterpret_cast<uintptr_t>(dE_dD) % 16)
    return DPC_EINVAL;
  return launch_bwd_mfma<double, double, true>(static_cast<hipStream_t>(stream), g, coeff, atype,
                                               nlist, em, nullptr, dE_dem, (const double*)T,
                                               (const double*)dE_dD);
}

extern "C" int dpc_se_a_tab_bwd(void* stream, dpc_dtype dtype, int nloc, int ntypes,
                                const int* sel, int m1, const dpc_range* ranges,
                                const void* coeff, const int* atype, const int* nlist,
                                const void* em, const void* dE_dT, void* dE_dem) {
  if (!dtype_ok(dtype)) return DPC_EINVAL;
  Geo g;
  const int st = make_geo(nloc, ntypes, sel, m1, 1, ranges, dtype == DPC_F64 ? 8 : 4, &g);
  if (st != DPC_OK) return st;
  if (nloc == 0) return DPC_OK;
  if (!coeff || !atype || !nlist || !em || !dE_dT || !dE_dem) return DPC_EINVAL;
  // rows are read and written 16 bytes at a time
  if (reinterpret_cast<uintptr_t>(em) % 16 || reinterpret_cast<uintptr_t>(dE_dem) % 16)
    return DPC_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (dtype) {
    case DPC_F64: return launch_bwd<double, double>(s, g, coeff, atype, nlist, em, dE_dT, dE_dem);
    case DPC_F32: return launch_bwd<float, float>(s, g, coeff, atype, nlist, em, dE_dT, dE_dem);
    default: return launch_bwd<float, double>(s, g, coeff, atype, nlist, em, dE_dT, dE_dem);
  }
}
