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
// 4 channels).  A wavefront processes NB atoms together.  Each atom's
// neighbour list is compacted, 64 slots at a time, into LDS records
// {t, interval offset, slot}; the wave then merges the NB record streams by
// interval (largest offset first) with the record, the R~ row (scalar loads)
// and the interval uniform across the wave.  The coefficients of the current
// interval stay in registers until the interval changes, so every record of
// any of the NB atoms that falls into the same interval reuses them:
// neighbours are distance sorted, and atoms of the same kind see the same
// distances, so the load traffic per neighbour falls with NB.
//
// Forward: acc[a][k] += g_m(t) * R~[k] per channel, then T and D = T (T<)^T.
// Backward: for every record each lane forms its share of
//   dE/dR~[k] = sum_m dT[m][k] g_m + (k == 0) sum_m g'_m sum_k' dT[m][k'] R~[k']
// over its channels; the shares of a batch of 8 records are summed across
// lanes through LDS (each lane adds a strip of the transposed batch, then four
// strips are combined).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "dpc.h"

#ifndef DPC_FWD_ATOMS_PER_WAVE
#define DPC_FWD_ATOMS_PER_WAVE 4
#endif
#ifndef DPC_BWD_ATOMS_PER_WAVE
#define DPC_BWD_ATOMS_PER_WAVE 2
#endif

namespace {

constexpr int kWaves = 4;      // wavefronts per workgroup
constexpr int kChunk = 64;     // neighbour slots compacted at a time (per atom)
constexpr int kBatch = 8;      // records per cross-lane reduction in the backward pass

struct PairRange {             // one ordered type pair's table, as the kernels see it
  double lo, d1, d2;
  int L1, L2;
  int offset;                  // element offset of the pair's coefficients
  int pad;
};

struct Geo {
  int nloc, nnei, ntypes, m1, m2, ld;
  int coeff_bytes;             // size of the coefficient buffer (bounds the buffer loads)
  int blk_end[DPC_MAX_TYPES];  // slot index one past the end of each sel block
  PairRange pr[DPC_MAX_TYPES * DPC_MAX_TYPES];
};

struct Rec {                   // one valid neighbour, as staged in LDS
  double t;                    // offset from the left node of its interval
  int off;                     // element offset of the interval's coefficient rows
  int slot;                    // neighbour slot; bit 30 set = beyond the table (clamped)
};
constexpr int kClamped = 1 << 30;
constexpr int kSlotMask = kClamped - 1;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));

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

// Compact the valid slots [s0, s1) (at most 64) of one atom into records;
// returns their count.  Invalid slots get a zero row in `zero_out` if given.
template <typename TI, typename TA>
__device__ __forceinline__ int compact(const Geo& g, int ai, const int* nli, const TI* emi,
                                       int s0, int s1, Rec* rec, TA* zero_out, int lane) {
  const int j = s0 + lane;
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
  if (valid) rec[lanes_below(mask)] = r;
  return __popcll(mask);
}

// Record stream of one atom: its current chunk of records in LDS and the
// head record (uniform values).
template <typename TI>
struct Stream {
  int ai;      // atom type, or -1 when the atom is absent or finished
  int next;    // first slot not compacted yet
  int n, c;    // records in the chunk, cursor
  int head;    // coefficient offset of the head record, -1 when exhausted
  int slot;    // slot (and clamp bit) of the head record
  TI t;        // offset of the head record
};

template <typename TI>
__device__ __forceinline__ void read_head(Stream<TI>& s, const Rec* rec) {
  const Rec r = rec[s.c];
  s.head = __builtin_amdgcn_readfirstlane(r.off);
  s.slot = __builtin_amdgcn_readfirstlane(r.slot);
  s.t = (TI)r.t;
}

// Move to the next record, compacting further chunks as needed.
template <typename TI, typename TA>
__device__ __forceinline__ void advance(Stream<TI>& s, const Geo& g, const int* nli,
                                        const TI* emi, Rec* rec, TA* zero_out, int lane) {
  if (++s.c < s.n) {
    read_head(s, rec);
    return;
  }
  while (s.next < g.nnei) {
    wave_sync();
    const int n = compact<TI, TA>(g, s.ai, nli, emi, s.next, min(g.nnei, s.next + kChunk), rec,
                                  zero_out, lane);
    s.next += kChunk;
    if (n > 0) {
      wave_sync();
      s.n = n;
      s.c = 0;
      read_head(s, rec);
      return;
    }
  }
  s.head = -1;
}

template <typename TI>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coeff_rsrc(const TI* coeff, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)coeff, (short)0, bytes, 0x00020000);
}

// Coefficients of t^q (q = 0..5) of the lane's CPL channels in the interval
// whose rows start at element `off`.  voff = byte offset of the lane's first
// channel inside a row.
template <typename TI, int CPL>
__device__ __forceinline__ void load_coef(__amdgpu_buffer_rsrc_t rs, int off, int ld, int voff,
                                          TI (&cf)[6][CPL]) {
  constexpr int kBytes = CPL * (int)sizeof(TI);
  const int soff = off * (int)sizeof(TI);
#pragma unroll
  for (int q = 0; q < 6; ++q) {
    const int vo = voff + q * ld * (int)sizeof(TI);
    if constexpr (kBytes == 32) {
      const v4i a = __builtin_amdgcn_raw_buffer_load_b128(rs, vo, soff, 0);
      const v4i b = __builtin_amdgcn_raw_buffer_load_b128(rs, vo + 16, soff, 0);
      TI pa[CPL / 2], pb[CPL / 2];
      __builtin_memcpy(pa, &a, sizeof(pa));
      __builtin_memcpy(pb, &b, sizeof(pb));
#pragma unroll
      for (int h = 0; h < CPL / 2; ++h) {
        cf[q][h] = pa[h];
        cf[q][h + CPL / 2] = pb[h];
      }
    } else if constexpr (kBytes == 16) {
      const v4i a = __builtin_amdgcn_raw_buffer_load_b128(rs, vo, soff, 0);
      TI pa[CPL];
      __builtin_memcpy(pa, &a, sizeof(pa));
#pragma unroll
      for (int h = 0; h < CPL; ++h) cf[q][h] = pa[h];
    } else if constexpr (kBytes == 8) {
      const v2i a = __builtin_amdgcn_raw_buffer_load_b64(rs, vo, soff, 0);
      TI pa[CPL];
      __builtin_memcpy(pa, &a, sizeof(pa));
#pragma unroll
      for (int h = 0; h < CPL; ++h) cf[q][h] = pa[h];
    } else {
      const int a = __builtin_amdgcn_raw_buffer_load_b32(rs, vo, soff, 0);
      cf[q][0] = __builtin_bit_cast(TI, a);
    }
  }
}

// ---------------------------------------------------------------------------
// forward: T and D
// ---------------------------------------------------------------------------
template <typename TI, typename TA, int CPL, int NB>
__global__ __launch_bounds__(64 * kWaves) void se_a_fwd_kernel(
    const Geo g, const TI* __restrict__ coeff, const int* __restrict__ atype,
    const int* __restrict__ nlist, const TI* __restrict__ em, TA* __restrict__ T,
    TA* __restrict__ D) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i0 = __builtin_amdgcn_readfirstlane((blockIdx.x * kWaves + wave) * NB);
  if (i0 >= g.nloc) return;
  const int nnei = g.nnei, m1 = g.m1, m2 = g.m2, ld = g.ld;
  Rec* rec0 = reinterpret_cast<Rec*>(smem) + (size_t)wave * NB * kChunk;
  TA* sT = reinterpret_cast<TA*>(reinterpret_cast<Rec*>(smem) + kWaves * NB * kChunk) +
           (size_t)wave * m2 * 4;
  const __amdgpu_buffer_rsrc_t rs = coeff_rsrc(coeff, g.coeff_bytes);
  const int c0 = min(lane * CPL, ld - CPL);
  const int voff = c0 * (int)sizeof(TI);
  const bool owner = lane * CPL < m1;

  Stream<TI> st[NB];
  TA acc[NB][CPL][4];
#pragma unroll
  for (int a = 0; a < NB; ++a) {
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[a][h][k] = (TA)0;
    }
    const int i = i0 + a;
    st[a].ai = -1;
    st[a].head = -1;
    st[a].next = 0;
    st[a].n = st[a].c = 0;
    st[a].slot = 0;
    st[a].t = (TI)0;
    if (i < g.nloc) {
      const int ai = __builtin_amdgcn_readfirstlane(atype[i]);
      if (ai < 0 || ai >= g.ntypes) {  // invalid type: the atom's outputs become NaN
        const TA nan = (TA)NAN;
        for (int e = lane; e < m1 * 4; e += 64) T[(size_t)i * m1 * 4 + e] = nan;
        for (int e = lane; e < m1 * m2; e += 64) D[(size_t)i * m1 * m2 + e] = nan;
      } else {
        st[a].ai = ai;
        st[a].c = -1;
        advance<TI, TA>(st[a], g, nlist + (size_t)i * nnei, em + (size_t)i * nnei * 4,
                        rec0 + a * kChunk, nullptr, lane);
      }
    }
  }

  TI cf[6][CPL];
#pragma unroll
  for (int q = 0; q < 6; ++q) {
#pragma unroll
    for (int h = 0; h < CPL; ++h) cf[q][h] = (TI)0;
  }
  int cur = -1;
  for (;;) {
    int key = st[0].head;
#pragma unroll
    for (int a = 1; a < NB; ++a) key = max(key, st[a].head);
    if (key < 0) break;
    if (key != cur) {
      cur = key;
      if (owner) load_coef<TI, CPL>(rs, key, ld, voff, cf);
    }
#pragma unroll
    for (int a = 0; a < NB; ++a) {
      const TI* emi = em + (size_t)(i0 + a) * nnei * 4;
      while (st[a].head == key) {
        const TI* R = emi + (size_t)(st[a].slot & kSlotMask) * 4;
        const TI r0 = R[0], r1 = R[1], r2 = R[2], r3 = R[3];
        const TI t = st[a].t;
#pragma unroll
        for (int h = 0; h < CPL; ++h) {
          TI gv = cf[5][h];
          gv = fma(gv, t, cf[4][h]);
          gv = fma(gv, t, cf[3][h]);
          gv = fma(gv, t, cf[2][h]);
          gv = fma(gv, t, cf[1][h]);
          gv = fma(gv, t, cf[0][h]);
          const TA ga = (TA)gv;
          acc[a][h][0] = fma(ga, (TA)r0, acc[a][h][0]);
          acc[a][h][1] = fma(ga, (TA)r1, acc[a][h][1]);
          acc[a][h][2] = fma(ga, (TA)r2, acc[a][h][2]);
          acc[a][h][3] = fma(ga, (TA)r3, acc[a][h][3]);
        }
        advance<TI, TA>(st[a], g, nlist + (size_t)(i0 + a) * nnei, emi, rec0 + a * kChunk,
                        nullptr, lane);
      }
    }
  }

  // T rows and D = T (T<)^T of each atom
#pragma unroll
  for (int a = 0; a < NB; ++a) {
    const int i = i0 + a;
    if (i >= g.nloc || st[a].ai < 0) continue;
    wave_sync();
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int m = lane * CPL + h;
      if (m < m1) {
        TA* Tm = T + ((size_t)i * m1 + m) * 4;
#pragma unroll
        for (int k = 0; k < 4; ++k) Tm[k] = acc[a][h][k];
      }
      if (m < m2) {
#pragma unroll
        for (int k = 0; k < 4; ++k) sT[m * 4 + k] = acc[a][h][k];
      }
    }
    wave_sync();
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int m = lane * CPL + h;
      if (m < m1) {
        TA* Dm = D + ((size_t)i * m1 + m) * m2;
        for (int n = 0; n < m2; ++n) {
          TA s = acc[a][h][0] * sT[n * 4 + 0];
          s = fma(acc[a][h][1], sT[n * 4 + 1], s);
          s = fma(acc[a][h][2], sT[n * 4 + 2], s);
          s = fma(acc[a][h][3], sT[n * 4 + 3], s);
          Dm[n] = s;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// backward: dE/dR~
// ---------------------------------------------------------------------------
// LDS of one wave for the cross-lane sums: for each of the kBatch buffered
// records b and component pair kk, a block of nlq*4 lanes x 16 bytes holding
// (share[2kk], share[2kk+1]) of every lane (zero for lanes without channels);
// blocks are 64 bytes past a multiple of 256 apart so that 16 lanes reading
// 16 bytes each touch every bank once.
__host__ __device__ constexpr int red_block_bytes(int nlq) {
  return 64 * nlq + ((64 - (64 * nlq) % 256) % 256 + 256) % 256;
}

template <typename TA>
struct RedLds {
  unsigned char* red;   // 2 * kBatch blocks
  TA* part;             // [16 groups][4 lanes][2] partial sums
  int* row;             // [kBatch] (atom within the wave) << 21 | slot of each buffered record
};

// Sum the shares of nb buffered records and write dE/dR~ rows.  Lane L adds
// the strip x = L % 4 (lanes x, x+4, ...) of block (b, kk) = (L / 8, (L / 4) % 2);
// the four strips of a block are then combined by lane x = 0.
template <typename TA, int NLQ>
__device__ __forceinline__ void reduce_batch(const RedLds<TA>& r, int nlq, int blk, int nb,
                                             TA* dR, int i0, int nnei, int lane) {
  const int G = lane >> 2, x = lane & 3, b = G >> 1, kk = G & 1;
  wave_sync();
  const unsigned char* base = r.red + (size_t)(b * 2 + kk) * blk + x * 16;
  TA s0 = 0, s1 = 0;
#pragma unroll
  for (int q = 0; q < NLQ; ++q) {
    if (q < nlq) {
      const TA* v = reinterpret_cast<const TA*>(base + q * 64);
      s0 += v[0];
      s1 += v[1];
    }
  }
  r.part[(G * 4 + x) * 2 + 0] = s0;
  r.part[(G * 4 + x) * 2 + 1] = s1;
  wave_sync();
  if (x == 0 && b < nb) {
#pragma unroll
    for (int y = 1; y < 4; ++y) {
      s0 += r.part[(G * 4 + y) * 2 + 0];
      s1 += r.part[(G * 4 + y) * 2 + 1];
    }
    const int packed = r.row[b];
    TA* o = dR + ((size_t)(i0 + (packed >> 21)) * nnei + (packed & ((1 << 21) - 1))) * 4 + 2 * kk;
    o[0] = s0;
    o[1] = s1;
  }
  wave_sync();
}

template <typename TI, typename TA, int CPL, int NB>
__global__ __launch_bounds__(64 * kWaves) void se_a_bwd_kernel(
    const Geo g, const TI* __restrict__ coeff, const int* __restrict__ atype,
    const int* __restrict__ nlist, const TI* __restrict__ em, const TI* __restrict__ dT,
    TA* __restrict__ dR) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NLQ = (64 + 3) / 4;            // strips of at most 64 lanes
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i0 = __builtin_amdgcn_readfirstlane((blockIdx.x * kWaves + wave) * NB);
  if (i0 >= g.nloc) return;
  const int nnei = g.nnei, m1 = g.m1, ld = g.ld;
  const int nl = (m1 + CPL - 1) / CPL;          // lanes that own channels
  const int nlq = (nl + 3) / 4;
  const int blk = red_block_bytes(nlq);
  const size_t wave_bytes = (size_t)NB * kChunk * sizeof(Rec) + 2 * kBatch * blk +
                            16 * 4 * 2 * sizeof(TA) + kBatch * sizeof(int);
  unsigned char* wbase = smem + wave * wave_bytes;
  Rec* rec0 = reinterpret_cast<Rec*>(wbase);
  RedLds<TA> rl;
  rl.red = wbase + (size_t)NB * kChunk * sizeof(Rec);
  rl.part = reinterpret_cast<TA*>(rl.red + 2 * kBatch * blk);
  rl.row = reinterpret_cast<int*>(rl.part + 16 * 4 * 2);
  const __amdgpu_buffer_rsrc_t rs = coeff_rsrc(coeff, g.coeff_bytes);
  const int c0 = min(lane * CPL, ld - CPL);
  const int voff = c0 * (int)sizeof(TI);
  const bool owner = lane < nl;

  // lanes without channels contribute zeros: clear the whole sum area once
  for (int e = lane; e < 2 * kBatch * blk / 16; e += 64)
    reinterpret_cast<v4i*>(rl.red)[e] = (v4i){0, 0, 0, 0};

  Stream<TI> st[NB];
  TA dt[NB][CPL][4];
#pragma unroll
  for (int a = 0; a < NB; ++a) {
    const int i = i0 + a;
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int m = lane * CPL + h;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        dt[a][h][k] = (i < g.nloc && m < m1) ? (TA)dT[((size_t)i * m1 + m) * 4 + k] : (TA)0;
    }
    st[a].ai = -1;
    st[a].head = -1;
    st[a].next = 0;
    st[a].n = st[a].c = 0;
    st[a].slot = 0;
    st[a].t = (TI)0;
    if (i < g.nloc) {
      const int ai = __builtin_amdgcn_readfirstlane(atype[i]);
      if (ai < 0 || ai >= g.ntypes) {  // invalid type: the atom's outputs become NaN
        for (int e = lane; e < nnei * 4; e += 64) dR[(size_t)i * nnei * 4 + e] = (TA)NAN;
      } else {
        st[a].ai = ai;
        st[a].c = -1;
        advance<TI, TA>(st[a], g, nlist + (size_t)i * nnei, em + (size_t)i * nnei * 4,
                        rec0 + a * kChunk, dR + (size_t)i * nnei * 4, lane);
      }
    }
  }

  TI cf[6][CPL];
#pragma unroll
  for (int q = 0; q < 6; ++q) {
#pragma unroll
    for (int h = 0; h < CPL; ++h) cf[q][h] = (TI)0;
  }
  int cur = -1;
  int nb = 0;
  for (;;) {
    int key = st[0].head;
#pragma unroll
    for (int a = 1; a < NB; ++a) key = max(key, st[a].head);
    if (key < 0) break;
    if (key != cur) {
      cur = key;
      if (owner) load_coef<TI, CPL>(rs, key, ld, voff, cf);
    }
#pragma unroll
    for (int a = 0; a < NB; ++a) {
      const TI* emi = em + (size_t)(i0 + a) * nnei * 4;
      while (st[a].head == key) {
        const int slot = st[a].slot & kSlotMask;
        const TI* R = emi + (size_t)slot * 4;
        const TI r0 = R[0], r1 = R[1], r2 = R[2], r3 = R[3];
        const TI t = st[a].t;
        TA p0 = 0, p1 = 0, p2 = 0, p3 = 0;
        if ((st[a].slot & kClamped) == 0) {
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
            const TA gv = (TA)v, gd = (TA)d;
            TA w = dt[a][h][0] * (TA)r0;
            w = fma(dt[a][h][1], (TA)r1, w);
            w = fma(dt[a][h][2], (TA)r2, w);
            w = fma(dt[a][h][3], (TA)r3, w);
            p0 = fma(dt[a][h][0], gv, fma(gd, w, p0));
            p1 = fma(dt[a][h][1], gv, p1);
            p2 = fma(dt[a][h][2], gv, p2);
            p3 = fma(dt[a][h][3], gv, p3);
          }
        } else {  // beyond the table: constant value, zero derivative
#pragma unroll
          for (int h = 0; h < CPL; ++h) {
            TI v = cf[5][h];
            v = fma(v, t, cf[4][h]);
            v = fma(v, t, cf[3][h]);
            v = fma(v, t, cf[2][h]);
            v = fma(v, t, cf[1][h]);
            v = fma(v, t, cf[0][h]);
            const TA gv = (TA)v;
            p0 = fma(dt[a][h][0], gv, p0);
            p1 = fma(dt[a][h][1], gv, p1);
            p2 = fma(dt[a][h][2], gv, p2);
            p3 = fma(dt[a][h][3], gv, p3);
          }
        }
        if (owner) {
          TA* o0 = reinterpret_cast<TA*>(rl.red + (size_t)(nb * 2 + 0) * blk + lane * 16);
          TA* o1 = reinterpret_cast<TA*>(rl.red + (size_t)(nb * 2 + 1) * blk + lane * 16);
          o0[0] = p0;
          o0[1] = p1;
          o1[0] = p2;
          o1[1] = p3;
        }
        if (lane == 0) rl.row[nb] = (a << 21) | slot;
        if (++nb == kBatch) {
          reduce_batch<TA, NLQ>(rl, nlq, blk, nb, dR, i0, nnei, lane);
          nb = 0;
        }
        advance<TI, TA>(st[a], g, nlist + (size_t)(i0 + a) * nnei, emi, rec0 + a * kChunk,
                        dR + (size_t)(i0 + a) * nnei * 4, lane);
      }
    }
  }
  if (nb > 0) reduce_batch<TA, NLQ>(rl, nlq, blk, nb, dR, i0, nnei, lane);
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
    if (e * (int64_t)elem_bytes >= (int64_t(1) << 31)) return DPC_ENOTSUP;
    end = e > end ? e : end;
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
  g->coeff_bytes = (int)(end * (int64_t)elem_bytes);
  return DPC_OK;
}

// Channels per lane: 1 (m1 <= 64), 2 (m1 <= 128) or 4 (m1 <= 256).
int channels_per_lane(int m1) { return m1 <= 64 ? 1 : (m1 <= 128 ? 2 : 4); }

template <typename TI, typename TA>
int launch_fwd(hipStream_t s, const Geo& g, const void* coeff, const int* atype, const int* nlist,
               const void* em, void* T, void* D) {
  constexpr int NB = DPC_FWD_ATOMS_PER_WAVE;
  const dim3 grid((g.nloc + kWaves * NB - 1) / (kWaves * NB)), block(64 * kWaves);
  const size_t shm =
      (size_t)kWaves * NB * kChunk * sizeof(Rec) + (size_t)kWaves * g.m2 * 4 * sizeof(TA);
  (void)hipGetLastError();  // report only what this launch raises
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, block, shm, s, g, (const TI*)coeff, atype, nlist,
                       (const TI*)em, (TA*)T, (TA*)D);
  };
  switch (channels_per_lane(g.m1)) {
    case 1: go(se_a_fwd_kernel<TI, TA, 1, NB>); break;
    case 2: go(se_a_fwd_kernel<TI, TA, 2, NB>); break;
    default: go(se_a_fwd_kernel<TI, TA, 4, NB>); break;
  }
  return launch_status();
}

template <typename TI, typename TA>
int launch_bwd(hipStream_t s, const Geo& g, const void* coeff, const int* atype, const int* nlist,
               const void* em, const void* dT, void* dR) {
  constexpr int NB = DPC_BWD_ATOMS_PER_WAVE;
  const dim3 grid((g.nloc + kWaves * NB - 1) / (kWaves * NB)), block(64 * kWaves);
  const int cpl = channels_per_lane(g.m1);
  const int nl = (g.m1 + cpl - 1) / cpl;
  const int blk = red_block_bytes((nl + 3) / 4);
  const size_t wave_bytes = (size_t)NB * kChunk * sizeof(Rec) + 2 * kBatch * blk +
                            16 * 4 * 2 * sizeof(TA) + kBatch * sizeof(int);
  const size_t shm = kWaves * wave_bytes;
  (void)hipGetLastError();  // report only what this launch raises
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, block, shm, s, g, (const TI*)coeff, atype, nlist,
                       (const TI*)em, (const TI*)dT, (TA*)dR);
  };
  switch (cpl) {
    case 1: go(se_a_bwd_kernel<TI, TA, 1, NB>); break;
    case 2: go(se_a_bwd_kernel<TI, TA, 2, NB>); break;
    default: go(se_a_bwd_kernel<TI, TA, 4, NB>); break;
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
  const int st = make_geo(nloc, ntypes, sel, m1, m2, ranges, dtype == DPC_F64 ? 8 : 4, &g);
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
  const int st = make_geo(nloc, ntypes, sel, m1, 1, ranges, dtype == DPC_F64 ? 8 : 4, &g);
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
