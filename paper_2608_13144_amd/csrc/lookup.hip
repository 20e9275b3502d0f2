// Batched certified lookup (Sec. 4.4, Eq. (13)-(15); Alg. 2).
//
// For query q and entry i the hit test is ||q - z_i|| < r_i, i.e.
//   ||q||^2 + ||z_i||^2 - 2 q.z_i < r_i^2.
// The dot products q.z_i of all B x n pairs are the dense part of the work
// (the N d term of Eq. (16)); they run on the matrix cores and are never
// stored.  Near the ball boundary the expanded form cancels badly (||z||^2 is
// ~1e3 while d^2 is ~1e-2 at the large workloads), so the matrix-core value
// is only a FILTER:
//   pass  <=>  fl(g_hat - Q_q) >= A_i,
//   Q_q = RD((1 - k) ||q||^2 / 2 - eta1 ||q|| - eta0),
//   A_i = RD(((1 - k - 4u) ||z_i||^2 - r_i^2) / 2 - eta1 ||z_i||),
// where k bounds |g_hat - q.z_i| / ((||q||^2 + ||z_i||^2) / 2) and eta1, eta0
// its absolute part (float16 or float32 operand rounding, sub-normals and
// float32 accumulation, doubled; filter_slack); for d <= 128 the float16
// filter accumulates onto -Q_q instead (acc >= A_i), which adds one more
// float32 rounding against Q_q, far inside that bound.  Every true hit
// passes.  A pair that passes is queued and re-checked after the scan as
// sum_k (q_k - z_ik)^2 in float64 from the original values, which decides the
// hit.  Hits are merged per query with a 64-bit atomic minimum of (float bits
// of d^2) << 32 | i, which orders by distance and then by index, independent
// of scheduling.
//
// Kernel layout (gfx950, wave64):
//  - workgroup = 8 waves (two per SIMD); wave w holds RT*16 queries as MFMA
//    A operands in registers for the whole sweep (float16 or float32,
//    converted once);
//  - the workgroup streams its slice of the cache through LDS in tiles of
//    128 entries (64 KiB, double-buffered), copied global -> LDS without
//    registers (lookup_dma_kernel), or, when the rows need a conversion,
//    register-staged tiles of 64 (lookup_kernel);
//  - per 16-entry column tile: KS k-steps of v_mfma_f32_16x16x32_f16 (or 4x
//    v_mfma_f32_16x16x4_f32), then the filter on the accumulators; a wave
//    ballot skips the queueing path unless a pair passed;
//  - grid = query blocks x cache slices; blocks are numbered so that the
//    blocks a given XCD runs (block id mod 8) share cache slices, so the
//    resident workgroups of an XCD read each cache tile from its L2 at about
//    the same time.  The indexed lookup instead gives each block (4 waves,
//    64-row tiles, two blocks per CU) one item of a work list: up to 256
//    queries of one cluster's query list (read through the list, in a
//    separate instantiation) against a chunk of that cluster's rows.  There a query meets its own cluster's rows, so pairs pass the
//    filter often: each wave queues them in LDS, hands the queue to the
//    global queue after its last tile in one reservation; waves past the
//    list end only copy;
//  - recheck_queue_kernel settles the global queue chip-wide; a pair that
//    finds the queue full is re-checked by its wave at once (same order of
//    sums, so the same d^2 either way).
#include <limits.h>

#include <mutex>

#include "lc_common.hpp"
#include "lc_index.hpp"

namespace lc {

constexpr int kLkThreads = 512;
constexpr int kLkWaves = kLkThreads / kWave;
constexpr int kTileN = 64;
constexpr int kColTile = 16;
constexpr int kXcds = 8;
constexpr unsigned long long kNoHit = ~0ull;

enum { kModeF16 = 0, kModeF32 = 1 };
// For d <= 128 the float16 filter starts each accumulator at -Q_q instead of
// zero, so the matrix core returns g - Q_q and the filter is one max per
// accumulator (there the filter's vector work, not the matrix core, is what
// limits); the extra fp32 rounding is far inside the float16 slack.  Wider
// rows keep the subtraction: the extra live registers would spill there.
// The fp32 filter, whose slack is tight, always subtracts Q_q after the
// contraction.
template <int MODE, int KS>
constexpr bool kFoldQ = MODE == kModeF16 && KS <= 4;

struct LookupParams {
  const float* zq;
  int64_t B;
  const void* cz;
  const float* cr;
  const float* cnorm2;
  int64_t n;
  int d;
  const float* qthr;
  unsigned long long* best;
  unsigned int* bflag;
  unsigned long long* stats;
  double kappa_c;        // 1 - k - 4u, applied to ||z_i||^2
  double eta1;           // absolute slack per unit of ||z_i||
  double range2;         // ||z_i||^2 from which an entry passes against everything
  const float* athr;     // [n_pad] per-entry filter thresholds A_i (+inf past n)
  // Prefix pruning: thresholds of the filter over features 0..31 (Q'_q per
  // query, A'_i per entry, +inf past n); null without the option.
  const float* qthr_p;
  const float* athr_p;
  const void* cimg;      // rows streamed by the DMA kernel (float16 image or z)
  int n_qblocks;
  int64_t slice_len;
  float* g_hat;          // dump mode only
  uint8_t* cand;         // dump mode only
  // Work-list mode (indexed lookup): block b takes the query positions
  // [items[4b], items[4b+1]) against cache rows [items[4b+2], items[4b+3])
  // instead of a slice; position j means query qlist[j] (j itself when
  // qlist is null).
  const int64_t* items;
  const int32_t* qlist;
  // float16 copy of the queries (the in-kernel conversion): the A operands
  // of the work-list kernel, half the bytes of the float32 rows every item
  // would otherwise gather.
  const uint16_t* zq16;
  // Index written into a hit's key: (emap ? emap[e] : e) + eoff.
  const int64_t* emap;
  int64_t eoff;
  // Global re-check queue (query position, cache row): pairs that pass the
  // filter are appended here and settled chip-wide after the scan (work-list
  // mode: each wave's LDS queue moves here in one reservation).  gq_count
  // counts reserved slots; a pair that finds no slot below gq_cap is
  // re-checked by its wave at once, and a slot a wave reserved but settled
  // itself holds position -1.  Null (filter dump): nothing is re-checked.
  int64_t* gq_pos;
  int64_t* gq_e;
  unsigned long long* gq_count;
  int64_t gq_cap;
};

// ------------------------------------------------------------- prep
// Filter thresholds.  A pair passes iff fl(g_hat - Q_q) >= A_i with
//   Q_q = RD((1 - k) ||q||^2 / 2 - eta1 ||q|| - eta0),
//   A_i = RD(((1 - k - 4u) ||z_i||^2 - r_i^2) / 2 - eta1 ||z_i|| - abs / 2)
// (k, eta1, eta0 from filter_slack).  A row whose squared norm reaches
// range2 (the float16 operands may not hold it) gets kPassAll: it passes
// against every live entry or query and the exact re-check decides.  A NaN
// norm gives a NaN threshold (never passes: NaN features have no hit), an
// infinite query norm likewise (its distance to every entry is infinite).
struct Thresholds {
  double kq;       // 1 - k
  double kappa_c;  // 1 - k - 4u
  double eta1;
  double eta0;
  double range2;
};

__device__ __forceinline__ float query_threshold(double s, const Thresholds& t) {
  if (s >= t.range2 && s < __builtin_inf()) return kPassAll;
  return f32_round_down(t.kq * s * 0.5 - t.eta1 * __builtin_sqrt(s) - t.eta0);
}

// +inf for rows that can never be hit (r_i <= 0 or NaN).
__device__ __forceinline__ float entry_threshold(float rr, float n2f, double kappa_c, double eta1, double range2) {
  if (!(rr > 0.0f)) return __builtin_inff();
  const double n2 = static_cast<double>(n2f);
  if (n2 >= range2 && n2 < __builtin_inf()) return kPassAll;
  const double r2 = static_cast<double>(rr) * static_cast<double>(rr);
  return f32_round_down((kappa_c * n2 - r2) * 0.5 - eta1 * __builtin_sqrt(n2) - 0.5 * kFilterAbsSlack);
}

// Prefix filter (features 0..kPrefixDims-1, the first float16 k-step).  The
// prefix of a squared distance is a lower bound of the whole, so a pair with
// ||q - z_i|| < r_i (a hit) or within the boundary band has a prefix below
// r_i^2 (1 + 1e-5)^2 < r_i^2 (1 + 3e-5); the thresholds are those of the
// full filter with d_pad = kPrefixDims, the prefix norms, and that widened
// ball, so such a pair always passes.  A row whose full squared norm
// reaches range2 passes (as in the full filter); a NaN or infinite query
// norm never does (it has no hit).
constexpr int kPrefixDims = 32;
constexpr double kPrefixBand = 3e-5;

__device__ __forceinline__ float prefix_query_threshold(double s, double sp, const Thresholds& t) {
  if (!(s < __builtin_inf())) return __builtin_nanf("");
  if (s >= t.range2) return kPassAll;
  return f32_round_down(t.kq * sp * 0.5 - t.eta1 * __builtin_sqrt(sp) - t.eta0);
}

__device__ __forceinline__ float prefix_entry_threshold(float rr, float n2f, double n2p, const Thresholds& t) {
  if (!(rr > 0.0f)) return __builtin_inff();
  const double n2 = static_cast<double>(n2f);
  if (n2 >= t.range2 && n2 < __builtin_inf()) return kPassAll;
  const double r2 = static_cast<double>(rr) * static_cast<double>(rr) * (1.0 + kPrefixBand);
  return f32_round_down((t.kappa_c * n2p - r2) * 0.5 - t.eta1 * __builtin_sqrt(n2p) - 0.5 * kFilterAbsSlack);
}

// Squared norm of the first kPrefixDims stored features of row i, in float64.
__device__ __forceinline__ double prefix_norm2(const void* cz, int store, int d, int64_t i) {
  double s = 0.0;
  if (store == LIPCACHE_BF16) {
    const uint4* row = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(cz) + i * d);
#pragma unroll
    for (int c = 0; c < kPrefixDims / 8; ++c) {
      const uint4 v = row[c];
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const double lo = static_cast<double>(__builtin_bit_cast(float, w[j] << 16));
        const double hi = static_cast<double>(__builtin_bit_cast(float, w[j] & 0xffff0000u));
        s = __builtin_fma(lo, lo, s);
        s = __builtin_fma(hi, hi, s);
      }
    }
  } else {
    const float4* row = reinterpret_cast<const float4*>(static_cast<const float*>(cz) + i * d);
#pragma unroll
    for (int c = 0; c < kPrefixDims / 4; ++c) {
      const float4 v = row[c];
      s = __builtin_fma(static_cast<double>(v.x), static_cast<double>(v.x), s);
      s = __builtin_fma(static_cast<double>(v.y), static_cast<double>(v.y), s);
      s = __builtin_fma(static_cast<double>(v.z), static_cast<double>(v.z), s);
      s = __builtin_fma(static_cast<double>(v.w), static_cast<double>(v.w), s);
    }
  }
  return s;
}

// Per-entry threshold of row i < n_pad (+inf for the padding past n).
__device__ __forceinline__ void write_athr(int64_t i, const float* __restrict__ cr, const float* __restrict__ cnorm2,
                                           int64_t n, int64_t n_pad, double kappa_c, double eta1, double range2,
                                           float* __restrict__ athr) {
  if (i >= n_pad) return;
  athr[i] = i < n ? entry_threshold(cr[i], cnorm2[i], kappa_c, eta1, range2) : __builtin_inff();
}

// The entries a prep launch also covers (athr == nullptr: none).
struct PrepEntries {
  const float* cr;
  const float* cnorm2;
  int64_t n;
  int64_t n_pad;
  float* athr;
  unsigned long long* gq_count;  // emptied for the scan that follows (nullable)
  double* qnorm;                 // ||q||^2 in float64 of every query (nullable)
  uint16_t* zq16;                // float16 copy of the queries (nullable)
  // prefix pruning (qthr_p == nullptr: off): Q'_q, A'_i [np_pad] and their
  // constants
  float* qthr_p;
  float* athr_p;
  int64_t np_pad;
  const void* cz;
  int store;
  Thresholds tp;
};

// Blocks [0, qblocks): one wave per query, Q_q, reset of the per-query state
// and (block 0) of the counters.  Blocks past qblocks: the per-entry
// thresholds A_i, 512 rows per block.  One launch for both.
__global__ void lookup_prep_kernel(const float* __restrict__ zq, int64_t B, int d, const Thresholds t,
                                   float* __restrict__ qthr, unsigned long long* __restrict__ best,
                                   unsigned int* __restrict__ bflag, unsigned long long* __restrict__ stats,
                                   unsigned qblocks, const PrepEntries pe) {
  if (blockIdx.x >= qblocks) {
    const int64_t i = static_cast<int64_t>(blockIdx.x - qblocks) * kLkThreads + threadIdx.x;
    write_athr(i, pe.cr, pe.cnorm2, pe.n, pe.n_pad, t.kappa_c, t.eta1, t.range2, pe.athr);
    if (pe.athr_p && i < pe.np_pad)
      pe.athr_p[i] = i < pe.n ? prefix_entry_threshold(pe.cr[i], pe.cnorm2[i], prefix_norm2(pe.cz, pe.store, d, i), pe.tp)
                              : __builtin_inff();
    return;
  }
  const int64_t q = static_cast<int64_t>(blockIdx.x) * kLkWaves + threadIdx.x / kWave;
  if (blockIdx.x == 0 && threadIdx.x < 4) stats[threadIdx.x] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 4 && pe.gq_count) *pe.gq_count = 0ull;
  if (q >= B) return;
  const float* row = zq + q * d;
  double s = 0.0, sp = 0.0;
  for (int k = lane_id(); k < d; k += kWave) {
    const float x = row[k];
    s = __builtin_fma(static_cast<double>(x), static_cast<double>(x), s);
    if (k < kPrefixDims) sp = s;
    if (pe.zq16) pe.zq16[q * d + k] = f16_bits(x);
  }
  s = wave_sum(s);
  if (pe.qthr_p) sp = wave_sum(sp);
  if (lane_id() == 0) {
    qthr[q] = query_threshold(s, t);
    best[q] = kNoHit;
    bflag[q] = 0u;
    if (pe.qnorm) pe.qnorm[q] = s;
    if (pe.qthr_p) pe.qthr_p[q] = prefix_query_threshold(s, sp, pe.tp);
  }
}

// Per-entry thresholds A_i, +inf for the padding past n; thread 0 also
// empties the global re-check queue of the scan that follows.
__global__ void lookup_athr_kernel(const float* __restrict__ cr, const float* __restrict__ cnorm2, int64_t n,
                                   int64_t n_pad, double kappa_c, double eta1, double range2,
                                   float* __restrict__ athr, unsigned long long* __restrict__ gq_count) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i == 0 && gq_count) *gq_count = 0ull;
  write_athr(i, cr, cnorm2, n, n_pad, kappa_c, eta1, range2, athr);
}

// ------------------------------------------------------------- finalize
__global__ void lookup_finalize_kernel(int64_t B, const unsigned long long* __restrict__ best,
                                       const unsigned int* __restrict__ bflag,
                                       const int32_t* __restrict__ clabel, int32_t* __restrict__ label_out,
                                       int64_t* __restrict__ index_out, float* __restrict__ dist2_out,
                                       uint8_t* __restrict__ band_out, unsigned long long* __restrict__ stats) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  bool hit = false, band = false;
  if (q < B) {
    const unsigned long long key = best[q];
    hit = key != kNoHit;
    band = bflag[q] != 0u;
    const int64_t i = hit ? static_cast<int64_t>(key & 0xffffffffull) : -1;
    label_out[q] = hit ? clabel[i] : LIPCACHE_MISS;
    if (index_out) index_out[q] = i;
    if (dist2_out) dist2_out[q] = hit ? __builtin_bit_cast(float, static_cast<uint32_t>(key >> 32)) : __builtin_inff();
    if (band_out) band_out[q] = band ? 1 : 0;
  }
  const unsigned long long nh = __builtin_popcountll(__ballot(hit));
  const unsigned long long nb = __builtin_popcountll(__ballot(band));
  if (lane_id() == 0) {
    if (nh) atomicAdd(&stats[LIPCACHE_STAT_HITS], nh);
    if (nb) atomicAdd(&stats[LIPCACHE_STAT_BAND_QUERIES], nb);
  }
}

// ------------------------------------------------------------- main kernel
// Block -> (query positions [q0, qend), cache rows).  Slice mode: consecutive
// blocks of one XCD (same id mod 8) take consecutive query blocks of one
// slice, so they read each tile from that XCD's L2 at about the same time.
// Work-list mode: the block's item.
__device__ __forceinline__ void block_work(const LookupParams& p, int64_t qblock, int64_t& q0, int64_t& qend,
                                           int64_t& e_begin, int64_t& e_end) {
  const int bid = static_cast<int>(blockIdx.x);
  if (p.items) {
    const int64_t* it = p.items + 4 * static_cast<int64_t>(bid);
    q0 = it[0];
    qend = it[1];
    e_begin = it[2];
    e_end = it[3] < p.n ? it[3] : p.n;
    return;
  }
  const int xcd = bid % kXcds;
  const int local = bid / kXcds;
  const int slice = xcd + kXcds * (local / p.n_qblocks);
  q0 = static_cast<int64_t>(local % p.n_qblocks) * qblock;
  qend = p.B;
  e_begin = static_cast<int64_t>(slice) * p.slice_len;
  e_end = e_begin + p.slice_len < p.n ? e_begin + p.slice_len : p.n;
}

// The query at position j of the block's range.
__device__ __forceinline__ int64_t query_at(const int32_t* qlist, int64_t j) { return qlist ? qlist[j] : j; }

template <int MODE>
struct ModeTraits;
template <>
struct ModeTraits<kModeF16> {
  static constexpr int kElemBytes = 2;
  static constexpr int kPerChunk = 8;                 // elements per 16-byte chunk
  static constexpr int kPerStep = 4 * kPerChunk;      // k per k-step (32)
};
template <>
struct ModeTraits<kModeF32> {
  static constexpr int kElemBytes = 4;
  static constexpr int kPerChunk = 4;
  static constexpr int kPerStep = 4 * kPerChunk;      // 16
};

// One k-step of the contraction for a 16x16 output tile.
template <int MODE>
__device__ __forceinline__ f32x4 mfma_step(u32x4 a, u32x4 b, f32x4 acc) {
  if constexpr (MODE == kModeF16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), acc,
                                                  0, 0, 0);
  } else {
    // Reinterpret the whole 16-byte chunk (a per-element bit cast of a vector
    // subscript is miscompiled to element 0 by this toolchain).
    const f32x4 af = __builtin_bit_cast(f32x4, a);
    const f32x4 bf = __builtin_bit_cast(f32x4, b);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[0], bf[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[1], bf[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[2], bf[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[3], bf[3], acc, 0, 0, 0);
    return acc;
  }
}

// Load PER consecutive elements [k0, k0 + PER) of a row as one 16-byte MFMA
// operand chunk of the mode's element type; zeros beyond d.  SRC is the
// element type in memory (LIPCACHE_F32, LIPCACHE_BF16, or LIPCACHE_F16 for
// rows already converted).
template <int MODE, int SRC>
__device__ __forceinline__ u32x4 load_chunk(const void* base, int64_t row, int d, int k0) {
  u32x4 v = {0u, 0u, 0u, 0u};
  if (k0 >= d) return v;
  if constexpr (MODE == kModeF16) {
    if constexpr (SRC == LIPCACHE_F32) {
      const f32x4* p = reinterpret_cast<const f32x4*>(static_cast<const float*>(base) + row * d + k0);
      const f32x4 x0 = p[0], x1 = p[1];
      const float f[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
      v = pack_f16x8(f);
    } else if constexpr (SRC == LIPCACHE_BF16) {
      const u32x4 h = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(base) + row * d + k0);
      float f[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f[2 * i] = __builtin_bit_cast(float, h[i] << 16);
        f[2 * i + 1] = __builtin_bit_cast(float, h[i] & 0xffff0000u);
      }
      v = pack_f16x8(f);
    } else {
      v = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(base) + row * d + k0);
    }
  } else {
    if constexpr (SRC == LIPCACHE_F32) {
      v = *reinterpret_cast<const u32x4*>(static_cast<const float*>(base) + row * d + k0);
    } else {
      const uint16_t* p = static_cast<const uint16_t*>(base) + row * d + k0;
      const uint2 h = *reinterpret_cast<const uint2*>(p);
      v[0] = h.x << 16;
      v[1] = h.x & 0xffff0000u;
      v[2] = h.y << 16;
      v[3] = h.y & 0xffff0000u;
    }
  }
  return v;
}

template <int SRC>
__device__ __forceinline__ double cache_value(const void* cz, int64_t row, int d, int k) {
  if constexpr (SRC == LIPCACHE_F32) {
    return static_cast<double>(static_cast<const float*>(cz)[row * d + k]);
  } else {
    return static_cast<double>(bf16_to_f32(static_cast<const uint16_t*>(cz)[row * d + k]));
  }
}

// Everything the exact re-check touches, passed by value so that calling it
// does not force the kernel arguments into scratch memory.
struct RecheckArgs {
  const float* zq;
  const void* cz;
  const float* cr;
  unsigned long long* best;
  unsigned int* bflag;
  unsigned long long* stats;
  int64_t qend;          // query positions at or past qend are padding
  int64_t n;
  int d;
  const int64_t* emap;
  int64_t eoff;
  const int32_t* qlist;
};

__device__ __forceinline__ RecheckArgs recheck_args(const LookupParams& p, int64_t qend, const int32_t* qlist) {
  return RecheckArgs{p.zq, p.cz, p.cr, p.best, p.bflag, p.stats, qend, p.n, p.d, p.emap, p.eoff, qlist};
}

// ||q - z_e||^2 of query row q and cache row e in float64 over the whole
// wave: lane-strided partial sums, then a fixed butterfly, so the value does
// not depend on scheduling or on which path evaluates the pair.
template <int SRC>
__device__ __forceinline__ double wave_dist2(const RecheckArgs& p, int64_t q, int64_t e) {
  const float* qr = p.zq + q * p.d;
  double part = 0.0;
  for (int k = lane_id(); k < p.d; k += kWave) {
    const double diff = static_cast<double>(qr[k]) - cache_value<SRC>(p.cz, e, p.d, k);
    part = __builtin_fma(diff, diff, part);
  }
  return wave_sum(part);
}

// Outcome of one re-checked pair (one lane): counters, band flag, and the
// packed (d^2, entry) key of a hit into the query's minimum.
__device__ __forceinline__ void record_pair(const RecheckArgs& p, int64_t q, int64_t e, double d2) {
  atomicAdd(&p.stats[LIPCACHE_STAT_RECHECKED], 1ull);
  const double r = static_cast<double>(p.cr[e]);
  const bool hit = d2 < r * r;
  if (__builtin_fabs(__builtin_sqrt(d2) - r) <= 1e-5 * r) {
    atomicAdd(&p.stats[LIPCACHE_STAT_BAND_PAIRS], 1ull);
    atomicOr(&p.bflag[q], 1u);
  }
  if (hit) {
    const float d2f = static_cast<float>(d2);
    const int64_t ek = (p.emap ? p.emap[e] : e) + p.eoff;
    const unsigned long long key = (static_cast<unsigned long long>(__builtin_bit_cast(uint32_t, d2f)) << 32) |
                                   static_cast<unsigned long long>(static_cast<uint32_t>(ek));
    atomicMin(&p.best[q], key);
  }
}

// Exact re-check of the pairs whose bits are set in `mask` (bit rt*4+i of a
// lane = accumulator i of row tile rt), one pair at a time by the whole wave.
template <int SRC>
__device__ __noinline__ void recheck_pairs(const RecheckArgs p, uint32_t mask, int64_t qwave, int64_t ebase) {
  const int lane = lane_id();
  while (true) {
    const unsigned long long bal = __ballot(mask != 0u);
    if (bal == 0ull) break;
    const int src = __builtin_ctzll(bal);
    const uint32_t msrc = static_cast<uint32_t>(__shfl(static_cast<int>(mask), src, kWave));
    const int bit = __builtin_ctz(msrc);
    if (lane == src) mask &= mask - 1u;
    const int rt = bit >> 2, i = bit & 3;
    const int64_t qpos = qwave + rt * 16 + 4 * (src >> 4) + i;
    const int64_t e = ebase + (src & 15);
    if (qpos >= p.qend || e >= p.n) continue;  // padded rows never pass; kept as a guard
    const int64_t q = query_at(p.qlist, qpos);
    const double d2 = wave_dist2<SRC>(p, q, e);
    if (lane == 0) record_pair(p, q, e, d2);
  }
}

// Work-list mode defers the re-check: a wave queues its passing pairs in
// LDS while it scans the item's tiles and settles them after its last tile
// (or when the queue is full), so a pair costs no barrier-coupled stall of
// the whole workgroup.
constexpr int kRq = 64;  // queued pairs per wave

struct RecheckQueue {
  int32_t* q;  // LDS: kRq query positions, relative to the wave's first
  int64_t* e;  // LDS: kRq cache rows
  int n;       // queued pairs (wave-uniform)
};

// Re-check of up to four pairs per pass: lane j < 4 brings pair j (valid,
// list position, cache row), fetches its query id, radius and key first,
// then every lane loads its features of all four rows before the sums (each
// pair keeps the lane-strided order of wave_dist2, so results equal the
// immediate path's bit for bit).  All 64 lanes call it; it returns the
// number of pairs re-checked (the caller adds it to the counter once, since
// thousands of waves settling at the same time would serialise on it).
template <int SRC>
__device__ __forceinline__ int settle_four(const RecheckArgs& p, bool valid, int64_t qpos, int64_t e) {
  constexpr int P = 4;
  const int lane = lane_id();
  int64_t mq = -1, me = 0, mk = 0;
  float mr = 0.0f;
  if (lane < P && valid && qpos < p.qend && e < p.n) {
    mq = query_at(p.qlist, qpos);
    me = e;
    mr = p.cr[e];
    mk = (p.emap ? p.emap[e] : e) + p.eoff;
  }
  int64_t q[P], ee[P];
  bool v[P];
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(mq)), j);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(mq >> 32)), j);
    const int64_t qj = static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
    const uint32_t elo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(me)), j);
    const uint32_t ehi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(me >> 32)), j);
    v[j] = qj >= 0;
    q[j] = v[j] ? qj : 0;
    ee[j] = static_cast<int64_t>((static_cast<uint64_t>(ehi) << 32) | elo);
  }
  double acc[P];
#pragma unroll
  for (int j = 0; j < P; ++j) acc[j] = 0.0;
#pragma unroll 4
  for (int k = lane; k < p.d; k += kWave) {
    float qa[P];
    double za[P];
#pragma unroll
    for (int j = 0; j < P; ++j) {
      qa[j] = p.zq[q[j] * p.d + k];
      za[j] = cache_value<SRC>(p.cz, ee[j], p.d, k);
    }
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const double diff = static_cast<double>(qa[j]) - za[j];
      acc[j] = __builtin_fma(diff, diff, acc[j]);
    }
  }
  int done = 0;
#pragma unroll
  for (int j = 0; j < P; ++j) {
    done += v[j] ? 1 : 0;
    const double d2 = wave_sum(acc[j]);
    if (lane == j && v[j]) {
      // record_pair with the radius and key fetched above (the re-check
      // count is the caller's)
      const double r = static_cast<double>(mr);
      if (__builtin_fabs(__builtin_sqrt(d2) - r) <= 1e-5 * r) {
        atomicAdd(&p.stats[LIPCACHE_STAT_BAND_PAIRS], 1ull);
        atomicOr(&p.bflag[mq], 1u);
      }
      if (d2 < r * r) {
        const float d2f = static_cast<float>(d2);
        const unsigned long long key = (static_cast<unsigned long long>(__builtin_bit_cast(uint32_t, d2f)) << 32) |
                                       static_cast<unsigned long long>(static_cast<uint32_t>(mk));
        atomicMin(&p.best[mq], key);
      }
    }
  }
  return done;
}

template <int SRC>
__device__ __noinline__ void settle_queue(const RecheckArgs p, const int32_t* rq_q, const int64_t* rq_e, int n,
                                          int64_t qwave) {
  const int lane = lane_id();
  int done = 0;
  for (int b = 0; b < n; b += 4) {
    const bool mine = lane < 4 && b + lane < n;
    done += settle_four<SRC>(p, mine, mine ? qwave + rq_q[b + lane] : 0, mine ? rq_e[b + lane] : 0);
  }
  if (lane == 0 && done) atomicAdd(&p.stats[LIPCACHE_STAT_RECHECKED], static_cast<unsigned long long>(done));
}

// The global re-check queue of a work-list scan: wave w of the grid takes
// four pairs at a time, w * 4 + i * (4 * waves).  Every wave's loop bound is
// the same, so the grid drains.
template <int SRC>
__global__ __launch_bounds__(256) void recheck_queue_kernel(const RecheckArgs p, const int64_t* __restrict__ gpos,
                                                            const int64_t* __restrict__ ge,
                                                            const unsigned long long* __restrict__ gcount,
                                                            int64_t cap) {
  __shared__ unsigned int block_done;
  const int lane = lane_id();
  if (threadIdx.x == 0) block_done = 0u;
  __syncthreads();
  const int64_t reserved = static_cast<int64_t>(*gcount);
  const int64_t total = reserved < cap ? reserved : cap;
  const int64_t waves = static_cast<int64_t>(gridDim.x) * (blockDim.x / kWave);
  const int64_t w = static_cast<int64_t>(blockIdx.x) * (blockDim.x / kWave) + threadIdx.x / kWave;
  int done = 0;
  for (int64_t b = w * 4; b < total; b += waves * 4) {
    const int64_t i = b + lane;
    const bool mine = lane < 4 && i < total;
    const int64_t pos = mine ? gpos[i] : -1;
    done += settle_four<SRC>(p, mine && pos >= 0, pos, mine ? ge[i] : 0);
  }
  if (lane == 0 && done) atomicAdd(&block_done, static_cast<unsigned int>(done));
  __syncthreads();
  if (threadIdx.x == 0 && block_done)
    atomicAdd(&p.stats[LIPCACHE_STAT_RECHECKED], static_cast<unsigned long long>(block_done));
}

// Reads a wave-uniform 64-bit value from lane 0.
__device__ __forceinline__ uint64_t lane0_u64(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v)), 0);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v >> 32)), 0);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Slice mode: appends the pairs of `mask` (bit rt*4+i of lane (m16, g) =
// query row 4g + i of row tile rt against entry ebase + m16) to the global
// re-check queue, one pair per lane and pass with one reservation per pass.
// Pairs that find no slot below the capacity are re-checked at once (a cold
// path: the queue holds several pairs per query).
template <int SRC>
__device__ __forceinline__ void enqueue_pairs(const LookupParams& lp, uint32_t mask, int64_t qwave, int64_t ebase,
                                              int64_t qend, const int32_t* qlist) {
  const int lane = lane_id();
  const uint64_t cap = static_cast<uint64_t>(lp.gq_cap);
  uint32_t rest = 0u;
  while (true) {
    const bool has = mask != 0u;
    const unsigned long long bal = __ballot(has);
    if (bal == 0ull) break;
    uint64_t base = 0;
    if (lane == 0) base = atomicAdd(lp.gq_count, static_cast<unsigned long long>(__popcll(bal)));
    base = lane0_u64(base);
    if (has) {
      const int bit = __builtin_ctz(mask);
      const uint64_t slot = base + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(bal >> 32),
                                                             __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bal), 0u));
      if (slot < cap) {
        lp.gq_pos[slot] = qwave + (bit >> 2) * 16 + 4 * (lane >> 4) + (bit & 3);
        lp.gq_e[slot] = ebase + (lane & 15);
      } else {
        rest |= 1u << bit;
      }
      mask &= mask - 1u;
    }
  }
  if (__ballot(rest != 0u) != 0ull) recheck_pairs<SRC>(recheck_args(lp, qend, qlist), rest, qwave, ebase);
}

// Work-list mode: moves the wave's LDS queue to the global queue when it
// has room (one 64-bit atomic reserves the slots), else settles it here.
// The queue was written by other lanes of this wave.
template <int SRC>
__device__ __forceinline__ void flush_queue(const LookupParams& lp, const RecheckArgs& p, RecheckQueue& rq,
                                            int64_t qwave) {
  if (rq.n == 0) return;
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_wave_barrier();
  const int lane = lane_id();
  if (lp.gq_pos) {
    unsigned long long base = 0;
    if (lane == 0) base = atomicAdd(lp.gq_count, static_cast<unsigned long long>(rq.n));
    const uint64_t b0 = lane0_u64(base);
    const uint64_t cap = static_cast<uint64_t>(lp.gq_cap);
    if (b0 + static_cast<uint64_t>(rq.n) <= cap) {
      for (int i = lane; i < rq.n; i += kWave) {
        lp.gq_pos[b0 + i] = qwave + rq.q[i];
        lp.gq_e[b0 + i] = rq.e[i];
      }
      rq.n = 0;
      return;
    }
    // no room: mark the reserved slots that exist, settle here
    for (int i = lane; i < rq.n; i += kWave)
      if (b0 + i < cap) lp.gq_pos[b0 + i] = -1;
  }
  settle_queue<SRC>(p, rq.q, rq.e, rq.n, qwave);
  rq.n = 0;
}

// Work-list mode: queues the pairs of `mask` (bit layout as enqueue_pairs)
// in the wave's LDS queue; pairs that do not fit are re-checked at once.
template <int SRC>
__device__ __forceinline__ void queue_pairs(const RecheckArgs& p, RecheckQueue& rq, uint32_t mask, int64_t qwave,
                                            int64_t ebase) {
  const int lane = lane_id();
  while (true) {
    const bool has = mask != 0u;
    const unsigned long long bal = __ballot(has);
    if (bal == 0ull) break;
    const int fresh = __popcll(bal);
    if (rq.n + fresh > kRq) {
      recheck_pairs<SRC>(p, mask, qwave, ebase);
      break;
    }
    if (has) {
      const int bit = __builtin_ctz(mask);
      const int slot = rq.n + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                  static_cast<uint32_t>(bal >> 32),
                                  __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bal), 0u)));
      rq.q[slot] = (bit >> 2) * 16 + 4 * (lane >> 4) + (bit & 3);
      rq.e[slot] = ebase + (lane & 15);
      mask &= mask - 1u;
    }
    rq.n += fresh;
  }
}

// Queries as MFMA A operands: lane holds row m16 of each row tile and k-chunk
// g of each k-step (the cache operand uses the same (k-step, chunk) -> k map,
// so the contraction covers every k exactly once).  Positions past qend load
// the last query (any finite values do): their thresholds are +inf.
template <int MODE, int KS, int RT, bool Q16 = false>
__device__ __forceinline__ void load_query_operands(const LookupParams& p, const int32_t* qlist, int64_t qwave,
                                                    int64_t qend, int m16, int g, u32x4 (&a)[RT][KS]) {
  using T = ModeTraits<MODE>;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    int64_t pos = qwave + rt * 16 + m16;
    pos = pos < qend ? pos : qend - 1;
    const int64_t row = query_at(qlist, pos);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int k0 = ks * T::kPerStep + g * T::kPerChunk;
      if constexpr (Q16) {
        a[rt][ks] = load_chunk<MODE, LIPCACHE_F16>(p.zq16, row, p.d, k0);
      } else {
        a[rt][ks] = load_chunk<MODE, LIPCACHE_F32>(p.zq, row, p.d, k0);
      }
    }
  }
}

template <int MODE, int KS, int RT, bool Q16>
__device__ __forceinline__ void load_queries(const LookupParams& p, const int32_t* qlist, int64_t qwave, int64_t qend,
                                             int m16, int g, u32x4 (&a)[RT][KS], float (&qt)[RT][4]) {
  load_query_operands<MODE, KS, RT, Q16>(p, qlist, qwave, qend, m16, g, a);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t qr = qwave + rt * 16 + 4 * g + i;
      qt[rt][i] = qr < qend ? p.qthr[query_at(qlist, qr)] : __builtin_inff();
    }
  }
}

template <int MODE, int SRC, int KS, int RT, bool DUMP, bool LIST>
__global__ __launch_bounds__(kLkThreads, 2) void lookup_kernel(const LookupParams p) {
  using T = ModeTraits<MODE>;
  constexpr int kDPad = KS * T::kPerStep;
  constexpr int kRowBytes = kDPad * T::kElemBytes + 16;   // +16: conflict-free B reads
  constexpr int kChunksPerRow = kDPad * T::kElemBytes / 16;
  __shared__ __attribute__((aligned(16))) unsigned char tile[kTileN * kRowBytes];
  __shared__ float athr[kTileN];

  int64_t q0, qend, e_begin, e_end;
  block_work(p, kLkWaves * RT * 16, q0, qend, e_begin, e_end);
  const int32_t* qlist = LIST ? p.qlist : nullptr;
  if constexpr (!LIST) qend = p.B;

  const int lane = lane_id();
  const int wave = uniform(static_cast<int>(threadIdx.x) / kWave);
  const int m16 = lane & 15;
  const int g = lane >> 4;
  const int64_t qwave = q0 + wave * (RT * 16);

  u32x4 a[RT][KS];
  float qt[RT][4];
  load_queries<MODE, KS, RT, LIST && MODE == kModeF16>(p, qlist, qwave, qend, m16, g, a, qt);

  for (int64_t t0 = e_begin; t0 < e_end; t0 += kTileN) {
    __syncthreads();
    for (int c = threadIdx.x; c < kTileN * kChunksPerRow; c += kLkThreads) {
      const int row = c / kChunksPerRow;
      const int cc = c % kChunksPerRow;
      const int64_t e = t0 + row;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (e < e_end) v = load_chunk<MODE, SRC>(p.cz, e, p.d, cc * T::kPerChunk);
      *reinterpret_cast<u32x4*>(tile + row * kRowBytes + cc * 16) = v;
    }
    if (threadIdx.x < kTileN) {
      const int64_t e = t0 + threadIdx.x;
      athr[threadIdx.x] =
          e < e_end ? entry_threshold(p.cr[e], p.cnorm2[e], p.kappa_c, p.eta1, p.range2) : __builtin_inff();
    }
    __syncthreads();

    const int64_t left = e_end - t0;
    const int nsub = left >= kTileN ? kTileN / kColTile : static_cast<int>((left + kColTile - 1) / kColTile);
    for (int sub = 0; sub < nsub; ++sub) {
      u32x4 bv[KS];
      const unsigned char* brow = tile + (sub * kColTile + m16) * kRowBytes + g * 16;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) bv[ks] = *reinterpret_cast<const u32x4*>(brow + ks * 64);
      f32x4 acc[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[rt] = mfma_step<MODE>(a[rt][ks], bv[ks], acc[rt]);
      }
      const float an = athr[sub * kColTile + m16];
      const int64_t ebase = t0 + sub * kColTile;
      if constexpr (DUMP) {
        uint32_t mask = 0u;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
          for (int i = 0; i < 4; ++i) mask |= static_cast<uint32_t>((acc[rt][i] - qt[rt][i]) >= an) << (rt * 4 + i);
        }
        const int64_t e = ebase + m16;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int64_t q = qwave + rt * 16 + 4 * g + i;
            if (q < p.B && e < e_end) {
              p.g_hat[q * p.n + e] = acc[rt][i];
              p.cand[q * p.n + e] = static_cast<uint8_t>((mask >> (rt * 4 + i)) & 1u);
            }
          }
        }
      } else {
        // Fast path: one subtract and one compare per pair, OR-ed as lane
        // masks; the per-lane bit mask is only built when some pair passed.
        bool any = false;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
          for (int i = 0; i < 4; ++i) any |= (acc[rt][i] - qt[rt][i]) >= an;
        }
        if (__ballot(any) != 0ull) {
          uint32_t mask = 0u;
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
            for (int i = 0; i < 4; ++i) mask |= static_cast<uint32_t>((acc[rt][i] - qt[rt][i]) >= an) << (rt * 4 + i);
          }
          enqueue_pairs<SRC>(p, mask, qwave, ebase, qend, qlist);
        }
      }
    }
  }
}

// ------------------------------------------------------------- DMA pipeline kernel
// Same contraction, filter and re-check as lookup_kernel, but the cache tiles
// already have the MFMA element type in memory (a bf16 store, the bf16 image
// of an fp32 store, or an fp32 store for the fp32 filter), so they move from
// global memory straight into LDS with global_load_lds_dwordx4 (no registers,
// no conversion), double-buffered: the copy of tile t+1 is issued right after
// the barrier that publishes tile t and overlaps its computation.
//
// LDS rows are not padded; instead 16-byte chunk c of row `row` is stored in
// slot c ^ swz(row), so the 16 lanes that read one k-chunk of 16 consecutive
// rows hit 16 different bank groups.  The swizzle is applied to the global
// addresses of the copy (a permutation within each row, so reads stay
// coalesced).
typedef __attribute__((address_space(3))) void lds_void_t;

template <int CPR>
__device__ __forceinline__ int lds_swizzle(int row) {
  constexpr int kRowsPerBankSweep = CPR >= 16 ? 1 : 16 / CPR;
  constexpr int kMask = (CPR >= 16 ? 16 : CPR) - 1;
  return (row / kRowsPerBankSweep) & kMask;
}

// vmcnt(0): wait for this wave's outstanding copies into LDS.
__device__ __forceinline__ void wait_copies() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Global -> LDS copies (global_load_lds, saddr form): lane i's BYTES bytes at
// sbase + voff land at LDS byte address lds + BYTES * i (sbase and lds
// wave-uniform).  Written as inline assembly because the compiler models the
// intrinsic form as an out-of-order LDS event: while one is in flight every
// wait for an ordinary LDS read degrades to lgkmcnt(0), which serialises the
// operand prefetch of the matrix loop behind the latest read.  The copy is
// only counted by vmcnt, which the kernel waits on explicitly (wait_copies)
// before the barrier that publishes a tile; an unknown extra vmcnt entry can
// only make the compiler's own vmcnt waits stricter.  M0 carries the LDS
// address; SALU writes to M0 need one wait state before the copy reads it.
template <int BYTES>
__device__ __forceinline__ void lds_copy(const void* sbase, uint32_t voff, const void* lds) {
  const uint32_t m = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_void_t*)lds));
  if constexpr (BYTES == 16) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(m)
                 : "memory", "m0");
  } else {
    static_assert(BYTES == 4, "16- or 4-byte copies");
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1" ::"v"(voff), "s"(sbase), "s"(m)
                 : "memory", "m0");
  }
}

// Waves per workgroup of the slice-mode DMA kernel.
#ifndef LC_DMA_WAVES
#define LC_DMA_WAVES 8
#endif
constexpr int kDmaWaves = LC_DMA_WAVES;
// Waves per workgroup of the work-list DMA kernel: a cluster's query list
// is short (a few hundred queries), so an item of 4 waves (256 queries) and
// 64-row tiles lets two items share a CU where one 8-wave item would leave
// most of its waves idle.
constexpr int kListWaves = 4;

// Cache rows per LDS tile of the DMA kernel with NW waves: 64 KiB per buffer
// for 8 waves, 32 KiB for 4 (rows of 64 * KS bytes in either element type),
// at most 128 rows.
template <int KS, int NW>
struct DmaTraits {
  static constexpr int kRows = NW == 8 ? (KS <= 8 ? 128 : 64) : (KS <= 8 ? 64 : 32);
  static constexpr int kAthr = kRows < kWave ? kWave : kRows;  // thresholds staged per tile
};
constexpr int kDmaMaxRows = 128;

// k-steps of a full tile the cache operands are read from LDS ahead of
// their use.
#ifndef LC_PREFETCH
#define LC_PREFETCH 3
#endif
constexpr int kPrefetch = LC_PREFETCH;

template <int MODE, int KS, int NW>
__device__ __forceinline__ void issue_tile(unsigned char* buf, float* athr_buf, const LookupParams& p, int64_t t0,
                                           int64_t e_end, int wave) {
  using T = ModeTraits<MODE>;
  constexpr int kThreads = NW * kWave;
  constexpr int kCPR = 4 * KS;  // 16-byte chunks per LDS row
  constexpr int kRows = DmaTraits<KS, NW>::kRows;
  constexpr int kIters = kRows * kCPR / kThreads;
  static_assert(kIters >= 1 && kIters * kThreads == kRows * kCPR, "whole copies per thread");
  constexpr int kRowsPerIter = kThreads / kCPR;
  const int d_chunks = p.d * T::kElemBytes / 16;
  const int row_bytes = p.d * T::kElemBytes;
  const int tid = static_cast<int>(threadIdx.x);
  const int r0 = tid / kCPR;
  const int cs = tid % kCPR;
  // Wave-uniform tile base; per-thread 32-bit offsets inside the tile.
  const unsigned char* base = static_cast<const unsigned char*>(p.cimg) + t0 * static_cast<int64_t>(row_bytes);
  // The swizzle repeats every 16 rows.  When a thread's rows are 16k apart
  // its chunk column is the same in every copy of a full tile, so one offset
  // serves them all and the row step goes into the scalar base (one live
  // VGPR instead of one per copy).
  constexpr bool kSameColumn = kRowsPerIter % 16 == 0;
  if (kSameColumn && e_end - t0 >= kRows) {
    int c = cs ^ lds_swizzle<kCPR>(r0);
    if (c >= d_chunks) c -= d_chunks;
    const uint32_t voff = static_cast<uint32_t>(r0 * row_bytes + c * 16);
#pragma unroll
    for (int j = 0; j < kIters; ++j)
      lds_copy<16>(base + static_cast<int64_t>(j * kRowsPerIter) * row_bytes, voff,
                   buf + (j * kThreads + wave * kWave) * 16);
  } else {
    // Rows past the slice end repeat its last row (their thresholds are +inf).
    const int last = e_end - t0 < kRows ? static_cast<int>(e_end - t0) - 1 : kRows - 1;
#pragma unroll
    for (int j = 0; j < kIters; ++j) {
      const int row = j * kRowsPerIter + r0;
      int c = cs ^ lds_swizzle<kCPR>(row);
      // Chunks past d hold a copy of a real chunk: the query operand is zero
      // there, so they add nothing.
      if (c >= d_chunks) c -= d_chunks;
      const int rr = row < last ? row : last;
      lds_copy<16>(base, static_cast<uint32_t>(rr * row_bytes + c * 16), buf + (j * kThreads + wave * kWave) * 16);
    }
  }
  // thresholds of the tile's rows (+inf padding past n): one wave per 64,
  // at least 64 (a tile of fewer rows stages the next ones too; the array
  // holds them: it is padded by kDmaMaxRows past the last tile start)
  if (wave < DmaTraits<KS, NW>::kAthr / kWave)
    lds_copy<4>(p.athr + t0 + wave * kWave, static_cast<uint32_t>(lane_id() * 4),
                static_cast<unsigned char*>(static_cast<void*>(athr_buf)) + wave * kWave * 4);
}

// The cache operand of (column tile `sub`, k-step ks) for this lane: chunk
// 4 ks + g of row sub*16 + m16.  For rows of >= 16 chunks the swizzle is a
// 4-bit XOR, so the slot splits into a part that depends on ks only through
// its low two bits and a multiple of 256 bytes: four base addresses and
// immediate offsets cover all k-steps.
template <int KS>
__device__ __forceinline__ u32x4 lds_operand(const unsigned char* buf, int sub, int ks, int m16, int g) {
  constexpr int kCPR = 4 * KS;
  const int row = sub * kColTile + m16;
  const int sw = lds_swizzle<kCPR>(row);
  if constexpr (kCPR >= 16) {
    const int off = row * kCPR * 16 + ((g ^ (sw & 3)) * 16) + (((ks & 3) ^ (sw >> 2)) * 64) + (ks >> 2) * 256;
    return *reinterpret_cast<const u32x4*>(buf + off);
  } else {
    return *reinterpret_cast<const u32x4*>(buf + row * kCPR * 16 + (((ks * 4 + g) ^ sw) * 16));
  }
}

// One LDS tile: for each 16-entry column tile, KS k-steps of RT MFMAs, then
// the filter.  The cache operands are read from LDS two k-steps ahead of
// their use (continuing into the next column tile), so LDS latency overlaps
// the MFMAs.  The filter takes max_j (acc_j - Q_j) over the lane's 16
// accumulators (max_j acc_j where they started at -Q_j; maxnum ignores NaN,
// so a NaN pair never hides another pair)
// and compares once against A_i; the exact per-pair mask is only rebuilt on
// the rare path.
// Rare path of one column tile: rebuild the exact per-pair mask and re-check.
template <int STORE, int RT, bool LIST>
__device__ __forceinline__ void filter_and_recheck(const LookupParams& p, const f32x4 (&acc)[RT], const f32x4 (&qt)[RT],
                                                   float an, int64_t qwave, int64_t qend, const int32_t* qlist,
                                                   int64_t ebase, RecheckQueue& rq) {
  uint32_t mask = 0u;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) mask |= static_cast<uint32_t>((acc[rt][i] - qt[rt][i]) >= an) << (rt * 4 + i);
  }
  if constexpr (LIST) {
    queue_pairs<STORE>(recheck_args(p, qend, qlist), rq, mask, qwave, ebase);
  } else {
    enqueue_pairs<STORE>(p, mask, qwave, ebase, qend, qlist);
  }
}

// A full LDS tile, software-pipelined: while the MFMAs of column tile s run,
// the same wave evaluates the filter of column tile s - 1 (its accumulators
// are kept one step longer), so the filter's VALU work fills the matrix
// pipe's shadow instead of following it.
template <int MODE, int STORE, int KS, int RT, int NW, bool LIST>
__device__ __forceinline__ void compute_full_tile(const unsigned char* buf, const float* athr_buf,
                                                  const LookupParams& p, int64_t t0, int64_t qwave, int64_t qend,
                                                  const int32_t* qlist, int m16, int g,
                                                  const u32x4 (&a)[RT][KS], const f32x4 (&qv)[RT],
                                                  RecheckQueue& rq) {
  constexpr int kSubs = DmaTraits<KS, NW>::kRows / kColTile;
  constexpr int kE = RT * 4;                      // accumulators per lane
  constexpr int kPer = (kE + KS - 1) / KS;        // filter terms folded into each k-step
  constexpr int kSteps = kSubs * KS;              // k-steps of the whole tile
  constexpr int kPre = kPrefetch < kSteps ? kPrefetch : kSteps;
  // Ring of the cache operands read ahead: step j of the tile (column tile
  // j / KS, k-step j % KS) uses slot j % kPre, filled kPre steps earlier.
  u32x4 bq[kPre];
#pragma unroll
  for (int j = 0; j < kPre; ++j) bq[j] = lds_operand<KS>(buf, j / KS, j % KS, m16, g);
  f32x4 accp[RT];
  float anp = 0.0f;
#pragma unroll
  for (int sub = 0; sub <= kSubs; ++sub) {
    const bool cur = sub < kSubs;   // compile-time after unrolling
    const bool prev = sub > 0;
    f32x4 acc[RT];
    float an = 0.0f;
    f32x4 qt[RT];
    if (prev) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) qt[rt] = kFoldQ<MODE, KS> ? f32x4{0.f, 0.f, 0.f, 0.f} : qv[rt];
    }
    if (cur) {
      an = athr_buf[sub * kColTile + m16];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt] = kFoldQ<MODE, KS> ? qv[rt] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (cur) {
        const int step = sub * KS + ks;
        const u32x4 op = bq[step % kPre];
        if (step + kPre < kSteps) bq[step % kPre] = lds_operand<KS>(buf, (step + kPre) / KS, (step + kPre) % KS, m16, g);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[rt] = mfma_step<MODE>(a[rt][ks], op, acc[rt]);
      }
      if (prev) {
#pragma unroll
        for (int e = ks * kPer; e < (ks + 1) * kPer && e < kE; ++e)
          mx = __builtin_fmaxf(mx, kFoldQ<MODE, KS> ? accp[e / 4][e % 4] : accp[e / 4][e % 4] - qt[e / 4][e % 4]);
      }
      // Keep the operand read for step + kPre in this step: left to itself
      // the scheduler sinks it next to its use and the wave stalls on the
      // LDS latency every few MFMAs.
      __builtin_amdgcn_sched_barrier(0);
    }
    if (prev) {
      // rare: the rare path is laid out of line, so the column tiles run as
      // one straight sequence and the common case takes no branch
      if (__builtin_expect(__ballot(mx >= anp) != 0ull, 0))
        filter_and_recheck<STORE, RT, LIST>(p, accp, qt, anp, qwave, qend, qlist, t0 + (sub - 1) * kColTile, rq);
    }
    if (cur) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) accp[rt] = acc[rt];
      anp = an;
    }
  }
}

// Thresholds of the lane's accumulator rows 4g .. 4g + 3 of each row tile
// (+inf past qend), negated where the accumulators start at -Q_q.
template <int RT>
__device__ __forceinline__ void load_thresholds(const float* thr, int64_t qwave, int64_t qend, const int32_t* qlist,
                                                int g, bool negate, f32x4 (&qv)[RT]) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t q = qwave + rt * 16 + 4 * g + i;
      const float qq = q < qend ? thr[query_at(qlist, q)] : __builtin_inff();
      qv[rt][i] = negate ? -qq : qq;
    }
  }
}

template <int MODE, int STORE, int KS, int RT, int NW, bool DUMP, bool LIST>
__device__ __forceinline__ void compute_tile(const unsigned char* buf, const float* athr_buf, const LookupParams& p,
                                             int64_t t0, int64_t e_end, int64_t qwave, int64_t qend,
                                             const int32_t* qlist, int m16, int g, const u32x4 (&a)[RT][KS],
                                             const f32x4 (&qv)[RT], RecheckQueue& rq) {
  constexpr int kRows = DmaTraits<KS, NW>::kRows;
  const int64_t left = e_end - t0;
  if constexpr (!DUMP) {
    if (left >= kRows) {
      compute_full_tile<MODE, STORE, KS, RT, NW, LIST>(buf, athr_buf, p, t0, qwave, qend, qlist, m16, g, a, qv, rq);
      return;
    }
  }
  const int nsub = left >= kRows ? kRows / kColTile : static_cast<int>((left + kColTile - 1) / kColTile);
  u32x4 b0 = lds_operand<KS>(buf, 0, 0, m16, g);
  u32x4 b1 = KS > 1 ? lds_operand<KS>(buf, 0, 1, m16, g) : b0;
  // Fully unrolled so every LDS address is a fixed offset from `buf`, which
  // lets the compiler see that these reads do not touch the other buffer
  // (whose copy is still in flight) and skip a wait on it.
#pragma unroll
  for (int sub = 0; sub < kRows / kColTile; ++sub) {
    if (sub >= nsub) break;
    // rows past the range end (real rows of the next range in work-list
    // mode) never pass
    const float an = t0 + sub * kColTile + m16 < e_end ? athr_buf[sub * kColTile + m16] : __builtin_inff();
    f32x4 acc[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[rt] = kFoldQ<MODE, KS> ? qv[rt] : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 cur = (ks & 1) ? b1 : b0;
      int nks = ks + 2, nsb = sub;
      if (nks >= KS) {
        nks -= KS;
        nsb += 1;
      }
      u32x4 pre = cur;
      if (KS > 1 && nsb < nsub) pre = lds_operand<KS>(buf, nsb, nks, m16, g);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt] = mfma_step<MODE>(a[rt][ks], cur, acc[rt]);
      if (ks & 1) {
        b1 = pre;
      } else {
        b0 = pre;
      }
    }
    if constexpr (KS == 1) {
      if (sub + 1 < nsub) b0 = lds_operand<KS>(buf, sub + 1, 0, m16, g);
    }
    const int64_t ebase = t0 + sub * kColTile;
    // Q_q of the four rows 4g..4g+3 of each row tile (this lane's
    // accumulators), or zero where the accumulators already hold g - Q_q
    f32x4 qt[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) qt[rt] = kFoldQ<MODE, KS> ? f32x4{0.f, 0.f, 0.f, 0.f} : qv[rt];
    if constexpr (DUMP) {
      const int64_t e = ebase + m16;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t q = qwave + rt * 16 + 4 * g + i;
          if (q < p.B && e < e_end) {
            p.g_hat[q * p.n + e] = kFoldQ<MODE, KS> ? acc[rt][i] - qv[rt][i] : acc[rt][i];
            p.cand[q * p.n + e] = static_cast<uint8_t>((acc[rt][i] - qt[rt][i]) >= an);
          }
        }
      }
    } else {
      float mx = -__builtin_inff();
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) mx = __builtin_fmaxf(mx, acc[rt][i] - qt[rt][i]);
      }
      if (__ballot(mx >= an) != 0ull) {
        uint32_t mask = 0u;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
          for (int i = 0; i < 4; ++i) mask |= static_cast<uint32_t>((acc[rt][i] - qt[rt][i]) >= an) << (rt * 4 + i);
        }
        if constexpr (LIST) {
          queue_pairs<STORE>(recheck_args(p, qend, qlist), rq, mask, qwave, ebase);
        } else {
          enqueue_pairs<STORE>(p, mask, qwave, ebase, qend, qlist);
        }
      }
    }
  }
}

// NW waves per workgroup (8, or 4 with two workgroups per CU), two waves
// per SIMD either way.
template <int MODE, int STORE, int KS, int RT, int NW, bool DUMP, bool LIST>
__global__ __launch_bounds__(NW * kWave, 2) void lookup_dma_kernel(const LookupParams p) {
  using T = ModeTraits<MODE>;
  constexpr int kCPR = 4 * KS;
  constexpr int kRows = DmaTraits<KS, NW>::kRows;
  constexpr int kTileBytes = kRows * kCPR * 16;
  __shared__ __attribute__((aligned(16))) unsigned char buf0[kTileBytes];
  __shared__ __attribute__((aligned(16))) unsigned char buf1[kTileBytes];
  __shared__ __attribute__((aligned(16))) float ath0[DmaTraits<KS, NW>::kAthr];
  __shared__ __attribute__((aligned(16))) float ath1[DmaTraits<KS, NW>::kAthr];
  __shared__ int64_t rq_e[LIST ? NW * kRq : 1];
  __shared__ int32_t rq_q[LIST ? NW * kRq : 1];

  int64_t q0, qend, e_begin, e_end;
  block_work(p, NW * RT * 16, q0, qend, e_begin, e_end);
  const int32_t* qlist = LIST ? p.qlist : nullptr;
  if constexpr (!LIST) qend = p.B;

  const int lane = lane_id();
  const int wave = uniform(static_cast<int>(threadIdx.x) / kWave);
  const int m16 = lane & 15;
  const int g = lane >> 4;
  const int64_t qwave = q0 + wave * (RT * 16);

  if (e_begin >= e_end) return;  // whole workgroup: an empty slice
  // Work-list mode: a wave whose queries all lie past the list's end only
  // moves its share of each tile (the copies and barriers are the block's).
  const bool active = !LIST || qwave < qend;
  issue_tile<MODE, KS, NW>(buf0, ath0, p, e_begin, e_end, wave);

  u32x4 a[RT][KS];
  if (active) load_query_operands<MODE, KS, RT, LIST && MODE == kModeF16>(p, qlist, qwave, qend, m16, g, a);
  RecheckQueue rq{rq_q + (LIST ? wave * kRq : 0), rq_e + (LIST ? wave * kRq : 0), 0};
  // Q_q of this lane's accumulator rows 4g .. 4g + 3 of each row tile, kept
  // in registers for the whole slice (reading them from LDS per column tile
  // costs a third of the operand traffic); +inf past B.  Negated where the
  // accumulators start at -Q_q.
  f32x4 qv[RT];
  load_thresholds<RT>(p.qthr, qwave, qend, qlist, g, kFoldQ<MODE, KS>, qv);

  for (int64_t t0 = e_begin;; t0 += 2 * kRows) {
    wait_copies();
    __syncthreads();
    const bool more1 = t0 + kRows < e_end;
    if (more1) issue_tile<MODE, KS, NW>(buf1, ath1, p, t0 + kRows, e_end, wave);
    if (active)
      compute_tile<MODE, STORE, KS, RT, NW, DUMP, LIST>(buf0, ath0, p, t0, e_end, qwave, qend, qlist, m16, g, a, qv, rq);
    if (!more1) break;
    wait_copies();
    __syncthreads();
    const bool more2 = t0 + 2 * kRows < e_end;
    if (more2) issue_tile<MODE, KS, NW>(buf0, ath0, p, t0 + 2 * kRows, e_end, wave);
    if (active)
      compute_tile<MODE, STORE, KS, RT, NW, DUMP, LIST>(buf1, ath1, p, t0 + kRows, e_end, qwave, qend, qlist, m16, g, a, qv, rq);
    if (!more2) break;
  }
  if constexpr (LIST) {
    if (active) flush_queue<STORE>(p, recheck_args(p, qend, qlist), rq, qwave);
  }
}

// ------------------------------------------------------------- pruned scan
// The pruned lookup (LIPCACHE_LOOKUP_PRUNE) streams only the prefix of every
// row: 64 bytes (features 0..31 of the float16 image) per row, 1024 rows per
// 64 KiB LDS tile, double-buffered, with the prefix thresholds A'_i of the
// tile's rows.  Each 16-entry column tile gets k-step 0 only; the rare column
// tiles where a pair passes the prefix filter are formed again from the
// image in global memory, exactly as the full kernel forms them, and go
// through the full filter and the re-check.
constexpr int kPrRows = 1024;                 // rows per prefix tile
constexpr int kPrSubs = kPrRows / kColTile;   // column tiles per prefix tile

// Copies rows [t0, t0 + kPrRows) of the prefix into an LDS tile (rows past
// e_end repeat its last row) and their thresholds A'_i.  Thread tid copies
// chunk tid % 4 of rows tid / 4 + 128 j; in the tile, chunk c of row r sits
// in slot c ^ swz(r) (the layout lds_operand<1> reads), and swz(r) =
// (r / 4) % 4 is the same for all of a thread's rows.
__device__ __forceinline__ void issue_prefix_tile(unsigned char* buf, float* athp_buf, const LookupParams& p,
                                                  int64_t t0, int64_t e_end, int wave) {
  constexpr int kThreads = kDmaWaves * kWave;
  constexpr int kRowsPerIter = kThreads / 4;
  constexpr int kIters = kPrRows / kRowsPerIter;
  const int row_bytes = p.d * 2;
  const int tid = static_cast<int>(threadIdx.x);
  const int r0 = tid / 4;
  const int c = (tid % 4) ^ lds_swizzle<4>(r0);
  const unsigned char* base = static_cast<const unsigned char*>(p.cimg) + t0 * static_cast<int64_t>(row_bytes);
  if (e_end - t0 >= kPrRows) {
    const uint32_t voff = static_cast<uint32_t>(r0 * row_bytes + c * 16);
#pragma unroll
    for (int j = 0; j < kIters; ++j)
      lds_copy<16>(base + static_cast<int64_t>(j * kRowsPerIter) * row_bytes, voff,
                   buf + (j * kThreads + wave * kWave) * 16);
  } else {
    const int last = static_cast<int>(e_end - t0) - 1;
#pragma unroll
    for (int j = 0; j < kIters; ++j) {
      const int row = j * kRowsPerIter + r0;
      const int rr = row < last ? row : last;
      lds_copy<16>(base, static_cast<uint32_t>(rr * row_bytes + c * 16), buf + (j * kThreads + wave * kWave) * 16);
    }
  }
  // thresholds: 1024 floats, two 64-float copies per wave (the array is
  // padded with +inf past n by more than a tile)
#pragma unroll
  for (int i = 0; i < kPrRows / (kDmaWaves * kWave); ++i) {
    const int w = wave * (kPrRows / (kDmaWaves * kWave)) + i;
    lds_copy<4>(p.athr_p + t0 + w * kWave, static_cast<uint32_t>(lane_id() * 4),
                static_cast<unsigned char*>(static_cast<void*>(athp_buf)) + w * kWave * 4);
  }
}

// Rare path of the pruned scan: column tile `sub` of the prefix tile at t0
// (rows e = t0 + 16 sub + m16, those at or past e_end never pass) formed as
// the full kernel forms it, from the image in global memory, then the full
// filter and the re-check.
template <int STORE, int KS, int RT>
__device__ __forceinline__ void prune_survivor(const LookupParams& p, int64_t t0, int sub, int64_t e_end,
                                               int64_t qwave, int64_t qend, int m16, int g,
                                               const u32x4 (&a)[RT][KS], RecheckQueue& rq) {
  constexpr bool kFold = kFoldQ<kModeF16, KS>;
  const int64_t ebase = t0 + static_cast<int64_t>(sub) * kColTile;
  const int64_t e = ebase + m16;
  const bool live = e < e_end;
  const int64_t er = live ? e : e_end - 1;
  f32x4 qf[RT];
  load_thresholds<RT>(p.qthr, qwave, qend, nullptr, g, kFold, qf);
  f32x4 acc[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = kFold ? qf[rt] : f32x4{0.f, 0.f, 0.f, 0.f};
  u32x4 b[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) b[ks] = load_chunk<kModeF16, LIPCACHE_F16>(p.cimg, er, p.d, ks * 32 + g * 8);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[rt] = mfma_step<kModeF16>(a[rt][ks], b[ks], acc[rt]);
  }
  f32x4 qt[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) qt[rt] = kFold ? f32x4{0.f, 0.f, 0.f, 0.f} : qf[rt];
  const float an = live ? p.athr[e] : __builtin_inff();
  float mx = -__builtin_inff();
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) mx = __builtin_fmaxf(mx, acc[rt][i] - qt[rt][i]);
  }
  if (__ballot(mx >= an) != 0ull) filter_and_recheck<STORE, RT, false>(p, acc, qt, an, qwave, qend, nullptr, ebase, rq);
}

// One prefix tile: k-step 0 of every column tile against the lane's 16
// queries (accumulators started at -Q'_q: the test is max_16(acc) >= A'_i),
// software-pipelined one column tile behind, with the operands read two
// column tiles ahead; passing column tiles are marked in a wave-uniform
// mask and formed again after the tile.  A partial tile (the end of a
// slice) takes a plain loop that also masks rows past e_end.
template <int STORE, int KS, int RT>
__device__ __forceinline__ void prune_tile(const unsigned char* buf, const float* athp_buf, const LookupParams& p,
                                           int64_t t0, int64_t e_end, int64_t qwave, int64_t qend, int m16, int g,
                                           const u32x4 (&a)[RT][KS], const f32x4 (&nqp)[RT], RecheckQueue& rq) {
  uint64_t pass = 0ull;
  if (e_end - t0 >= kPrRows) {
    u32x4 bq[2];
    bq[0] = lds_operand<1>(buf, 0, 0, m16, g);
    bq[1] = lds_operand<1>(buf, 1, 0, m16, g);
    f32x4 pacc[RT];
    float anp = 0.0f;
#pragma unroll
    for (int sub = 0; sub <= kPrSubs; ++sub) {
      const bool cur = sub < kPrSubs;  // compile-time after unrolling
      const bool prev = sub > 0;
      f32x4 acc[RT];
      float an = 0.0f;
      if (cur) {
        const u32x4 op = bq[sub & 1];
        if (sub + 2 < kPrSubs) bq[sub & 1] = lds_operand<1>(buf, sub + 2, 0, m16, g);
        an = athp_buf[sub * kColTile + m16];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[rt] = mfma_step<kModeF16>(a[rt][0], op, nqp[rt]);
      }
      if (prev) {
        float mx = -__builtin_inff();
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = __builtin_fmaxf(mx, pacc[rt][i]);
        }
        pass |= __ballot(mx >= anp) != 0ull ? 1ull << (sub - 1) : 0ull;
      }
      if (cur) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) pacc[rt] = acc[rt];
        anp = an;
      }
    }
  } else {
    const int64_t left = e_end - t0;
    const int nsub = static_cast<int>((left + kColTile - 1) / kColTile);
#pragma unroll 1
    for (int sub = 0; sub < nsub; ++sub) {
      const u32x4 op = lds_operand<1>(buf, sub, 0, m16, g);
      const float an = sub * kColTile + m16 < left ? athp_buf[sub * kColTile + m16] : __builtin_inff();
      float mx = -__builtin_inff();
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const f32x4 acc = mfma_step<kModeF16>(a[rt][0], op, nqp[rt]);
#pragma unroll
        for (int i = 0; i < 4; ++i) mx = __builtin_fmaxf(mx, acc[i]);
      }
      pass |= __ballot(mx >= an) != 0ull ? 1ull << sub : 0ull;
    }
  }
  if (__builtin_expect(pass != 0ull, 0)) {
#pragma unroll 1
    for (int sub = 0; sub < kPrSubs; ++sub)
      if ((pass >> sub) & 1ull) prune_survivor<STORE, KS, RT>(p, t0, sub, e_end, qwave, qend, m16, g, a, rq);
  }
}

// The pruned scan (slice mode): one 512-thread workgroup per (query block,
// cache slice), 8 waves of RT row tiles of queries, the query operands of
// all KS k-steps in registers (the survivors need them), the negated prefix
// thresholds of the lane's 16 queries as the start value of k-step 0.
template <int STORE, int KS, int RT>
__global__ __launch_bounds__(kDmaWaves * kWave, 2) void lookup_prune_kernel(const LookupParams p) {
  static_assert(KS >= 2, "a prefix shorter than the row");
  __shared__ __attribute__((aligned(16))) unsigned char buf0[kPrRows * 64];
  __shared__ __attribute__((aligned(16))) unsigned char buf1[kPrRows * 64];
  __shared__ __attribute__((aligned(16))) float athp0[kPrRows];
  __shared__ __attribute__((aligned(16))) float athp1[kPrRows];

  int64_t q0, qend, e_begin, e_end;
  block_work(p, kDmaWaves * RT * 16, q0, qend, e_begin, e_end);
  qend = p.B;
  const int lane = lane_id();
  const int wave = uniform(static_cast<int>(threadIdx.x) / kWave);
  const int m16 = lane & 15;
  const int g = lane >> 4;
  const int64_t qwave = q0 + wave * (RT * 16);
  if (e_begin >= e_end) return;  // whole workgroup: an empty slice
  issue_prefix_tile(buf0, athp0, p, e_begin, e_end, wave);

  u32x4 a[RT][KS];
  load_query_operands<kModeF16, KS, RT, false>(p, nullptr, qwave, qend, m16, g, a);
  f32x4 nqp[RT];
  load_thresholds<RT>(p.qthr_p, qwave, qend, nullptr, g, true, nqp);
  RecheckQueue rq{nullptr, nullptr, 0};

  for (int64_t t0 = e_begin;; t0 += 2 * kPrRows) {
    wait_copies();
    __syncthreads();
    const bool more1 = t0 + kPrRows < e_end;
    if (more1) issue_prefix_tile(buf1, athp1, p, t0 + kPrRows, e_end, wave);
    prune_tile<STORE, KS, RT>(buf0, athp0, p, t0, e_end, qwave, qend, m16, g, a, nqp, rq);
    if (!more1) break;
    wait_copies();
    __syncthreads();
    const bool more2 = t0 + 2 * kPrRows < e_end;
    if (more2) issue_prefix_tile(buf0, athp0, p, t0 + 2 * kPrRows, e_end, wave);
    prune_tile<STORE, KS, RT>(buf1, athp1, p, t0 + kPrRows, e_end, qwave, qend, m16, g, a, nqp, rq);
    if (!more2) break;
  }
}

// ------------------------------------------------------------- dispatch
struct Plan {
  int ks = 0;
  int rt = 0;
  int d_pad = 0;
  int qblock = 0;
  bool dma = false;
  int waves = 0;      // waves per workgroup
  int tile_rows = 0;  // cache rows per LDS tile of the chosen kernel
};

inline int rt_for(int ks) { return ks <= 8 ? 4 : (ks == 16 ? 2 : 1); }

inline bool make_plan(int precision, const lipcache_cache* c, bool list, Plan& pl, int list_waves = kListWaves) {
  const int per_step = precision == LIPCACHE_F16 ? 32 : 16;
  int ks = precision == LIPCACHE_F16 ? 1 : 2;
  while (ks * per_step < c->d) ks *= 2;
  if (ks > 32) return false;
  pl.ks = ks;
  pl.rt = rt_for(ks);
  pl.d_pad = ks * per_step;
  // The DMA kernel needs rows already in the MFMA element type (the float16
  // image, or an fp32 store for the fp32 filter) and two LDS tiles of at
  // most 64 KiB.
  const bool same_type = precision == LIPCACHE_F16 ? c->zimg != nullptr : c->store_dtype == LIPCACHE_F32;
  pl.dma = same_type && ks <= 16;
  pl.waves = pl.dma ? (list ? list_waves : kDmaWaves) : kLkWaves;
  pl.qblock = pl.waves * pl.rt * 16;
  if (pl.dma) {
    pl.tile_rows = pl.waves == 8 ? (ks <= 8 ? 128 : 64) : (ks <= 8 ? 64 : 32);  // DmaTraits<KS, NW>::kRows
  } else {
    pl.tile_rows = kTileN;
  }
  return true;
}

// Kernel variants: the lookup, the filter dump, and the work-list lookup of
// the cluster index.
enum { kVarLookup = 0, kVarDump = 1, kVarList = 2, kVarList8 = 3 };

template <int MODE, int SRC, int KS, int VAR>
hipError_t launch_v1(const LookupParams& p, unsigned grid, hipStream_t s) {
  hipLaunchKernelGGL((lookup_kernel<MODE, SRC, KS, (KS <= 8 ? 4 : (KS == 16 ? 2 : 1)), VAR == kVarDump,
                                    VAR == kVarList || VAR == kVarList8>),
                     dim3(grid), dim3(kLkThreads), 0, s, p);
  return hipGetLastError();
}

template <int MODE, int STORE, int KS, int VAR>
hipError_t launch_dma(const LookupParams& p, unsigned grid, hipStream_t s) {
  if constexpr (KS <= 16) {
    constexpr int kNW = VAR == kVarList ? kListWaves : kDmaWaves;
    hipLaunchKernelGGL((lookup_dma_kernel<MODE, STORE, KS, (KS <= 8 ? 4 : 2), kNW, VAR == kVarDump,
                                          VAR == kVarList || VAR == kVarList8>),
                       dim3(grid), dim3(kNW * kWave), 0, s, p);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

template <int MODE, int SRC, int VAR>
hipError_t launch_ks(const Plan& pl, const LookupParams& p, unsigned grid, hipStream_t s) {
  switch (pl.ks) {
#define LC_CASE(K) \
  case K: return pl.dma ? launch_dma<MODE, SRC, K, VAR>(p, grid, s) : launch_v1<MODE, SRC, K, VAR>(p, grid, s);
    LC_CASE(1)
    LC_CASE(2)
    LC_CASE(4)
    LC_CASE(8)
    LC_CASE(16)
    LC_CASE(32)
#undef LC_CASE
    default: return hipErrorInvalidValue;
  }
}

template <int VAR>
hipError_t launch_lookup(int precision, int store, const Plan& pl, const LookupParams& p, unsigned grid,
                         hipStream_t s) {
  if (precision == LIPCACHE_F16) {
    return store == LIPCACHE_F32 ? launch_ks<kModeF16, LIPCACHE_F32, VAR>(pl, p, grid, s)
                                 : launch_ks<kModeF16, LIPCACHE_BF16, VAR>(pl, p, grid, s);
  }
  return store == LIPCACHE_F32 ? launch_ks<kModeF32, LIPCACHE_F32, VAR>(pl, p, grid, s)
                               : launch_ks<kModeF32, LIPCACHE_BF16, VAR>(pl, p, grid, s);
}

// The pruned scan (float16 image, 2 <= KS <= 16; see prune_consts).
template <int STORE>
hipError_t launch_prune_store(const Plan& pl, const LookupParams& p, unsigned grid, hipStream_t s) {
  switch (pl.ks) {
#define LC_PCASE(K)                                                                                            \
  case K:                                                                                                      \
    hipLaunchKernelGGL((lookup_prune_kernel<STORE, K, (K <= 8 ? 4 : 2)>), dim3(grid), dim3(kDmaWaves * kWave), 0, \
                       s, p);                                                                                  \
    return hipGetLastError();
    LC_PCASE(2)
    LC_PCASE(4)
    LC_PCASE(8)
    LC_PCASE(16)
#undef LC_PCASE
    default: return hipErrorInvalidValue;
  }
}

inline hipError_t launch_prune(int store, const Plan& pl, const LookupParams& p, unsigned grid, hipStream_t s) {
  return store == LIPCACHE_F32 ? launch_prune_store<LIPCACHE_F32>(pl, p, grid, s)
                               : launch_prune_store<LIPCACHE_BF16>(pl, p, grid, s);
}

// Workgroups a slice scan aims for (at least a few per CU, for balance).
#ifndef LC_GRID_TARGET
#define LC_GRID_TARGET 256
#endif
constexpr int64_t kGridTarget = LC_GRID_TARGET;

// The global re-check queue of a scan (workspace memory): 4 B + 65536
// pairs; a pair that finds it full is re-checked by its wave at once.
struct GlobalRecheckWs {
  int64_t* pos;
  int64_t* e;
  unsigned long long* count;
  int64_t cap;
};

inline int64_t gq_capacity(int64_t B) { return 4 * (B > 0 ? B : 0) + 65536; }

struct Workspace {
  float* qthr;
  unsigned long long* best;
  unsigned int* bflag;
  unsigned long long* stats;
  float* athr;
  GlobalRecheckWs gq;
  float* qthr_p;  // pruned lookup only: Q'_q [B], A'_i [athp_len(N)]
  float* athr_p;
};

// A_i padded with +inf so that any tile that starts below n reads thresholds
// only from this array.
inline int64_t athr_len(int64_t n) {
  return ((n > 0 ? n : 0) + kDmaMaxRows - 1) / kDmaMaxRows * kDmaMaxRows + kDmaMaxRows;
}

// A'_i of the pruned scan, padded with +inf so that a prefix tile starting
// below n reads only this array.
inline int64_t athp_len(int64_t n) { return ((n > 0 ? n : 0) + kPrRows - 1) / kPrRows * kPrRows + kPrRows; }

inline size_t ws_layout(int64_t B, int64_t N, Workspace* w, void* base, bool prune = false) {
  const size_t nb = static_cast<size_t>(B > 0 ? B : 0);
  const int64_t cap = gq_capacity(B);
  size_t off = 0;
  const size_t o_best = off;
  off = align_up(off + nb * 8, 256);
  const size_t o_qthr = off;
  off = align_up(off + nb * 4, 256);
  const size_t o_flag = off;
  off = align_up(off + nb * 4, 256);
  const size_t o_stats = off;
  off = align_up(off + 4 * 8, 256);
  const size_t o_gqc = off;
  off = align_up(off + 8, 256);
  const size_t o_gqp = off;
  off = align_up(off + static_cast<size_t>(cap) * 8, 256);
  const size_t o_gqe = off;
  off = align_up(off + static_cast<size_t>(cap) * 8, 256);
  const size_t o_athr = off;
  off = align_up(off + static_cast<size_t>(athr_len(N)) * 4, 256);
  const size_t o_qp = off;
  if (prune) off = align_up(off + nb * 4, 256);
  const size_t o_ap = off;
  if (prune) off = align_up(off + static_cast<size_t>(athp_len(N)) * 4, 256);
  if (w && base) {
    char* b = static_cast<char*>(base);
    w->best = reinterpret_cast<unsigned long long*>(b + o_best);
    w->qthr = reinterpret_cast<float*>(b + o_qthr);
    w->bflag = reinterpret_cast<unsigned int*>(b + o_flag);
    w->stats = reinterpret_cast<unsigned long long*>(b + o_stats);
    w->gq = GlobalRecheckWs{reinterpret_cast<int64_t*>(b + o_gqp), reinterpret_cast<int64_t*>(b + o_gqe),
                            reinterpret_cast<unsigned long long*>(b + o_gqc), cap};
    w->athr = reinterpret_cast<float*>(b + o_athr);
    w->qthr_p = prune ? reinterpret_cast<float*>(b + o_qp) : nullptr;
    w->athr_p = prune ? reinterpret_cast<float*>(b + o_ap) : nullptr;
  }
  return off;
}

inline bool cache_ok(const lipcache_cache* c) {
  if (!c) return false;
  if (c->d < 32 || c->d > 1024 || c->d % 32 != 0) return false;
  if (c->store_dtype != LIPCACHE_F32 && c->store_dtype != LIPCACHE_BF16) return false;
  if (c->n < 0 || c->capacity < 0 || c->n > c->capacity) return false;
  if (c->n >= static_cast<int64_t>(UINT_MAX)) return false;
  if (c->capacity > 0 && (!c->z || !c->r || !c->label || !c->norm2)) return false;
  if ((reinterpret_cast<uintptr_t>(c->z) & 15u) != 0) return false;
  if ((reinterpret_cast<uintptr_t>(c->zimg) & 15u) != 0) return false;
  return true;
}

// Filter constants of one lookup (depend on precision, store and d) and
// the kernel plans of a slice scan and of a work-list scan.
struct FilterConsts {
  Plan pl;
  Plan pl_list;    // work-list scan: 4-wave blocks (short cluster lists)
  Plan pl_list8;   // work-list scan: 8-wave blocks (long cluster lists)
  Thresholds t;
  bool prune = false;  // pruned slice scan (prefix thresholds tp)
  Thresholds tp;
};

// Precision argument: the filter precision, optionally | LIPCACHE_LOOKUP_PRUNE.
inline int32_t filter_precision(int32_t precision) { return precision & ~LIPCACHE_LOOKUP_PRUNE; }
inline bool wants_prune(int32_t precision) { return (precision & LIPCACHE_LOOKUP_PRUNE) != 0; }

lipcache_status lookup_consts(const lipcache_cache* c, int32_t precision, FilterConsts& fc) {
  if (!make_plan(precision, c, false, fc.pl) || !make_plan(precision, c, true, fc.pl_list) ||
      !make_plan(precision, c, true, fc.pl_list8, kDmaWaves))
    return LIPCACHE_EUNSUPPORTED;
  if (precision == LIPCACHE_F32 && (fc.pl.ks > 32 || c->d > 512)) return LIPCACHE_EUNSUPPORTED;
  const FilterSlack fs = filter_slack(precision, c->store_dtype, fc.pl.d_pad);
  const double u32 = 1.0 / 16777216.0;
  fc.t.kq = 1.0 - fs.kappa;
  fc.t.kappa_c = 1.0 - fs.kappa - 4.0 * u32;
  fc.t.eta1 = fs.eta1;
  fc.t.eta0 = fs.eta0;
  fc.t.range2 = fs.range2;
  return LIPCACHE_OK;
}

// The pruned scan runs where the slice kernel is the float16 DMA kernel with
// at least two k-steps, on caches of at least kPruneMinRows rows (fewer fill
// too few 1024-row prefix tiles to pay for the prefix thresholds); elsewhere
// the option changes nothing.
constexpr int64_t kPruneMinRows = 32 * kPrRows;

void prune_consts(const lipcache_cache* c, int32_t precision, FilterConsts& fc) {
  fc.prune = precision == LIPCACHE_F16 && fc.pl.dma && fc.pl.ks >= 2 && fc.pl.ks <= 16 && c->n >= kPruneMinRows;
  if (!fc.prune) return;
  const FilterSlack fs = filter_slack(precision, c->store_dtype, kPrefixDims);
  const double u32 = 1.0 / 16777216.0;
  // The prefix accumulation starts at -Q'_q, which adds gam |Q'_q| to its
  // rounding error (gam for the kPrefixDims products and the start value):
  // Q'_q = RD((1 - kappa - gam) s / 2 - (1 + 2 gam)(eta1 sqrt(s) + eta0))
  // keeps every pair the unfolded test would pass, for either sign of Q'_q.
  const double n = static_cast<double>(kPrefixDims) + 2.0;
  const double gam = n * u32 / (1.0 - n * u32);
  fc.tp.kq = 1.0 - fs.kappa - gam;
  fc.tp.kappa_c = 1.0 - fs.kappa - 4.0 * u32;
  fc.tp.eta1 = fs.eta1 * (1.0 + 2.0 * gam);
  fc.tp.eta0 = fs.eta0 * (1.0 + 2.0 * gam);
  fc.tp.range2 = fs.range2;
}

// Stage 1: Q_q, and the reset of best / band flags / counters; with `view`
// also the thresholds A_i of its rows and the emptying of the re-check queue
// of the scan that follows (in the same launch); with qnorm / zq16 also
// ||q||^2 and the float16 copy of the queries (the indexed lookup's plan).
lipcache_status lookup_stage_prep(const float* zq, int64_t B, int d, const FilterConsts& fc, float* qthr,
                                  unsigned long long* best, unsigned int* bflag, unsigned long long* stats,
                                  hipStream_t s, const lipcache_cache* view = nullptr, float* athr = nullptr,
                                  unsigned long long* gq_count = nullptr, double* qnorm = nullptr,
                                  uint16_t* zq16 = nullptr, float* qthr_p = nullptr, float* athr_p = nullptr) {
  const int64_t qblocks = B > 0 ? (B + kLkWaves - 1) / kLkWaves : 1;
  PrepEntries pe{nullptr, nullptr, 0, 0, nullptr, nullptr, qnorm, zq16, nullptr, nullptr, 0, nullptr, 0, fc.tp};
  int64_t eblocks = 0;
  if (view && view->n > 0) {
    const bool pr = qthr_p && athr_p;
    pe = PrepEntries{view->r, view->norm2, view->n, athr_len(view->n), athr, gq_count, qnorm, zq16,
                     pr ? qthr_p : nullptr, pr ? athr_p : nullptr, pr ? athp_len(view->n) : 0, view->z,
                     view->store_dtype, fc.tp};
    const int64_t cover = pe.np_pad > pe.n_pad ? pe.np_pad : pe.n_pad;
    eblocks = (cover + kLkThreads - 1) / kLkThreads;
  }
  if (qblocks + eblocks > INT_MAX) return LIPCACHE_EUNSUPPORTED;
  hipLaunchKernelGGL(lookup_prep_kernel, dim3(static_cast<unsigned>(qblocks + eblocks)), dim3(kLkThreads), 0, s, zq,
                     B, d, fc.t, qthr, best, bflag, stats, static_cast<unsigned>(qblocks), pe);
  LC_LAUNCHED();
  return LIPCACHE_OK;
}

// Stage 2: the filter kernel of `view` (its n rows) against the B queries,
// over cache slices or, with `items`, over a work list of n_items (query
// positions, row range) items whose positions index qlist; then the
// chip-wide re-check of the pairs it queued in `gq`.  Hits are keyed by
// (emap ? emap[e] : e) + eoff.  athr needs athr_len(view->n) floats.
lipcache_status lookup_stage_scan(const lipcache_cache* view, int32_t precision, const FilterConsts& fc,
                                  const float* zq, int64_t B, const float* qthr, unsigned long long* best,
                                  unsigned int* bflag, unsigned long long* stats, float* athr,
                                  const int64_t* items, int64_t n_items, const int32_t* qlist, const uint16_t* zq16,
                                  const int64_t* emap, int64_t eoff, bool dump, float* g_hat, uint8_t* cand,
                                  const GlobalRecheckWs& gq, hipStream_t s, bool athr_ready = false,
                                  const float* qthr_p = nullptr, const float* athr_p = nullptr) {
  if (B <= 0 || view->n <= 0) return LIPCACHE_OK;
  if (items && n_items <= 0) return LIPCACHE_OK;
  if (!athr_ready) {
    const int64_t n_pad = athr_len(view->n);
    hipLaunchKernelGGL(lookup_athr_kernel, dim3(static_cast<unsigned>((n_pad + 255) / 256)), dim3(256), 0, s,
                       view->r, view->norm2, view->n, n_pad, fc.t.kappa_c, fc.t.eta1, fc.t.range2, athr,
                       dump ? nullptr : gq.count);
    LC_LAUNCHED();
  }
  const Plan& pl = items ? fc.pl_list : fc.pl;
  LookupParams p;
  p.zq = zq;
  p.B = B;
  p.cz = view->z;
  p.cr = view->r;
  p.cnorm2 = view->norm2;
  p.n = view->n;
  p.d = view->d;
  p.qthr = qthr;
  p.best = best;
  p.bflag = bflag;
  p.stats = stats;
  p.kappa_c = fc.t.kappa_c;
  p.eta1 = fc.t.eta1;
  p.range2 = fc.t.range2;
  p.athr = athr;
  p.qthr_p = qthr_p;
  p.athr_p = athr_p;
  p.cimg = precision == LIPCACHE_F16 ? view->zimg : view->z;
  p.n_qblocks = static_cast<int>((B + pl.qblock - 1) / pl.qblock);
  p.g_hat = g_hat;
  p.cand = cand;
  p.items = items;
  p.qlist = qlist;
  p.zq16 = zq16;
  p.emap = emap;
  p.eoff = eoff;
  p.gq_pos = dump ? nullptr : gq.pos;
  p.gq_e = dump ? nullptr : gq.e;
  p.gq_count = dump ? nullptr : gq.count;
  p.gq_cap = dump ? 0 : gq.cap;
  int64_t grid = n_items;
  p.slice_len = 0;
  const bool prune = qthr_p && athr_p && !items && !dump;
  if (!items) {
    // Cache slices: a multiple of 8 (one set per XCD), enough blocks to fill
    // the chip (~kGridTarget), but at least 4 tiles per slice.
    const int64_t tile_rows = prune ? kPrRows : pl.tile_rows;
    const int64_t tiles = (view->n + tile_rows - 1) / tile_rows;
    int64_t s8 = (kGridTarget + kXcds * p.n_qblocks - 1) / (kXcds * static_cast<int64_t>(p.n_qblocks));
    int64_t s8_max = tiles / (kXcds * 4);
    if (s8_max < 1) s8_max = 1;
    if (s8 > s8_max) s8 = s8_max;
    if (s8 < 1) s8 = 1;
    const int64_t slices = kXcds * s8;
    p.slice_len = ((tiles + slices - 1) / slices) * tile_rows;
    grid = slices * p.n_qblocks;
  }
  if (grid > INT_MAX) return LIPCACHE_EUNSUPPORTED;
  const unsigned gu = static_cast<unsigned>(grid);
  const hipError_t e = dump    ? launch_lookup<kVarDump>(precision, view->store_dtype, pl, p, gu, s)
                       : items ? (pl.waves == kListWaves ? launch_lookup<kVarList>(precision, view->store_dtype, pl, p, gu, s)
                                                         : launch_lookup<kVarList8>(precision, view->store_dtype, pl, p, gu, s))
                       : prune ? launch_prune(view->store_dtype, pl, p, gu, s)
                               : launch_lookup<kVarLookup>(precision, view->store_dtype, pl, p, gu, s);
  if (e != hipSuccess) return LIPCACHE_EHIP;
  if (dump) return LIPCACHE_OK;
  // the pairs the scan's waves queued, one chip-wide pass
  const RecheckArgs ra{zq, view->z, view->r, best, bflag, stats, static_cast<int64_t>(LLONG_MAX), view->n, view->d,
                       emap, eoff, qlist};
  int64_t blocks = (gq.cap + 15) / 16;
  if (blocks > 512) blocks = 512;
  if (view->store_dtype == LIPCACHE_BF16) {
    hipLaunchKernelGGL(recheck_queue_kernel<LIPCACHE_BF16>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, ra,
                       gq.pos, gq.e, gq.count, gq.cap);
  } else {
    hipLaunchKernelGGL(recheck_queue_kernel<LIPCACHE_F32>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, ra,
                       gq.pos, gq.e, gq.count, gq.cap);
  }
  LC_LAUNCHED();
  return LIPCACHE_OK;
}

// Stage 3: per query, label / index / d^2 / band flag, and the hit and band
// counts.
lipcache_status lookup_stage_finalize(int64_t B, const unsigned long long* best, const unsigned int* bflag,
                                      const int32_t* clabel, int32_t* label_out, int64_t* index_out,
                                      float* dist2_out, uint8_t* band_flag, unsigned long long* stats,
                                      hipStream_t s) {
  if (B <= 0) return LIPCACHE_OK;
  hipLaunchKernelGGL(lookup_finalize_kernel, dim3(static_cast<unsigned>((B + 255) / 256)), dim3(256), 0, s, B, best,
                     bflag, clabel, label_out, index_out, dist2_out, band_flag, stats);
  LC_LAUNCHED();
  return LIPCACHE_OK;
}

inline bool precision_ok(int32_t precision) { return precision == LIPCACHE_F16 || precision == LIPCACHE_F32; }

// Host-side validation shared by the lookup entry points (nothing launched).
lipcache_status lookup_check(const lipcache_cache* c, const float* zq, int64_t B, int32_t precision, bool dump,
                             const int32_t* label_out, const float* g_hat, const uint8_t* cand) {
  if (!cache_ok(c) || B < 0) return LIPCACHE_EINVAL;
  if (!precision_ok(precision)) return LIPCACHE_EINVAL;
  if (B > 0 && (!zq || (!dump && !label_out))) return LIPCACHE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(zq) & 15u) != 0) return LIPCACHE_EINVAL;
  if (B > static_cast<int64_t>(INT_MAX) / 2) return LIPCACHE_EINVAL;
  if (dump && (!g_hat || !cand || B * c->n > (1ll << 26))) return LIPCACHE_EINVAL;
  return LIPCACHE_OK;
}

// The whole lookup on a workspace laid out by ws_layout(B, c->n).
lipcache_status lookup_on(const lipcache_cache* c, const float* zq, int64_t B, int32_t precision,
                          const FilterConsts& fc, int32_t* label_out, int64_t* index_out, float* dist2_out,
                          uint64_t* stats, uint8_t* band_flag, void* ws, hipStream_t s, bool dump, float* g_hat,
                          uint8_t* cand) {
  Workspace w;
  ws_layout(B, c->n, &w, ws, fc.prune);
  unsigned long long* st = stats ? reinterpret_cast<unsigned long long*>(stats) : w.stats;
  lipcache_status r = lookup_stage_prep(zq, B, c->d, fc, w.qthr, w.best, w.bflag, st, s, c, w.athr,
                                       dump ? nullptr : w.gq.count, nullptr, nullptr, w.qthr_p, w.athr_p);
  if (r != LIPCACHE_OK) return r;
  r = lookup_stage_scan(c, precision, fc, zq, B, w.qthr, w.best, w.bflag, st, w.athr, nullptr, 0, nullptr, nullptr,
                        nullptr, 0, dump, g_hat, cand, w.gq, s, true, w.qthr_p, w.athr_p);
  if (r != LIPCACHE_OK) return r;
  if (dump) return LIPCACHE_OK;
  return lookup_stage_finalize(B, w.best, w.bflag, c->label, label_out, index_out, dist2_out, band_flag, st, s);
}

lipcache_status run_lookup(const lipcache_cache* c, const float* zq, int64_t B, int32_t precision_arg,
                           int32_t* label_out, int64_t* index_out, float* dist2_out, uint64_t* stats,
                           uint8_t* band_flag, void* ws, size_t ws_bytes, hipStream_t s, bool dump,
                           float* g_hat, uint8_t* cand) {
  const int32_t precision = filter_precision(precision_arg);
  if (dump && wants_prune(precision_arg)) return LIPCACHE_EINVAL;
  const lipcache_status vs = lookup_check(c, zq, B, precision, dump, label_out, g_hat, cand);
  if (vs != LIPCACHE_OK) return vs;
  FilterConsts fc;
  const lipcache_status cs = lookup_consts(c, precision, fc);
  if (cs != LIPCACHE_OK) return cs;
  if (wants_prune(precision_arg)) prune_consts(c, precision, fc);
  const size_t need = ws_layout(B, c->n, nullptr, nullptr, wants_prune(precision_arg));
  if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;
  return lookup_on(c, zq, B, precision, fc, label_out, index_out, dist2_out, stats, band_flag, ws, s, dump, g_hat,
                   cand);
}

// Workspace of an indexed lookup: the dense lookup's buffers (thresholds
// sized for the larger of the indexed part and the tail), the plan's, then
// the float16 copy of the queries.
struct IndexedTail {
  size_t q16, total;
};

inline IndexedTail indexed_ws_layout(int64_t B, int64_t n, int d, int K, int64_t n_indexed, Workspace* w,
                                     IndexPlanWs* pw, void* base) {
  const int64_t tail = n - n_indexed;
  const size_t lk = ws_layout(B, n_indexed > tail ? n_indexed : tail, w, base);
  char* pb = base ? static_cast<char*>(base) + lk : nullptr;
  IndexedTail t;
  t.q16 = lk + index_plan_layout(B, d, K, n_indexed, kLkWaves * 16, pw, pb);
  t.total = t.q16 + align_up(static_cast<size_t>(B) * d * 2, 256);
  return t;
}

lipcache_status run_lookup_indexed(const lipcache_cache* c, const lipcache_index* idx, const float* zq, int64_t B,
                                   int32_t precision, int32_t* label_out, int64_t* index_out, float* dist2_out,
                                   uint64_t* stats, uint8_t* band_flag, int64_t* pairs, void* ws, size_t ws_bytes,
                                   hipStream_t s) {
  if (!cache_ok(c) || !idx || B < 0) return LIPCACHE_EINVAL;
  if (!precision_ok(precision)) return LIPCACHE_EINVAL;
  if (B > 0 && (!zq || !label_out)) return LIPCACHE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(zq) & 15u) != 0) return LIPCACHE_EINVAL;
  if (B > static_cast<int64_t>(INT_MAX) / 2) return LIPCACHE_EINVAL;
  const lipcache_cache& so = idx->sorted;
  if (idx->K < 1 || idx->K > 65536 || idx->n_indexed < 1 || idx->n_indexed > c->n) return LIPCACHE_EINVAL;
  if (so.n != idx->n_indexed || so.d != c->d || so.store_dtype != c->store_dtype || !cache_ok(&so))
    return LIPCACHE_EINVAL;
  if (!idx->perm || !idx->offsets || !idx->centers || !idx->bound) return LIPCACHE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(idx->centers) & 15u) != 0) return LIPCACHE_EINVAL;
  // the float16 filter streams the images when the cache has one
  if (precision == LIPCACHE_F16 && (c->zimg == nullptr) != (so.zimg == nullptr)) return LIPCACHE_EINVAL;
  FilterConsts fc;
  const lipcache_status cs = lookup_consts(c, precision, fc);
  if (cs != LIPCACHE_OK) return cs;
  const size_t need = indexed_ws_layout(B, c->n, c->d, idx->K, idx->n_indexed, nullptr, nullptr, nullptr).total;
  if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;
  Workspace w;
  IndexPlanWs pw;
  const IndexedTail tl = indexed_ws_layout(B, c->n, c->d, idx->K, idx->n_indexed, &w, &pw, ws);
  char* wsb = static_cast<char*>(ws);
  unsigned long long* st = stats ? reinterpret_cast<unsigned long long*>(stats) : w.stats;
  if (B == 0) {
    lipcache_status r = lookup_stage_prep(zq, 0, c->d, fc, w.qthr, w.best, w.bflag, st, s);
    if (r == LIPCACHE_OK && pairs) *pairs = 0;
    return r;
  }
  // one pass over the queries: Q_q and the per-query state, ||q||^2 and the
  // float16 copy for the plan (and the float16 scan), and A_i of the sorted rows
  uint16_t* zq16 = reinterpret_cast<uint16_t*>(wsb + tl.q16);
  lipcache_status r =
      lookup_stage_prep(zq, B, c->d, fc, w.qthr, w.best, w.bflag, st, s, &so, w.athr, w.gq.count, pw.qnorm, zq16);
  if (r != LIPCACHE_OK) return r;
  int64_t n_items = 0, idx_pairs = 0;
  bool long_items = false;
  r = index_query_plan(idx, zq16, B, c->d, fc.pl_list.qblock, fc.pl_list8.qblock, pw, n_items, idx_pairs, long_items,
                       s);
  if (r != LIPCACHE_OK) return r;
  // Long lists (most items full) run 8-wave blocks sharing 128-row tiles
  // (the slice scan's shape, half the tile bytes per pair), short lists
  // 4-wave blocks, two per CU.
  FilterConsts fl = fc;
  if (long_items) fl.pl_list = fc.pl_list8;
  r = lookup_stage_scan(&so, precision, fl, zq, B, w.qthr, w.best, w.bflag, st, w.athr, pw.items, n_items, pw.qlist,
                        precision == LIPCACHE_F16 ? zq16 : nullptr, idx->perm, 0, false, nullptr, nullptr, w.gq, s,
                        true);
  if (r != LIPCACHE_OK) return r;
  const int64_t tail = c->n - idx->n_indexed;
  if (tail > 0) {
    // rows appended after the build: a dense scan of the cache's tail
    lipcache_cache view = *c;
    const size_t esz = c->store_dtype == LIPCACHE_BF16 ? 2 : 4;
    const size_t off = static_cast<size_t>(idx->n_indexed) * c->d;
    view.z = static_cast<char*>(c->z) + off * esz;
    view.zimg = c->zimg ? static_cast<char*>(c->zimg) + off * 2 : nullptr;
    view.r = c->r + idx->n_indexed;
    view.label = c->label + idx->n_indexed;
    view.norm2 = c->norm2 + idx->n_indexed;
    view.n = tail;
    view.capacity = tail;
    r = lookup_stage_scan(&view, precision, fc, zq, B, w.qthr, w.best, w.bflag, st, w.athr, nullptr, 0, nullptr,
                          nullptr, nullptr, idx->n_indexed, false, nullptr, nullptr, w.gq, s);
    if (r != LIPCACHE_OK) return r;
  }
  if (pairs) *pairs = idx_pairs + B * tail;
  return lookup_stage_finalize(B, w.best, w.bflag, c->label, label_out, index_out, dist2_out, band_flag, st, s);
}

// ------------------------------------------------------------- allocation-free entry
// The workspace of lipcache_lookup_noalloc: one file-scope device array per
// GPU, held until the process ends.  Host code never uses the array's name
// as an address: hipGetSymbolAddress gives each device's own copy, looked up
// once per device (with that device current) and kept in scratch_ptr.
constexpr size_t kNoAllocBytes = LIPCACHE_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
static std::mutex scratch_mutex;
static void* scratch_ptr[kMaxDevices];

// This device's copy of `scratch`, or nullptr if it cannot be had.
void* device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p || !aligned256(p)) return nullptr;
    scratch_ptr[dev] = p;
  }
  return scratch_ptr[dev];
}

}  // namespace lc

using namespace lc;

extern "C" size_t lipcache_lookup_indexed_workspace_bytes(int64_t B, int64_t n, int32_t d, int32_t K,
                                                          int64_t n_indexed) {
  if (B < 0 || n < 1 || d < 1 || K < 1 || n_indexed < 1 || n_indexed > n) return 0;
  return indexed_ws_layout(B, n, d, K, n_indexed, nullptr, nullptr, nullptr).total;
}

extern "C" lipcache_status lipcache_lookup_indexed(const lipcache_cache* c, const lipcache_index* idx,
                                                   const float* zq, int64_t B, int32_t precision,
                                                   int32_t* label_out, int64_t* index_out, float* dist2_out,
                                                   uint64_t* stats, uint8_t* band_flag, int64_t* pairs, void* ws,
                                                   size_t ws_bytes, lipcache_stream_t stream) {
  return run_lookup_indexed(c, idx, zq, B, precision, label_out, index_out, dist2_out, stats, band_flag, pairs, ws,
                            ws_bytes, reinterpret_cast<hipStream_t>(stream));
}

extern "C" int32_t lipcache_lookup_prunes(const lipcache_cache* c, int32_t precision_arg) {
  if (!wants_prune(precision_arg) || !cache_ok(c)) return 0;
  const int32_t precision = filter_precision(precision_arg);
  if (!precision_ok(precision)) return 0;
  FilterConsts fc;
  if (lookup_consts(c, precision, fc) != LIPCACHE_OK) return 0;
  prune_consts(c, precision, fc);
  return fc.prune ? 1 : 0;
}

extern "C" size_t lipcache_lookup_workspace_bytes(int64_t B, int64_t N, int32_t d, int32_t precision) {
  (void)d;
  return ws_layout(B, N, nullptr, nullptr, wants_prune(precision));
}

extern "C" lipcache_status lipcache_lookup(const lipcache_cache* c, const float* zq, int64_t B, int32_t precision,
                                           int32_t* label_out, int64_t* index_out, float* dist2_out,
                                           uint64_t* stats, uint8_t* band_flag, void* ws, size_t ws_bytes,
                                           lipcache_stream_t stream) {
  return run_lookup(c, zq, B, precision, label_out, index_out, dist2_out, stats, band_flag, ws, ws_bytes,
                    reinterpret_cast<hipStream_t>(stream), false, nullptr, nullptr);
}

extern "C" lipcache_status lipcache_lookup_filter_dump(const lipcache_cache* c, const float* zq, int64_t B,
                                                       int32_t precision, float* g_hat, uint8_t* cand, void* ws,
                                                       size_t ws_bytes, lipcache_stream_t stream) {
  return run_lookup(c, zq, B, precision, nullptr, nullptr, nullptr, nullptr, nullptr, ws, ws_bytes,
                    reinterpret_cast<hipStream_t>(stream), true, g_hat, cand);
}

extern "C" lipcache_status lipcache_lookup_noalloc(const lipcache_cache* c, const float* zq, int64_t B,
                                                   int32_t precision_arg, int32_t* label_out, int64_t* index_out,
                                                   float* dist2_out, uint64_t* stats, uint8_t* band_flag,
                                                   lipcache_stream_t stream) {
  const int32_t precision = filter_precision(precision_arg);
  const lipcache_status vs = lookup_check(c, zq, B, precision, false, label_out, nullptr, nullptr);
  if (vs != LIPCACHE_OK) return vs;
  FilterConsts fc;
  const lipcache_status cs = lookup_consts(c, precision, fc);
  if (cs != LIPCACHE_OK) return cs;
  if (wants_prune(precision_arg)) prune_consts(c, precision, fc);
  if (ws_layout(B, c->n, nullptr, nullptr, wants_prune(precision_arg)) > kNoAllocBytes) return LIPCACHE_EWORKSPACE;
  void* ws = device_scratch();
  if (!ws) return LIPCACHE_EHIP;
  return lookup_on(c, zq, B, precision, fc, label_out, index_out, dist2_out, stats, band_flag, ws,
                   reinterpret_cast<hipStream_t>(stream), false, nullptr, nullptr);
}
