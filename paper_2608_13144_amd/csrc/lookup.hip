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
//   Q_q = RD((1 - k) ||q||^2 / 2),  A_i = RD(((1 - k - 4u) ||z_i||^2 - r_i^2) / 2),
// where k bounds |g_hat - q.z_i| / ((||q||^2 + ||z_i||^2) / 2) (bf16 operand
// rounding and float32 accumulation, doubled).  Every true hit passes; a pair
// that passes is re-checked as sum_k (q_k - z_ik)^2 in float64 from the
// original values, which decides the hit.  Hits are merged per query with a
// 64-bit atomic minimum of (float bits of d^2) << 32 | i, which orders by
// distance and then by index, independent of scheduling.
//
// Kernel layout (gfx950, wave64):
//  - workgroup = 4 waves; wave w holds RT*16 queries as MFMA A operands in
//    registers for the whole sweep (bf16 or float32, converted once);
//  - the workgroup streams its slice of the cache through LDS in tiles of 64
//    entries (converted to the MFMA element type on the way in; rows padded
//    by 16 bytes so the B-operand reads are free of bank conflicts);
//  - per 16-entry column tile: KS k-steps of v_mfma_f32_16x16x32_bf16 (or 4x
//    v_mfma_f32_16x16x4_f32), then the one-subtract-one-compare filter on the
//    accumulators; a wave ballot skips the re-check path unless a pair passed;
//  - grid = query blocks x cache slices; blocks are numbered so that the
//    blocks a given XCD runs (block id mod 8) share cache slices, so the 64
//    resident workgroups of an XCD read each cache tile from its L2 at about
//    the same time.
#include <limits.h>

#include "lc_common.hpp"

namespace lc {

constexpr int kLkThreads = 256;
constexpr int kLkWaves = kLkThreads / kWave;
constexpr int kTileN = 64;
constexpr int kColTile = 16;
constexpr int kXcds = 8;
constexpr unsigned long long kNoHit = ~0ull;

enum { kModeBF16 = 0, kModeF32 = 1 };

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
  int n_qblocks;
  int64_t slice_len;
  float* g_hat;          // dump mode only
  uint8_t* cand;         // dump mode only
};

// ------------------------------------------------------------- prep
// One wave per query: Q_q, reset of the per-query state and of the counters.
__global__ void lookup_prep_kernel(const float* __restrict__ zq, int64_t B, int d, double kq,
                                   float* __restrict__ qthr, unsigned long long* __restrict__ best,
                                   unsigned int* __restrict__ bflag, unsigned long long* __restrict__ stats) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * kLkWaves + threadIdx.x / kWave;
  if (blockIdx.x == 0 && threadIdx.x < 4) stats[threadIdx.x] = 0;
  if (q >= B) return;
  const float* row = zq + q * d;
  double s = 0.0;
  for (int k = lane_id(); k < d; k += kWave) s = __builtin_fma(static_cast<double>(row[k]), static_cast<double>(row[k]), s);
  s = wave_sum(s);
  if (lane_id() == 0) {
    qthr[q] = f32_round_down(kq * s * 0.5 - 0.5 * kFilterAbsSlack);
    best[q] = kNoHit;
    bflag[q] = 0u;
  }
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
template <int MODE>
struct ModeTraits;
template <>
struct ModeTraits<kModeBF16> {
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
  if constexpr (MODE == kModeBF16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   acc, 0, 0, 0);
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
// operand chunk of the mode's element type; zeros beyond d.
template <int MODE, int SRC>
__device__ __forceinline__ u32x4 load_chunk(const void* base, int64_t row, int d, int k0) {
  u32x4 v = {0u, 0u, 0u, 0u};
  if (k0 >= d) return v;
  if constexpr (MODE == kModeBF16) {
    if constexpr (SRC == LIPCACHE_F32) {
      const f32x4* p = reinterpret_cast<const f32x4*>(static_cast<const float*>(base) + row * d + k0);
      const f32x4 x0 = p[0], x1 = p[1];
      const float f[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
      v = pack_bf16x8(f);
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

// Exact re-check of the pairs whose bits are set in `mask` (bit rt*4+i of a
// lane = accumulator i of row tile rt).  The whole wave evaluates one pair
// at a time: sum_k (q_k - z_ik)^2 in float64, lane-strided then a fixed
// butterfly, so the result does not depend on scheduling.
template <int SRC, int RT>
__device__ __noinline__ void recheck_pairs(const LookupParams& p, uint32_t mask, int64_t qwave, int64_t ebase) {
  const int lane = lane_id();
  while (true) {
    const unsigned long long bal = __ballot(mask != 0u);
    if (bal == 0ull) break;
    const int src = __builtin_ctzll(bal);
    const uint32_t msrc = static_cast<uint32_t>(__shfl(static_cast<int>(mask), src, kWave));
    const int bit = __builtin_ctz(msrc);
    if (lane == src) mask &= mask - 1u;
    const int rt = bit >> 2, i = bit & 3;
    const int64_t q = qwave + rt * 16 + 4 * (src >> 4) + i;
    const int64_t e = ebase + (src & 15);
    if (q >= p.B || e >= p.n) continue;  // padded rows never pass; kept as a guard
    const float* qr = p.zq + q * p.d;
    double part = 0.0;
    for (int k = lane; k < p.d; k += kWave) {
      const double diff = static_cast<double>(qr[k]) - cache_value<SRC>(p.cz, e, p.d, k);
      part = __builtin_fma(diff, diff, part);
    }
    const double d2 = wave_sum(part);
    if (lane == 0) {
      atomicAdd(&p.stats[LIPCACHE_STAT_RECHECKED], 1ull);
      const double r = static_cast<double>(p.cr[e]);
      const bool hit = d2 < r * r;
      if (__builtin_fabs(__builtin_sqrt(d2) - r) <= 1e-5 * r) {
        atomicAdd(&p.stats[LIPCACHE_STAT_BAND_PAIRS], 1ull);
        atomicOr(&p.bflag[q], 1u);
      }
      if (hit) {
        const float d2f = static_cast<float>(d2);
        const unsigned long long key =
            (static_cast<unsigned long long>(__builtin_bit_cast(uint32_t, d2f)) << 32) |
            static_cast<unsigned long long>(static_cast<uint32_t>(e));
        atomicMin(&p.best[q], key);
      }
    }
  }
}

template <int MODE, int SRC, int KS, int RT, bool DUMP>
__global__ __launch_bounds__(kLkThreads, 2) void lookup_kernel(const LookupParams p) {
  using T = ModeTraits<MODE>;
  constexpr int kDPad = KS * T::kPerStep;
  constexpr int kRowBytes = kDPad * T::kElemBytes + 16;   // +16: conflict-free B reads
  constexpr int kChunksPerRow = kDPad * T::kElemBytes / 16;
  __shared__ __attribute__((aligned(16))) unsigned char tile[kTileN * kRowBytes];
  __shared__ float athr[kTileN];

  // Block -> (query block, cache slice).  Consecutive blocks of one XCD
  // (same id mod 8) take consecutive query blocks of one slice.
  const int bid = static_cast<int>(blockIdx.x);
  const int xcd = bid % kXcds;
  const int local = bid / kXcds;
  const int slice = xcd + kXcds * (local / p.n_qblocks);
  const int qb = local % p.n_qblocks;

  const int lane = lane_id();
  const int wave = uniform(static_cast<int>(threadIdx.x) / kWave);
  const int m16 = lane & 15;
  const int g = lane >> 4;
  const int64_t qwave = static_cast<int64_t>(qb) * (kLkWaves * RT * 16) + wave * (RT * 16);

  // Queries as A operands: lane holds row m16 of each row tile, k-chunk g of
  // each k-step.  The same (k-step, chunk) -> k map is used for the cache
  // operand, so the contraction covers every k exactly once.
  u32x4 a[RT][KS];
  float qt[RT][4];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int64_t row = qwave + rt * 16 + m16;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      a[rt][ks] = row < p.B ? load_chunk<MODE, LIPCACHE_F32>(p.zq, row, p.d, ks * T::kPerStep + g * T::kPerChunk)
                            : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t qr = qwave + rt * 16 + 4 * g + i;
      qt[rt][i] = qr < p.B ? p.qthr[qr] : __builtin_inff();
    }
  }

  const int64_t e_begin = static_cast<int64_t>(slice) * p.slice_len;
  const int64_t e_end = e_begin + p.slice_len < p.n ? e_begin + p.slice_len : p.n;
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
      float at = __builtin_inff();
      if (e < e_end) {
        const float rr = p.cr[e];
        if (rr > 0.0f) {
          const double r2 = static_cast<double>(rr) * static_cast<double>(rr);
          at = f32_round_down((p.kappa_c * static_cast<double>(p.cnorm2[e]) - r2) * 0.5 - 0.5 * kFilterAbsSlack);
        }
      }
      athr[threadIdx.x] = at;
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
          recheck_pairs<SRC, RT>(p, mask, qwave, ebase);
        }
      }
    }
  }
}

// ------------------------------------------------------------- dispatch
struct Plan {
  int ks = 0;
  int rt = 0;
  int d_pad = 0;
  int qblock = 0;
};

inline bool make_plan(int precision, int d, Plan& pl) {
  const int per_step = precision == LIPCACHE_BF16 ? 32 : 16;
  const int max_ks = precision == LIPCACHE_BF16 ? 32 : 32;
  int ks = precision == LIPCACHE_BF16 ? 1 : 2;
  while (ks * per_step < d) ks *= 2;
  if (ks > max_ks) return false;
  pl.ks = ks;
  pl.rt = 32 / ks > 4 ? 4 : (32 / ks < 1 ? 1 : 32 / ks);
  pl.d_pad = ks * per_step;
  pl.qblock = kLkWaves * pl.rt * 16;
  return true;
}

template <int MODE, int SRC, int KS, int RT, bool DUMP>
hipError_t launch_one(const LookupParams& p, unsigned grid, hipStream_t s) {
  hipLaunchKernelGGL((lookup_kernel<MODE, SRC, KS, RT, DUMP>), dim3(grid), dim3(kLkThreads), 0, s, p);
  return hipGetLastError();
}

template <int MODE, int SRC, bool DUMP>
hipError_t launch_mode(const Plan& pl, const LookupParams& p, unsigned grid, hipStream_t s) {
  switch (pl.ks) {
    case 1: return launch_one<MODE, SRC, 1, 4, DUMP>(p, grid, s);
    case 2: return launch_one<MODE, SRC, 2, 4, DUMP>(p, grid, s);
    case 4: return launch_one<MODE, SRC, 4, 4, DUMP>(p, grid, s);
    case 8: return launch_one<MODE, SRC, 8, 4, DUMP>(p, grid, s);
    case 16: return launch_one<MODE, SRC, 16, 2, DUMP>(p, grid, s);
    case 32: return launch_one<MODE, SRC, 32, 1, DUMP>(p, grid, s);
    default: return hipErrorInvalidValue;
  }
}

struct Workspace {
  float* qthr;
  unsigned long long* best;
  unsigned int* bflag;
  unsigned long long* stats;
};

inline size_t ws_layout(int64_t B, Workspace* w, void* base) {
  const size_t nb = static_cast<size_t>(B > 0 ? B : 0);
  size_t off = 0;
  const size_t o_best = off;
  off = align_up(off + nb * 8, 256);
  const size_t o_qthr = off;
  off = align_up(off + nb * 4, 256);
  const size_t o_flag = off;
  off = align_up(off + nb * 4, 256);
  const size_t o_stats = off;
  off = align_up(off + 4 * 8, 256);
  if (w && base) {
    char* b = static_cast<char*>(base);
    w->best = reinterpret_cast<unsigned long long*>(b + o_best);
    w->qthr = reinterpret_cast<float*>(b + o_qthr);
    w->bflag = reinterpret_cast<unsigned int*>(b + o_flag);
    w->stats = reinterpret_cast<unsigned long long*>(b + o_stats);
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
  return true;
}

lipcache_status run_lookup(const lipcache_cache* c, const float* zq, int64_t B, int32_t precision,
                           int32_t* label_out, int64_t* index_out, float* dist2_out, uint64_t* stats,
                           uint8_t* band_flag, void* ws, size_t ws_bytes, hipStream_t s, bool dump,
                           float* g_hat, uint8_t* cand) {
  if (!cache_ok(c) || B < 0) return LIPCACHE_EINVAL;
  if (precision != LIPCACHE_BF16 && precision != LIPCACHE_F32) return LIPCACHE_EINVAL;
  if (B > 0 && (!zq || (!dump && !label_out))) return LIPCACHE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(zq) & 15u) != 0) return LIPCACHE_EINVAL;
  if (B > static_cast<int64_t>(INT_MAX) / 2) return LIPCACHE_EINVAL;
  if (dump && (!g_hat || !cand || B * c->n > (1ll << 26))) return LIPCACHE_EINVAL;
  Plan pl;
  if (!make_plan(precision, c->d, pl)) return LIPCACHE_EUNSUPPORTED;
  const size_t need = ws_layout(B, nullptr, nullptr);
  if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;
  Workspace w;
  ws_layout(B, &w, ws);
  unsigned long long* st = stats ? reinterpret_cast<unsigned long long*>(stats) : w.stats;

  const double kappa = filter_kappa(precision, c->store_dtype, pl.d_pad);
  const double u32 = 1.0 / 16777216.0;
  const unsigned prep_grid = static_cast<unsigned>(B > 0 ? (B + kLkWaves - 1) / kLkWaves : 1);
  hipLaunchKernelGGL(lookup_prep_kernel, dim3(prep_grid), dim3(kLkThreads), 0, s, zq, B, c->d, 1.0 - kappa,
                     w.qthr, w.best, w.bflag, st);
  LC_LAUNCHED();

  if (B > 0 && c->n > 0) {
    LookupParams p;
    p.zq = zq;
    p.B = B;
    p.cz = c->z;
    p.cr = c->r;
    p.cnorm2 = c->norm2;
    p.n = c->n;
    p.d = c->d;
    p.qthr = w.qthr;
    p.best = w.best;
    p.bflag = w.bflag;
    p.stats = st;
    p.kappa_c = 1.0 - kappa - 4.0 * u32;
    p.n_qblocks = static_cast<int>((B + pl.qblock - 1) / pl.qblock);
    p.g_hat = g_hat;
    p.cand = cand;
    // Cache slices: a multiple of 8 (one set per XCD), enough blocks to fill
    // the chip (~1024), but at least 4 tiles per slice.
    const int64_t tiles = (c->n + kTileN - 1) / kTileN;
    int64_t s8 = (1024 + kXcds * p.n_qblocks - 1) / (kXcds * static_cast<int64_t>(p.n_qblocks));
    int64_t s8_max = tiles / (kXcds * 4);
    if (s8_max < 1) s8_max = 1;
    if (s8 > s8_max) s8 = s8_max;
    if (s8 < 1) s8 = 1;
    const int64_t slices = kXcds * s8;
    p.slice_len = ((tiles + slices - 1) / slices) * kTileN;
    const int64_t grid = slices * p.n_qblocks;
    if (grid > INT_MAX) return LIPCACHE_EUNSUPPORTED;
    hipError_t e;
    const bool f32src = c->store_dtype == LIPCACHE_F32;
    if (precision == LIPCACHE_BF16) {
      if (dump)
        e = f32src ? launch_mode<kModeBF16, LIPCACHE_F32, true>(pl, p, static_cast<unsigned>(grid), s)
                   : launch_mode<kModeBF16, LIPCACHE_BF16, true>(pl, p, static_cast<unsigned>(grid), s);
      else
        e = f32src ? launch_mode<kModeBF16, LIPCACHE_F32, false>(pl, p, static_cast<unsigned>(grid), s)
                   : launch_mode<kModeBF16, LIPCACHE_BF16, false>(pl, p, static_cast<unsigned>(grid), s);
    } else {
      if (dump)
        e = f32src ? launch_mode<kModeF32, LIPCACHE_F32, true>(pl, p, static_cast<unsigned>(grid), s)
                   : launch_mode<kModeF32, LIPCACHE_BF16, true>(pl, p, static_cast<unsigned>(grid), s);
      else
        e = f32src ? launch_mode<kModeF32, LIPCACHE_F32, false>(pl, p, static_cast<unsigned>(grid), s)
                   : launch_mode<kModeF32, LIPCACHE_BF16, false>(pl, p, static_cast<unsigned>(grid), s);
    }
    if (e != hipSuccess) return LIPCACHE_EHIP;
  }
  if (!dump && B > 0) {
    hipLaunchKernelGGL(lookup_finalize_kernel, dim3(static_cast<unsigned>((B + 255) / 256)), dim3(256), 0, s, B,
                       w.best, w.bflag, c->label, label_out, index_out, dist2_out, band_flag, st);
    LC_LAUNCHED();
  }
  return LIPCACHE_OK;
}

}  // namespace lc

using namespace lc;

extern "C" size_t lipcache_lookup_workspace_bytes(int64_t B, int64_t N, int32_t d, int32_t precision) {
  (void)N;
  (void)d;
  (void)precision;
  return ws_layout(B, nullptr, nullptr);
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
