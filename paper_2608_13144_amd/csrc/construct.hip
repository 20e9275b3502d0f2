// Offline construction of the feature store (Sec. 4.3, Alg. 1).
//
// Candidates (z_i, payload y~_i, certified radius r_i) are eligible when
// r_i > 0 and, with the cache-centre label-consistency flag, when the guard
// label equals the payload.  At most `budget` entries are appended, at most
// `per_class` per payload label when that budget is set.  Strategies:
//
//   radius de-dup - visit eligible candidates by decreasing r (ties: lower
//                   index), skip a full class, skip a duplicate (strictly
//                   inside the ball of an entry already in the cache), append
//                   the rest.
//   priority      - the same visit by a caller-given priority (random keys
//                   give the random strategy), no duplicate test.
//   K-center      - farthest-first traversal from the largest-radius
//                   candidate, per class when a per-class budget is set.
//
// Device plan.  A stable LSD radix sort (four 8-bit passes over a 32-bit
// descending key; ties keep index order) orders the eligible candidates.
// The greedy visit then runs in chunks of kChunk candidates: the chunk is
// looked up against the cache (lipcache_lookup: a hit means a duplicate),
// an exact float64 relation "b lies in the ball of a" is formed for all
// pairs a < b of the chunk (bit matrix), one workgroup decides the chunk in
// order (64 candidates at a time where no relation row is set, else one by
// one with the AND of the relation row and the accepted bits; class counts in
// LDS), and lipcache_insert appends the accepted rows in visit order.
// K-center keeps every candidate's squared distance to the chosen set in
// float64.  With a per-class budget each class is traversed by one workgroup
// (candidates sorted by class), and the total budget is applied in class
// order afterwards; otherwise a fused update/arg-max kernel alternates with a
// one-block reduction, with no host round trip per pick.
#include <limits.h>

#include "lc_common.hpp"
#include "lc_sort.hpp"

namespace lc {

constexpr int kChunk = 1024;              // candidates per greedy step
constexpr int kChunkWords = kChunk / 32;  // relation row length in 32-bit words
constexpr int kMaxClasses = 16384;        // class counts live in LDS
constexpr uint32_t kNotEligible = 0xFFFFFFFFu;

__global__ void fill_u64_kernel(unsigned long long* __restrict__ p, int64_t n, unsigned long long v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Larger float -> smaller key (finite floats; order-preserving bit trick).
__device__ __forceinline__ uint32_t descending_key(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~u;
}

__device__ __forceinline__ bool eligible(int64_t i, const float* __restrict__ r, const float* __restrict__ prio,
                                         const int32_t* __restrict__ label, const int32_t* __restrict__ guard,
                                         int n_classes) {
  bool e = r[i] > 0.0f;
  if (guard) e = e && guard[i] == label[i];
  if (n_classes > 0) e = e && label[i] >= 0 && label[i] < n_classes;
  if (prio) e = e && prio[i] == prio[i];
  return e;
}

__global__ void construct_keys_kernel(const float* __restrict__ r, const float* __restrict__ prio,
                                      const int32_t* __restrict__ label, const int32_t* __restrict__ guard,
                                      int64_t n, int n_classes, uint32_t* __restrict__ keys,
                                      uint32_t* __restrict__ vals, unsigned long long* __restrict__ n_elig) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const bool e = i < n && eligible(i, r, prio, label, guard, n_classes);
  if (i < n) {
    keys[i] = e ? descending_key(prio ? prio[i] : r[i]) : kNotEligible;
    vals[i] = static_cast<uint32_t>(i);
  }
  const unsigned long long bal = __ballot(e);
  if (lane_id() == 0 && bal != 0ull) atomicAdd(n_elig, static_cast<unsigned long long>(__builtin_popcountll(bal)));
}

// The next chunk of the greedy visit: the first kChunk candidates, from
// position cursor[0] of the visit order on, whose class still has room
// (every candidate without a per-class budget).  A candidate of a full class
// would be skipped by the one-by-one visit without touching the accepted set,
// the class counts or the total, so leaving it out changes no decision.  One
// workgroup scans windows of kCompactPer x 1024 positions (thread t takes
// kCompactPer consecutive ones; a workgroup prefix sum of the per-thread
// counts places them); cursor[0] becomes the position after the last
// candidate taken (or the end), cursor[1] the chunk's size, cand[] its
// candidates in order.
constexpr int kCompactPer = 8;

__global__ __launch_bounds__(1024) void construct_compact_kernel(const uint32_t* __restrict__ order, int64_t n_elig,
                                                                 const int32_t* __restrict__ label,
                                                                 const int32_t* __restrict__ class_count,
                                                                 int per_class, unsigned long long* __restrict__ cursor,
                                                                 uint32_t* __restrict__ cand) {
  constexpr int kWaves = 1024 / kWave;
  constexpr int kWindow = 1024 * kCompactPer;
  __shared__ int wsum[kWaves];
  __shared__ int64_t s_cur;
  __shared__ int s_k;
  const int t = static_cast<int>(threadIdx.x);
  const int lane = lane_id(), wave = t / kWave;
  if (t == 0) {
    s_cur = static_cast<int64_t>(cursor[0]);
    s_k = 0;
  }
  __syncthreads();
  while (true) {
    const int64_t cur = s_cur;
    const int k = s_k;
    if (k >= kChunk || cur >= n_elig) break;  // uniform
    const int64_t p0 = cur + static_cast<int64_t>(t) * kCompactPer;
    uint32_t ci[kCompactPer];
    bool f[kCompactPer];
#pragma unroll
    for (int j = 0; j < kCompactPer; ++j) {
      f[j] = p0 + j < n_elig;
      ci[j] = f[j] ? order[p0 + j] : 0u;
    }
    if (per_class > 0) {
      int cl[kCompactPer];
#pragma unroll
      for (int j = 0; j < kCompactPer; ++j) cl[j] = f[j] ? label[ci[j]] : 0;
#pragma unroll
      for (int j = 0; j < kCompactPer; ++j) f[j] = f[j] && class_count[cl[j]] < per_class;
    }
    int mine = 0;
#pragma unroll
    for (int j = 0; j < kCompactPer; ++j) mine += f[j] ? 1 : 0;
    // inclusive prefix of the per-thread counts within the wave
    int incl = mine;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int o = __shfl_up(incl, off, kWave);
      if (lane >= off) incl += o;
    }
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    int before = 0, total = 0;
    for (int w = 0; w < kWaves; ++w) {
      before += w < wave ? wsum[w] : 0;
      total += wsum[w];
    }
    int r = k + before + incl - mine;  // chunk slot of this thread's first flagged candidate
    int64_t last_pos = -1;            // position of the candidate that fills the chunk, if this thread holds it
#pragma unroll
    for (int j = 0; j < kCompactPer; ++j) {
      if (f[j]) {
        if (r < kChunk) cand[r] = ci[j];
        if (r == kChunk - 1) last_pos = p0 + j;
        ++r;
      }
    }
    __syncthreads();  // s_cur, s_k and wsum are read; update them
    if (k + total <= kChunk) {
      if (t == 0) {
        s_k = k + total;
        s_cur = cur + kWindow < n_elig ? cur + kWindow : n_elig;
      }
    } else if (last_pos >= 0) {
      s_k = kChunk;
      s_cur = last_pos + 1;
    }
    __syncthreads();
  }
  if (t == 0) {
    cursor[0] = static_cast<unsigned long long>(s_cur);
    cursor[1] = static_cast<unsigned long long>(s_k);
  }
}

// Chunk rows in visit order: the stored values (bf16-rounded for a bf16
// cache) as float32, with their payload and radius.  One wave per row.
__global__ void construct_gather_kernel(const float* __restrict__ z, const int32_t* __restrict__ label,
                                        const float* __restrict__ r, const uint32_t* __restrict__ order, int k, int d,
                                        int bf16, float* __restrict__ zc, int32_t* __restrict__ lc,
                                        float* __restrict__ rc, int64_t* __restrict__ src_c) {
  const int j = static_cast<int>(blockIdx.x) * (blockDim.x / kWave) + static_cast<int>(threadIdx.x) / kWave;
  if (j >= k) return;
  const int64_t src = order[j];
  const float* zr = z + src * d;
  float* out = zc + static_cast<int64_t>(j) * d;
  for (int c = lane_id(); c < d; c += kWave) out[c] = bf16 ? bf16_round_f32(zr[c]) : zr[c];
  if (lane_id() == 0) {
    lc[j] = label[src];
    rc[j] = r[src];
    src_c[j] = src;
  }
}

// rel[b * kChunkWords + a / 32] bit a % 32 set iff a < b and
// ||z_b - z_a||^2 < r_a^2 (float64 over the chunk's stored values).  A block
// of 1024 threads takes a 32 x 32 tile of (b, a) pairs, rows staged in LDS
// 64 elements at a time; each wave covers two b rows, and one ballot per
// wave gives their two words.
__global__ __launch_bounds__(1024) void construct_relation_kernel(const float* __restrict__ zc,
                                                                  const float* __restrict__ rc, int k, int d,
                                                                  uint32_t* __restrict__ rel) {
  __shared__ float za[32][65];
  __shared__ float zb[32][65];
  const int tb = static_cast<int>(blockIdx.y);  // tile of b rows
  const int ta = static_cast<int>(blockIdx.x);  // tile of a rows
  const int t = static_cast<int>(threadIdx.x);
  const int bl = t / 32, al = t % 32;
  const int b = tb * 32 + bl, a = ta * 32 + al;
  bool inside = false;
  if (ta <= tb) {
    double acc = 0.0;
    for (int c0 = 0; c0 < d; c0 += 64) {
      __syncthreads();
      for (int e = t; e < 32 * 64; e += 1024) {
        const int row = e / 64, col = e % 64;
        const int ra = ta * 32 + row, rb = tb * 32 + row;
        const bool in_row = c0 + col < d;
        za[row][col] = (ra < k && in_row) ? zc[static_cast<int64_t>(ra) * d + c0 + col] : 0.0f;
        zb[row][col] = (rb < k && in_row) ? zc[static_cast<int64_t>(rb) * d + c0 + col] : 0.0f;
      }
      __syncthreads();
#pragma unroll 8
      for (int c = 0; c < 64; ++c) {
        const double diff = static_cast<double>(zb[bl][c]) - static_cast<double>(za[al][c]);
        acc = __builtin_fma(diff, diff, acc);
      }
    }
    if (a < b && b < k) {
      const double ra = static_cast<double>(rc[a]);
      inside = acc < ra * ra;
    }
  }
  const unsigned long long bal = __ballot(inside);
  const int lane = lane_id();
  if (b < k && (lane == 0 || lane == 32)) {
    const uint32_t word = lane == 0 ? static_cast<uint32_t>(bal) : static_cast<uint32_t>(bal >> 32);
    rel[static_cast<int64_t>(b) * kChunkWords + ta] = word;
  }
}

struct AcceptParams {
  int k;
  int dedup;
  const int32_t* dup_label;   // lookup result per chunk candidate (MISS = not inside a cached ball); may be null
  const uint32_t* rel;        // chunk relation; null without de-dup
  const int32_t* lc;          // payload labels of the chunk
  const int64_t* src_c;       // candidate index of each chunk row
  int32_t* sel;               // out: LIPCACHE_MISS = append, 0 = skip
  int32_t* class_count;       // [n_classes] running counts (global)
  int n_classes;
  int per_class;
  unsigned long long* total;  // running number appended
  unsigned long long budget;
  int64_t* selected_out;      // may be null
};

// One workgroup decides the chunk in visit order.  All threads stage the
// relation, the chunk's labels, the lookup verdicts, a per-row "has any
// relation bit" flag and the class counts in LDS; wave 0 then walks the
// chunk: lane l keeps bits 32 l .. 32 l + 31 of the accepted set, so
// "inside an accepted earlier ball" is one AND per lane and one ballot,
// needed only for rows that have a relation bit at all.
__global__ __launch_bounds__(1024) void construct_accept_kernel(const AcceptParams p) {
  __shared__ uint32_t srel[kChunk * kChunkWords];  // 128 KiB
  __shared__ int32_t scount[kMaxClasses / 16];      // the first 1024 classes; the rest from global
  __shared__ int32_t slab[kChunk];
  __shared__ uint8_t sfree[kChunk];                 // not inside a cached ball
  __shared__ uint8_t srow[kChunk];                  // relation row j has a bit
  const int t = static_cast<int>(threadIdx.x);
  if (p.dedup) {
    for (int e = t; e < p.k * kChunkWords; e += 1024) srel[e] = p.rel[e];
  }
  if (t < p.k) {
    slab[t] = p.lc[t];
    sfree[t] = p.dup_label ? (p.dup_label[t] == LIPCACHE_MISS ? 1 : 0) : 1;
  }
  const int cached = p.n_classes < kMaxClasses / 16 ? p.n_classes : kMaxClasses / 16;
  if (p.per_class > 0)
    for (int c = t; c < cached; c += 1024) scount[c] = p.class_count[c];
  __syncthreads();
  if (t < p.k) {
    uint32_t any = 0u;
    if (p.dedup) {
      const int words = (t + 31) / 32;  // only a < t can be set
      for (int w = 0; w < words; ++w) any |= srel[t * kChunkWords + w];
    }
    srow[t] = any != 0u ? 1 : 0;
  }
  __syncthreads();
  if (t >= kWave) return;
  const int lane = t;
  const unsigned long long lt = (1ull << lane) - 1ull;
  uint32_t acc_bits = 0u;  // lane's word of the accepted set (lanes >= kChunkWords stay 0)
  unsigned long long total = *p.total;
  // Windows of 64 candidates.  Without relation rows a window is decided at
  // once: the k-th free candidate of class c in the window passes its class
  // test iff count[c] + k < per_class, and the passers are taken in order up
  // to the total budget - exactly what the one-by-one visit does.  A window
  // with a relation row is walked one candidate at a time.
  for (int w0 = 0; w0 < p.k; w0 += kWave) {
    const int j = w0 + lane;
    const bool in = j < p.k;
    const int c = in ? slab[j] : 0;
    const bool fr = in && sfree[j] != 0;
    const bool rel = __ballot(in && srow[j] != 0) != 0ull;
    if (!rel) {
      bool pass = fr;
      unsigned long long same = 0ull;
      if (p.per_class > 0) {
        same = __ballot(fr);
#pragma unroll
        for (int b = 0; b < 14; ++b) {
          const bool bit = (c >> b) & 1;
          const unsigned long long bal = __ballot(bit);
          same &= bit ? bal : ~bal;
        }
        const int rank = __builtin_popcountll(same & lt);
        if (fr) {
          const int cnt = c < cached ? scount[c] : p.class_count[c];
          pass = cnt + rank < p.per_class;
        }
      }
      const unsigned long long pm = __ballot(pass);
      const unsigned long long grank = static_cast<unsigned long long>(__builtin_popcountll(pm & lt));
      const bool take = pass && total + grank < p.budget;
      const unsigned long long tm = __ballot(take);
      if (in) p.sel[j] = take ? LIPCACHE_MISS : 0;
      if (take && p.selected_out) p.selected_out[total + grank] = p.src_c[j];
      if (p.per_class > 0 && fr && __builtin_popcountll(same & lt) == 0) {
        const int add = __builtin_popcountll(same & tm);  // taken members of this lane's class group
        if (add) {
          if (c < cached) {
            scount[c] += add;
          } else {
            p.class_count[c] += add;
          }
        }
      }
      if (lane == (w0 >> 5)) acc_bits |= static_cast<uint32_t>(tm);
      if (lane == (w0 >> 5) + 1) acc_bits |= static_cast<uint32_t>(tm >> 32);
      total += static_cast<unsigned long long>(__builtin_popcountll(tm));
      continue;
    }
    const int jend = w0 + kWave < p.k ? w0 + kWave : p.k;
    for (int jj = w0; jj < jend; ++jj) {
      const int cj = slab[jj];
      bool take = total < p.budget && sfree[jj] != 0;
      if (take && p.per_class > 0) {
        const int cnt = cj < cached ? scount[cj] : p.class_count[cj];
        take = cnt < p.per_class;
      }
      if (take && srow[jj] != 0) {
        const uint32_t row = lane < kChunkWords ? srel[jj * kChunkWords + lane] : 0u;
        take = __ballot((row & acc_bits) != 0u) == 0ull;
      }
      if (lane == 0) p.sel[jj] = take ? LIPCACHE_MISS : 0;
      if (take) {
        if (lane == jj / 32) acc_bits |= 1u << (jj % 32);
        if (lane == 0) {
          if (p.per_class > 0) {
            if (cj < cached) {
              scount[cj] += 1;
            } else {
              p.class_count[cj] += 1;
            }
          }
          if (p.selected_out) p.selected_out[total] = p.src_c[jj];
        }
        total += 1;
      }
    }
  }
  if (lane == 0) *p.total = total;
  if (p.per_class > 0)
    for (int c = lane; c < cached; c += kWave) p.class_count[c] = scount[c];
}

// ---------------------------------------------------------------- K-center
struct KcParams {
  const float* z;
  const float* r;
  const float* prio;
  const int32_t* label;
  const int32_t* guard;
  int64_t n;
  int d;
  int bf16;
  int n_classes;
  int group;                 // -1: all eligible candidates, else this payload label
  double* mind;              // [n] squared distance to the chosen set; < 0: not a candidate
  int64_t* pick;             // [1] newest pick (-1: none)
  double* part_v;            // [blocks] block maxima
  int64_t* part_i;           // [blocks] their indices
  unsigned long long* total; // appended so far (all groups)
  unsigned long long budget;
  int64_t* picks;            // [budget] picks in order
  int* group_count;          // [1] picks in the current group
  int limit;                 // picks allowed in this group
};

__device__ __forceinline__ float stored(const KcParams& p, int64_t i, int c) {
  const float v = p.z[i * p.d + c];
  return p.bf16 ? bf16_round_f32(v) : v;
}

__device__ __forceinline__ double dist2(const KcParams& p, int64_t i, int64_t j) {
  double acc = 0.0;
  for (int c = 0; c < p.d; ++c) {
    const double diff = static_cast<double>(stored(p, i, c)) - static_cast<double>(stored(p, j, c));
    acc = __builtin_fma(diff, diff, acc);
  }
  return acc;
}

// Block arg-max of (v, -i): larger v, then lower index.
__device__ __forceinline__ void better(double& v, int64_t& i, double v2, int64_t i2) {
  if (v2 > v || (v2 == v && i2 >= 0 && (i < 0 || i2 < i))) {
    v = v2;
    i = i2;
  }
}

__device__ void block_argmax(double v, int64_t i, double* sv, int64_t* si, double& out_v, int64_t& out_i) {
  const int t = static_cast<int>(threadIdx.x);
  sv[t] = v;
  si[t] = i;
  __syncthreads();
  for (int s = static_cast<int>(blockDim.x) / 2; s > 0; s >>= 1) {
    if (t < s) {
      double a = sv[t];
      int64_t ai = si[t];
      better(a, ai, sv[t + s], si[t + s]);
      sv[t] = a;
      si[t] = ai;
    }
    __syncthreads();
  }
  out_v = sv[0];
  out_i = si[0];
}

// The group's start: its first candidate in visit order (largest r, lower
// index).  One block walks the order 256 positions at a time.
__global__ __launch_bounds__(256) void kcenter_start_kernel(const int32_t* __restrict__ label,
                                                            const uint32_t* __restrict__ order, int64_t n_elig,
                                                            int group, int64_t* __restrict__ start) {
  __shared__ unsigned long long best;
  if (threadIdx.x == 0) best = ~0ull;
  __syncthreads();
  for (int64_t base = 0; base < n_elig; base += 256) {
    const int64_t q = base + threadIdx.x;
    if (q < n_elig && (group < 0 || label[order[q]] == group)) atomicMin(&best, static_cast<unsigned long long>(q));
    __syncthreads();
    const bool found = best != ~0ull;
    __syncthreads();
    if (found) break;
  }
  if (threadIdx.x == 0) *start = best != ~0ull ? static_cast<int64_t>(order[best]) : -1;
}

// First step of a group: mind = squared distance to the start.
__global__ __launch_bounds__(256) void kcenter_init_kernel(const KcParams p, const int64_t* __restrict__ start) {
  const int64_t s = *start;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < p.n) {
    const bool in = s >= 0 && eligible(i, p.r, p.prio, p.label, p.guard, p.n_classes) &&
                    (p.group < 0 || p.label[i] == p.group);
    p.mind[i] = (!in || i == s) ? -1.0 : dist2(p, i, s);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const bool ok = s >= 0 && *p.total < p.budget && p.limit > 0;
    *p.pick = ok ? s : -1;
    *p.group_count = ok ? 1 : 0;
    if (ok) {
      p.picks[*p.total] = s;
      *p.total += 1ull;
    }
  }
}

// Fold the newest pick into mind (unless it is -1), then block arg-max.
__global__ __launch_bounds__(256) void kcenter_step_kernel(const KcParams p) {
  __shared__ double sv[256];
  __shared__ int64_t si[256];
  const int64_t pk = *p.pick;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  double v = -1.0;
  int64_t vi = -1;
  if (i < p.n) {
    double m = p.mind[i];
    if (m >= 0.0 && pk >= 0) {
      if (i == pk) {
        m = -1.0;
      } else {
        const double d2 = dist2(p, i, pk);
        m = d2 < m ? d2 : m;
      }
      p.mind[i] = m;
    }
    if (m >= 0.0) {
      v = m;
      vi = i;
    }
  }
  double ov;
  int64_t oi;
  block_argmax(v, vi, sv, si, ov, oi);
  if (threadIdx.x == 0) {
    p.part_v[blockIdx.x] = ov;
    p.part_i[blockIdx.x] = oi;
  }
}

// Reduce the block maxima to the next pick.
__global__ __launch_bounds__(256) void kcenter_pick_kernel(const KcParams p, int nblocks) {
  __shared__ double sv[256];
  __shared__ int64_t si[256];
  double v = -1.0;
  int64_t vi = -1;
  for (int b = threadIdx.x; b < nblocks; b += 256) better(v, vi, p.part_v[b], p.part_i[b]);
  double ov;
  int64_t oi;
  block_argmax(v, vi, sv, si, ov, oi);
  if (threadIdx.x == 0) {
    const bool ok = oi >= 0 && ov >= 0.0 && *p.total < p.budget && *p.group_count < p.limit;
    *p.pick = ok ? oi : -1;
    if (ok) {
      p.picks[*p.total] = oi;
      *p.total += 1ull;
      *p.group_count += 1;
    }
  }
}

// ------------------------------------------------- per-class K-center
// With a per-class budget every class is traversed on its own, so the
// classes run side by side: their eligible candidates are sorted by class
// (stably, so each class list keeps the visit order and starts at its
// largest radius), one workgroup walks one class, and the total budget is
// applied afterwards in ascending class order (a traversal's first k picks
// do not depend on how many follow).

// keys / vals of the class sort: label and candidate of visit position q;
// class sizes counted per workgroup of 4096 positions in LDS (n_classes <=
// kMaxClasses), one atomic per class it saw.
__global__ __launch_bounds__(256) void class_keys_kernel(const int32_t* __restrict__ label,
                                                         const uint32_t* __restrict__ order, int64_t n_elig,
                                                         int n_classes, uint32_t* __restrict__ keys,
                                                         uint32_t* __restrict__ vals, uint32_t* __restrict__ ccount) {
  __shared__ uint32_t h[kMaxClasses];
  for (int c = threadIdx.x; c < n_classes; c += 256) h[c] = 0u;
  __syncthreads();
  const int64_t q0 = static_cast<int64_t>(blockIdx.x) * 4096;
  for (int64_t q = q0 + threadIdx.x; q < q0 + 4096 && q < n_elig; q += 256) {
    const uint32_t i = order[q];
    const uint32_t c = static_cast<uint32_t>(label[i]);  // in [0, n_classes): eligibility
    keys[q] = c;
    vals[q] = i;
    atomicAdd(&h[c], 1u);
  }
  __syncthreads();
  for (int c = threadIdx.x; c < n_classes; c += 256)
    if (h[c]) atomicAdd(&ccount[c], h[c]);
}

constexpr int kKcThreads = 1024;
constexpr int kKcPickLds = 2048;  // picks whose distances to the newest pick are kept (pruning)
constexpr int kKcWin = 4096;      // candidates per window of a pass

// Squared distances (float64 of the stored values) of R rows to the staged
// row prow, one 16-lane group per row set: lane lr of the group sums
// features 4 lr + 64 u + e of each row, then a fixed butterfly over the
// group.  All R x U loads are issued before the first sum.
template <int U, int R>
__device__ __forceinline__ void group_dist2(const float* __restrict__ z, int d, int bf16, const int64_t (&row)[R],
                                            const bool (&ok)[R], const float* prow, int lr, double (&out)[R]) {
  f32x4 v[R][U];
#pragma unroll
  for (int r = 0; r < R; ++r) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = 4 * lr + 64 * u;
      v[r][u] = (ok[r] && k < d) ? *reinterpret_cast<const f32x4*>(z + row[r] * d + k) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    double part = 0.0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = 4 * lr + 64 * u;
      if (k < d) {
        const f32x4 pv = *reinterpret_cast<const f32x4*>(prow + k);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float sv_ = bf16 ? bf16_round_f32(v[r][u][e]) : v[r][u][e];
          const double diff = static_cast<double>(sv_) - static_cast<double>(pv[e]);
          part = __builtin_fma(diff, diff, part);
        }
      }
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) part += __shfl_xor(part, off, kWave);
    out[r] = part;
  }
}

// Farthest-first traversal of class blockIdx.x over its list
// list[coff[c] .. coff[c + 1]): up to min(per_class, budget, size) picks into
// cpicks[coff[c] ..], their number into ccount[c].  mind[coff[c] + j] holds
// candidate j's squared distance to the chosen set (-1 once chosen) and
// own[coff[c] + j] the pick that set it.  A pass (one pick) takes the
// candidates in windows of kKcWin: every thread reads the distance and owner
// of its candidates of the window and lists in LDS those whose distance to
// the newest pick (staged in LDS) is needed; then each 16-lane group sums
// those distances in float64 over the stored values, R rows at a time with
// all their loads in flight.  The block arg-max takes the larger distance,
// then the lower candidate index.  U = row chunks of 64 features per lane
// (d <= 64 U); wide rows run 512 threads.
//
// Pruning (exact).  With a = own[j] and D the computed distance between pick
// a and the newest pick p, the triangle inequality gives ||z_j - p|| >= D -
// ||z_j - a||.  When D >= 2 sqrt(mind_j) (1 + 1e-9), that bound exceeds
// sqrt(mind_j) (1 + 1e-9 - 3 gamma), gamma <= 1024 * 2^-53 the relative
// error of a float64 sum of squares, so the computed squared distance would
// be above mind_j and the minimum would not change: the row is not read.
// The picks, the distances and the arg-max are those of the full update.
template <int U, int THREADS>
__global__ __launch_bounds__(THREADS) void kcenter_class_kernel(const float* __restrict__ z, int d, int bf16,
                                                                   const uint32_t* __restrict__ list,
                                                                   const int64_t* __restrict__ coff, int per_class,
                                                                   int64_t budget, double* __restrict__ mind,
                                                                   int32_t* __restrict__ own,
                                                                   int64_t* __restrict__ cpicks,
                                                                   uint32_t* __restrict__ ccount) {
  constexpr int R = U >= 8 ? 16 / U : 4;  // rows per group per step (R x U <= 16 chunks in flight)
  constexpr int kWaves = THREADS / kWave;
  constexpr int kGroups = 4 * kWaves;      // 16-lane groups of the block
  __shared__ __attribute__((aligned(16))) float prow[1024];
  __shared__ double dpp[kKcPickLds];       // distance of pick q to the newest pick
  __shared__ int32_t lj[kKcWin];           // the window's listed candidates: position,
  __shared__ uint32_t lc[kKcWin];          // candidate index
  __shared__ double lm[kKcWin];            // and current distance
  __shared__ int s_n;
  __shared__ double sv[kWaves];
  __shared__ int64_t si[kWaves];
  __shared__ int64_t s_pick;
  const int c = static_cast<int>(blockIdx.x);
  const int t = static_cast<int>(threadIdx.x);
  const int lane = lane_id(), wave = t / kWave;
  const int grp = lane >> 4, lr = lane & 15;
  const int gid = 4 * wave + grp;
  const int64_t j0 = coff[c];
  const int64_t nc = coff[c + 1] - j0;
  int64_t lim = per_class < nc ? per_class : nc;
  lim = budget < lim ? budget : lim;
  if (lim <= 0) {
    if (t == 0) ccount[c] = 0u;
    return;
  }
  int64_t pick = list[j0];
  if (t == 0) cpicks[j0] = pick;
  int64_t cnt = 1;
  for (int pass = 0; cnt < lim; ++pass) {
    __syncthreads();
    for (int k = t; k < d; k += THREADS) {
      const float v = z[pick * d + k];
      prow[k] = bf16 ? bf16_round_f32(v) : v;
    }
    __syncthreads();
    // distances of the earlier picks to the newest one (index cnt - 1)
    const int np = static_cast<int>(cnt - 1 < kKcPickLds ? cnt - 1 : kKcPickLds);
    for (int q0 = gid; q0 < np; q0 += kGroups * R) {
      int64_t row[R];
      bool ok[R];
      double dd[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int q = q0 + r * kGroups;
        ok[r] = q < np;
        row[r] = ok[r] ? cpicks[j0 + q] : 0;
      }
      group_dist2<U, R>(z, d, bf16, row, ok, prow, lr, dd);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int q = q0 + r * kGroups;
        if (ok[r] && lr == 0) dpp[q] = __builtin_sqrt(dd[r]);
      }
    }
    __syncthreads();
    const int32_t cur = static_cast<int32_t>(cnt - 1);
    double bv = -1.0;
    int64_t bi = -1;
    for (int64_t w0 = 0; w0 < nc; w0 += kKcWin) {
      const int wn = static_cast<int>(nc - w0 < kKcWin ? nc - w0 : kKcWin);
      if (t == 0) s_n = 0;
      __syncthreads();
      // phase 1: distances and owners of the window; list what must be
      // measured, take the rest into the arg-max as they are
      for (int i0 = 0; i0 < wn; i0 += THREADS) {
        const int i = i0 + t;
        const bool in = i < wn;
        const int64_t j = w0 + (in ? i : 0);
        const uint32_t cand = list[j0 + j];
        double m = pass == 0 ? __builtin_inf() : mind[j0 + j];
        const int32_t a = pass == 0 ? -1 : own[j0 + j];
        bool need = false;
        if (in && m >= 0.0) {
          if (static_cast<int64_t>(cand) == pick) {
            m = -1.0;
            mind[j0 + j] = m;
          } else {
            need = pass == 0 || a < 0 || a >= np || !(dpp[a] >= 2.0 * __builtin_sqrt(m) * (1.0 + 1e-9));
          }
        }
        const unsigned long long bal = __ballot(need);
        int base = 0;
        if (lane == 0 && bal) base = atomicAdd(&s_n, __builtin_popcountll(bal));
        base = __shfl(base, 0, kWave);
        if (need) {
          const int slot = base + __builtin_popcountll(bal & ((1ull << lane) - 1ull));
          lj[slot] = static_cast<int32_t>(i);
          lc[slot] = cand;
          lm[slot] = m;
        } else if (in) {
          better(bv, bi, m >= 0.0 ? m : -1.0, m >= 0.0 ? static_cast<int64_t>(cand) : -1);
        }
      }
      __syncthreads();
      const int nl = s_n;
      // phase 2: the listed candidates, R per group per step
      for (int s0 = gid; s0 < nl; s0 += kGroups * R) {
        int64_t row[R];
        bool ok[R];
        double dd[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const int sl = s0 + r * kGroups;
          ok[r] = sl < nl;
          row[r] = ok[r] ? static_cast<int64_t>(lc[sl]) : 0;
        }
        group_dist2<U, R>(z, d, bf16, row, ok, prow, lr, dd);
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const int sl = s0 + r * kGroups;
          if (!ok[r]) continue;
          double m = lm[sl];
          const int64_t j = w0 + lj[sl];
          if (dd[r] < m) {
            m = dd[r];
            if (lr == 0) {
              mind[j0 + j] = m;
              own[j0 + j] = cur;
            }
          } else if (pass == 0 && lr == 0) {
            mind[j0 + j] = m;  // the first pass writes every distance (inf stays for NaN rows)
            own[j0 + j] = cur;
          }
          better(bv, bi, m, row[r]);
        }
      }
      __syncthreads();  // the list is read; the next window may overwrite it
    }
    // wave: merge all lanes (phase 1 leaves each lane its own candidates);
    // block: merge the waves
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double ov = __shfl_xor(bv, off, kWave);
      const int64_t oi = __shfl_xor(bi, off, kWave);
      better(bv, bi, ov, oi);
    }
    if (lane == 0) {
      sv[wave] = bv;
      si[wave] = bi;
    }
    __syncthreads();
    if (t == 0) {
      double v = -1.0;
      int64_t i = -1;
      for (int w = 0; w < kWaves; ++w) better(v, i, sv[w], si[w]);
      s_pick = (i >= 0 && v >= 0.0) ? i : -1;
      if (s_pick >= 0) cpicks[j0 + cnt] = s_pick;
    }
    __syncthreads();
    pick = s_pick;
    if (pick < 0) break;
    ++cnt;
  }
  if (t == 0) ccount[c] = static_cast<uint32_t>(cnt);
}

// The total budget over the classes in ascending order: class c appends
// min(ccount[c], what is left) of its picks, in pick order, to picks[];
// total = the number appended.  One block; thread 0 takes the prefix.
__global__ __launch_bounds__(1024) void kcenter_budget_kernel(const uint32_t* __restrict__ ccount,
                                                              const int64_t* __restrict__ coff, int n_classes,
                                                              int64_t budget, const int64_t* __restrict__ cpicks,
                                                              int64_t* __restrict__ picks, int64_t* __restrict__ dst,
                                                              unsigned long long* __restrict__ total) {
  if (threadIdx.x == 0) {
    int64_t run = 0;
    for (int c = 0; c < n_classes; ++c) {
      int64_t take = ccount[c];
      if (take > budget - run) take = budget - run;
      dst[2 * c] = run;
      dst[2 * c + 1] = take;
      run += take;
    }
    *total = static_cast<unsigned long long>(run);
  }
  __syncthreads();
  for (int c = 0; c < n_classes; ++c) {
    const int64_t base = dst[2 * c], take = dst[2 * c + 1];
    for (int64_t q = threadIdx.x; q < take; q += blockDim.x) picks[base + q] = cpicks[coff[c] + q];
  }
}

// Rows of the picks [t0, t0 + k) as float32 stored values, with their
// payload and radius (for the append).
__global__ void kcenter_gather_kernel(const float* __restrict__ z, const int32_t* __restrict__ label,
                                      const float* __restrict__ r, const int64_t* __restrict__ picks, int64_t t0,
                                      int k, int d, int bf16, float* __restrict__ zc, int32_t* __restrict__ lc,
                                      float* __restrict__ rc) {
  const int j = static_cast<int>(blockIdx.x) * (blockDim.x / kWave) + static_cast<int>(threadIdx.x) / kWave;
  if (j >= k) return;
  const int64_t src = picks[t0 + j];
  const float* zr = z + src * d;
  float* out = zc + static_cast<int64_t>(j) * d;
  for (int c = lane_id(); c < d; c += kWave) out[c] = bf16 ? bf16_round_f32(zr[c]) : zr[c];
  if (lane_id() == 0) {
    lc[j] = label[src];
    rc[j] = r[src];
  }
}

// ------------------------------------------------------------- workspace
struct CWs {
  uint32_t* keys[2];
  uint32_t* vals[2];
  uint32_t* hist;
  uint32_t* dsum;
  uint32_t* dbase;
  unsigned long long* counters;  // [0] eligible, [1] appended
  float* zc;
  int32_t* lc;
  float* rc;
  int64_t* src_c;
  uint32_t* cand;       // [kChunk] candidates of the current chunk, in visit order
  int32_t* dup;
  int32_t* sel;
  uint32_t* rel;
  int32_t* class_count;
  double* mind;
  int64_t* pick;
  int64_t* start;
  int* group_count;
  double* part_v;
  int64_t* part_i;
  int64_t* picks;
  int64_t* cpicks;      // [n] per-class picks (per-class K-center)
  int32_t* own;         // [n] the pick that set mind (per-class K-center)
  uint32_t* ccount;     // [n_classes] candidates, then picks, per class
  int64_t* coff;        // [n_classes + 1] class list offsets
  int64_t* cdst;        // [2 n_classes] output offset and count per class
  void* sub_ws;  // lookup / insert workspace
  size_t sub_bytes;
  size_t total;
};

inline size_t sub_ws_bytes(const lipcache_cache* c) {
  const size_t a = lipcache_lookup_workspace_bytes(kChunk, c->capacity, c->d, LIPCACHE_F16);
  const size_t b = lipcache_insert_workspace_bytes(kChunk);
  return a > b ? a : b;
}

inline CWs cws_layout(int64_t n, int d, int n_classes, int64_t budget, size_t sub_bytes, char* base) {
  CWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off = align_up(off + bytes, 256);
    return p;
  };
  const int64_t nb = (n + kSortThreads - 1) / kSortThreads;
  for (int s = 0; s < 2; ++s) {
    w.keys[s] = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(n) * 4));
    w.vals[s] = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(n) * 4));
  }
  w.hist = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(nb) * kBins * 4));
  w.dsum = reinterpret_cast<uint32_t*>(take(kBins * 4));
  w.dbase = reinterpret_cast<uint32_t*>(take(kBins * 4));
  w.counters = reinterpret_cast<unsigned long long*>(take(64));
  w.zc = reinterpret_cast<float*>(take(static_cast<size_t>(kChunk) * d * 4));
  w.lc = reinterpret_cast<int32_t*>(take(kChunk * 4));
  w.rc = reinterpret_cast<float*>(take(kChunk * 4));
  w.src_c = reinterpret_cast<int64_t*>(take(kChunk * 8));
  w.cand = reinterpret_cast<uint32_t*>(take(kChunk * 4));
  w.dup = reinterpret_cast<int32_t*>(take(kChunk * 4));
  w.sel = reinterpret_cast<int32_t*>(take(kChunk * 4));
  w.rel = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(kChunk) * kChunkWords * 4));
  w.class_count = reinterpret_cast<int32_t*>(take(static_cast<size_t>(n_classes > 0 ? n_classes : 1) * 4));
  w.mind = reinterpret_cast<double*>(take(static_cast<size_t>(n) * 8));
  w.pick = reinterpret_cast<int64_t*>(take(8));
  w.start = reinterpret_cast<int64_t*>(take(8));
  w.group_count = reinterpret_cast<int*>(take(8));
  const int64_t kb = (n + 255) / 256;
  w.part_v = reinterpret_cast<double*>(take(static_cast<size_t>(kb) * 8));
  w.part_i = reinterpret_cast<int64_t*>(take(static_cast<size_t>(kb) * 8));
  w.picks = reinterpret_cast<int64_t*>(take(static_cast<size_t>(budget > 0 ? budget : 1) * 8));
  const size_t nc = static_cast<size_t>(n_classes > 0 ? n_classes : 1);
  w.cpicks = reinterpret_cast<int64_t*>(take(static_cast<size_t>(n > 0 ? n : 1) * 8));
  w.own = reinterpret_cast<int32_t*>(take(static_cast<size_t>(n > 0 ? n : 1) * 4));
  w.ccount = reinterpret_cast<uint32_t*>(take(nc * 4));
  w.coff = reinterpret_cast<int64_t*>(take((nc + 1) * 8));
  w.cdst = reinterpret_cast<int64_t*>(take(2 * nc * 8));
  w.sub_ws = take(sub_bytes);
  w.sub_bytes = sub_bytes;
  w.total = off;
  return w;
}

}  // namespace lc

using namespace lc;

extern "C" size_t lipcache_construct_workspace_bytes(const lipcache_cache* c, int64_t N, int32_t n_classes,
                                                     int64_t budget) {
  if (!c || N < 0 || c->capacity < 0 || c->d < 1) return 0;
  const int64_t free_rows = c->capacity - c->n;
  const int64_t b = budget < 0 ? free_rows : budget;
  return cws_layout(N, c->d, n_classes, b, sub_ws_bytes(c), nullptr).total;
}

extern "C" lipcache_status lipcache_construct(lipcache_cache* c, const float* z, const int32_t* label,
                                              const float* r, const int32_t* guard_label, const float* priority,
                                              int64_t N, int32_t strategy, int64_t budget, int32_t per_class,
                                              int32_t n_classes, int64_t* selected_out, int64_t* appended,
                                              void* ws, size_t ws_bytes, lipcache_stream_t stream) {
  if (!c || N < 0 || N > INT32_MAX) return N > INT32_MAX ? LIPCACHE_EUNSUPPORTED : LIPCACHE_EINVAL;
  if (c->d < 32 || c->d > 1024 || c->d % 32 != 0) return LIPCACHE_EINVAL;
  if (c->store_dtype != LIPCACHE_F32 && c->store_dtype != LIPCACHE_BF16) return LIPCACHE_EINVAL;
  if (c->n < 0 || c->capacity < 0 || c->n > c->capacity) return LIPCACHE_EINVAL;
  if (c->capacity > 0 && (!c->z || !c->r || !c->label || !c->norm2)) return LIPCACHE_EINVAL;
  if (strategy != LIPCACHE_SELECT_RADIUS_DEDUP && strategy != LIPCACHE_SELECT_PRIORITY &&
      strategy != LIPCACHE_SELECT_KCENTER)
    return LIPCACHE_EINVAL;
  if (N > 0 && (!z || !label || !r)) return LIPCACHE_EINVAL;
  if (strategy == LIPCACHE_SELECT_PRIORITY && N > 0 && !priority) return LIPCACHE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(z) & 15u) != 0) return LIPCACHE_EINVAL;
  if (per_class < 0) return LIPCACHE_EINVAL;
  if (per_class > 0 && (n_classes < 1 || n_classes > kMaxClasses)) return LIPCACHE_EINVAL;
  const int64_t free_rows = c->capacity - c->n;
  const int64_t bud = budget < 0 ? free_rows : budget;
  if (bud > free_rows) return LIPCACHE_ECAPACITY;
  const size_t need = lipcache_construct_workspace_bytes(c, N, n_classes, budget);
  if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;
  if (appended) *appended = 0;
  if (N == 0 || bud == 0) return LIPCACHE_OK;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  CWs w = cws_layout(N, c->d, n_classes, bud, sub_ws_bytes(c), static_cast<char*>(ws));
  const int d = c->d;
  const int bf16 = c->store_dtype == LIPCACHE_BF16 ? 1 : 0;
  const int ncls = per_class > 0 ? n_classes : 0;
  const float* prio = strategy == LIPCACHE_SELECT_PRIORITY ? priority : nullptr;

  // ---- eligibility and visit order (stable radix sort by descending key)
  hipLaunchKernelGGL(fill_u64_kernel, dim3(1), dim3(64), 0, s, w.counters, 8, 0ull);
  LC_LAUNCHED();
  if (ncls > 0) {
    hipLaunchKernelGGL(fill_i32_kernel, dim3(static_cast<unsigned>((ncls + 255) / 256)), dim3(256), 0, s,
                       w.class_count, static_cast<int64_t>(ncls), 0);
    LC_LAUNCHED();
  }
  const unsigned g256 = static_cast<unsigned>((N + 255) / 256);
  hipLaunchKernelGGL(construct_keys_kernel, dim3(g256), dim3(256), 0, s, r, prio, label, guard_label, N, ncls,
                     w.keys[0], w.vals[0], w.counters);
  LC_LAUNCHED();
  int cur = 0;
  LC_HIP(radix_sort_u32(w.keys, w.vals, N, 4, w.hist, w.dsum, w.dbase, cur, s));
  const uint32_t* order = w.vals[cur];
  unsigned long long host_cnt[2] = {0ull, 0ull};
  LC_HIP(read_back(host_cnt, w.counters, 16, s));
  const int64_t n_elig = static_cast<int64_t>(host_cnt[0]);
  if (n_elig == 0) return LIPCACHE_OK;
  unsigned long long* total_dev = w.counters + 1;

  int64_t added = 0;
  if (strategy != LIPCACHE_SELECT_KCENTER) {
    const int dedup = strategy == LIPCACHE_SELECT_RADIUS_DEDUP ? 1 : 0;
    // counters[2], [3]: visit cursor and size of the next chunk
    unsigned long long* cursor = w.counters + 2;
    auto next_chunk = [&]() {
      hipLaunchKernelGGL(construct_compact_kernel, dim3(1), dim3(1024), 0, s, order, n_elig, label, w.class_count,
                         per_class, cursor, w.cand);
      return hipGetLastError();
    };
    LC_HIP(next_chunk());
    unsigned long long cur_k[2] = {0ull, 0ull};
    LC_HIP(read_back(cur_k, cursor, 16, s));
    while (cur_k[1] > 0 && added < bud) {
      const int k = static_cast<int>(cur_k[1]);
      hipLaunchKernelGGL(construct_gather_kernel, dim3(static_cast<unsigned>((k + 3) / 4)), dim3(256), 0, s, z, label,
                         r, w.cand, k, d, bf16, w.zc, w.lc, w.rc, w.src_c);
      LC_LAUNCHED();
      const int32_t* dup = nullptr;
      if (dedup) {
        if (c->n > 0) {
          const lipcache_status st = lipcache_lookup(c, w.zc, k, LIPCACHE_F16, w.dup, nullptr, nullptr, nullptr,
                                                     nullptr, w.sub_ws, w.sub_bytes, stream);
          if (st != LIPCACHE_OK) return st;
          dup = w.dup;
        }
        const unsigned tiles = static_cast<unsigned>((k + 31) / 32);
        hipLaunchKernelGGL(construct_relation_kernel, dim3(tiles, tiles), dim3(1024), 0, s, w.zc, w.rc, k, d, w.rel);
        LC_LAUNCHED();
      }
      AcceptParams ap;
      ap.k = k;
      ap.dedup = dedup;
      ap.dup_label = dup;
      ap.rel = dedup ? w.rel : nullptr;
      ap.lc = w.lc;
      ap.src_c = w.src_c;
      ap.sel = w.sel;
      ap.class_count = w.class_count;
      ap.n_classes = ncls;
      ap.per_class = per_class;
      ap.total = total_dev;
      ap.budget = static_cast<unsigned long long>(bud);
      ap.selected_out = selected_out;
      hipLaunchKernelGGL(construct_accept_kernel, dim3(1), dim3(1024), 0, s, ap);
      LC_LAUNCHED();
      // the next chunk, from the class counts this one leaves (its
      // candidates were copied to zc by the gather above)
      LC_HIP(next_chunk());
      int64_t got = 0;
      const lipcache_status st = lipcache_insert(c, w.zc, w.lc, w.rc, w.sel, k, &got, w.sub_ws, w.sub_bytes, stream);
      if (st != LIPCACHE_OK) return st;
      added += got;
      LC_HIP(read_back(cur_k, cursor, 16, s));
    }
  } else {
    if (per_class > 0) {
      // every class on its own workgroup, then the total budget in class order
      hipLaunchKernelGGL(fill_i32_kernel, dim3(static_cast<unsigned>((ncls + 255) / 256)), dim3(256), 0, s,
                         reinterpret_cast<int32_t*>(w.ccount), static_cast<int64_t>(ncls), 0);
      LC_LAUNCHED();
      const int other = cur ^ 1;
      hipLaunchKernelGGL(class_keys_kernel, dim3(static_cast<unsigned>((n_elig + 4095) / 4096)), dim3(256), 0, s,
                         label, order, n_elig, ncls, w.keys[other], w.vals[other], w.ccount);
      LC_LAUNCHED();
      int ccur = other;
      LC_HIP(radix_sort_u32(w.keys, w.vals, n_elig, ncls <= 256 ? 1 : 2, w.hist, w.dsum, w.dbase, ccur, s));
      hipLaunchKernelGGL(exclusive_scan_kernel, dim3(1), dim3(1024), 0, s, w.ccount, ncls, w.coff);
      LC_LAUNCHED();
      const dim3 kgrid(static_cast<unsigned>(ncls));
      const uint32_t* clist = w.vals[ccur];
      if (d <= 64)
        hipLaunchKernelGGL((kcenter_class_kernel<1, kKcThreads>), kgrid, dim3(kKcThreads), 0, s, z, d, bf16, clist, w.coff,
                           per_class, bud, w.mind, w.own, w.cpicks, w.ccount);
      else if (d <= 128)
        hipLaunchKernelGGL((kcenter_class_kernel<2, kKcThreads>), kgrid, dim3(kKcThreads), 0, s, z, d, bf16, clist, w.coff,
                           per_class, bud, w.mind, w.own, w.cpicks, w.ccount);
      else if (d <= 256)
        hipLaunchKernelGGL((kcenter_class_kernel<4, kKcThreads>), kgrid, dim3(kKcThreads), 0, s, z, d, bf16, clist, w.coff,
                           per_class, bud, w.mind, w.own, w.cpicks, w.ccount);
      else if (d <= 512)
        hipLaunchKernelGGL((kcenter_class_kernel<8, 512>), kgrid, dim3(512), 0, s, z, d, bf16, clist, w.coff,
                           per_class, bud, w.mind, w.own, w.cpicks, w.ccount);
      else
        hipLaunchKernelGGL((kcenter_class_kernel<16, 512>), kgrid, dim3(512), 0, s, z, d, bf16, clist, w.coff,
                           per_class, bud, w.mind, w.own, w.cpicks, w.ccount);
      LC_LAUNCHED();
      hipLaunchKernelGGL(kcenter_budget_kernel, dim3(1), dim3(1024), 0, s, w.ccount, w.coff, ncls, bud, w.cpicks,
                         w.picks, w.cdst, total_dev);
      LC_LAUNCHED();
    } else {
      // one traversal over all eligible candidates
      const int64_t kb = (N + 255) / 256;
      KcParams kp;
      kp.z = z;
      kp.r = r;
      kp.prio = nullptr;
      kp.label = label;
      kp.guard = guard_label;
      kp.n = N;
      kp.d = d;
      kp.bf16 = bf16;
      kp.n_classes = ncls;
      kp.group = -1;
      kp.mind = w.mind;
      kp.pick = w.pick;
      kp.part_v = w.part_v;
      kp.part_i = w.part_i;
      kp.total = total_dev;
      kp.budget = static_cast<unsigned long long>(bud);
      kp.picks = w.picks;
      kp.group_count = w.group_count;
      kp.limit = static_cast<int>(bud < INT_MAX ? bud : INT_MAX);
      hipLaunchKernelGGL(kcenter_start_kernel, dim3(1), dim3(256), 0, s, label, order, n_elig, kp.group, w.start);
      LC_LAUNCHED();
      hipLaunchKernelGGL(kcenter_init_kernel, dim3(static_cast<unsigned>(kb)), dim3(256), 0, s, kp, w.start);
      LC_LAUNCHED();
      const int64_t steps = (bud < n_elig ? bud : n_elig) - 1;
      for (int64_t it = 0; it < steps; ++it) {
        hipLaunchKernelGGL(kcenter_step_kernel, dim3(static_cast<unsigned>(kb)), dim3(256), 0, s, kp);
        LC_LAUNCHED();
        hipLaunchKernelGGL(kcenter_pick_kernel, dim3(1), dim3(256), 0, s, kp, static_cast<int>(kb));
        LC_LAUNCHED();
      }
    }
    LC_HIP(read_back(host_cnt, w.counters, 16, s));
    const int64_t npick = static_cast<int64_t>(host_cnt[1]);
    if (selected_out && npick > 0)
      LC_HIP(hipMemcpyAsync(selected_out, w.picks, static_cast<size_t>(npick) * 8, hipMemcpyDeviceToDevice, s));
    for (int64_t t0 = 0; t0 < npick; t0 += kChunk) {
      const int k = static_cast<int>(npick - t0 < kChunk ? npick - t0 : kChunk);
      hipLaunchKernelGGL(kcenter_gather_kernel, dim3(static_cast<unsigned>((k + 3) / 4)), dim3(256), 0, s, z, label, r,
                         w.picks, t0, k, d, bf16, w.zc, w.lc, w.rc);
      LC_LAUNCHED();
      int64_t got = 0;
      const lipcache_status st = lipcache_insert(c, w.zc, w.lc, w.rc, nullptr, k, &got, w.sub_ws, w.sub_bytes, stream);
      if (st != LIPCACHE_OK) return st;
      added += got;
    }
  }
  if (appended) *appended = added;
  return LIPCACHE_OK;
}
