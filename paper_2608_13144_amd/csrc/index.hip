// Exact cluster index for a sublinear lookup.
//
// Build: K centres start at evenly spaced cache rows; `iters` Lloyd
// iterations assign every live row to its nearest centre (float32 tiles in
// LDS) and move each centre to the float64 mean of its rows.  After the
// final assignment a stable radix sort by cluster gives the row order, the
// cluster offsets come from the counts, and R_c = max over live members of
// ||z_i - mu_c|| + r_i is taken in float64 and rounded up to float32.  The
// indexed rows are copied into a cluster-ordered cache.  Any partition
// gives exact answers; the iterations only make the clusters tight.
//
// Query plan: for every query the clusters with ||q - mu_c|| < R_c (the
// float32 distance keeps a cluster whenever its rounding error could hide
// one), and the nearest cluster; queries are sorted by nearest cluster so
// that a block of them shares few clusters; each block's union of needed
// clusters becomes work items for the fused lookup kernel.
#include <limits.h>

#include "lc_common.hpp"
#include "lc_index.hpp"
#include "lc_sort.hpp"

namespace lc {

constexpr int kTq = 64;   // queries (or rows) per distance tile
constexpr int kTc = 64;   // centres per distance tile
constexpr int kTd = 32;   // feature columns per LDS stage

__device__ __forceinline__ float stored_value(const void* z, int store, int64_t i, int d, int k) {
  if (store == LIPCACHE_BF16) return bf16_to_f32(static_cast<const uint16_t*>(z)[i * d + k]);
  return static_cast<const float*>(z)[i * d + k];
}

// Rows `rows` (n of them, float32 or bf16 storage) against K centres: the
// nearest centre (ties: lower index) among those with usable[c] != 0 (all
// when usable is null), and optionally the candidate mask
// mask[r][c / 32] |= bit for ||x_r - mu_c||^2 < R_c^2 (1 + slack_rel).
// Block: 256 threads, kTq rows; loops over all centre tiles.  Thread t
// owns rows 4 (t / 16) .. +3 and centres 4 (t % 16) .. +3 of each tile.
__global__ __launch_bounds__(256) void nearest_centre_kernel(const void* __restrict__ rows, int store, int64_t n,
                                                             int d, const float* __restrict__ centres, int K,
                                                             const float* __restrict__ bound, double slack_rel,
                                                             uint32_t* __restrict__ mask,
                                                             uint32_t* __restrict__ nearest) {
  __shared__ float xs[kTq][kTd + 1];
  __shared__ float cs[kTc][kTd + 1];
  __shared__ float bestv[kTq][16];
  __shared__ int besti[kTq][16];
  const int t = static_cast<int>(threadIdx.x);
  const int tr = t / 16, tc = t % 16;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kTq;
  const int words = (K + 31) / 32;
  float bv[4];
  int bi[4];
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    bv[a] = __builtin_inff();
    bi[a] = INT_MAX;
  }
  for (int c0 = 0; c0 < K; c0 += kTc) {
    float acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = 0.0f;
    for (int k0 = 0; k0 < d; k0 += kTd) {
      __syncthreads();
      for (int e = t; e < kTq * kTd; e += 256) {
        const int rr = e / kTd, kk = e % kTd;
        const int64_t row = r0 + rr;
        const int c = c0 + rr;
        xs[rr][kk] = row < n ? stored_value(rows, store, row, d, k0 + kk) : 0.0f;
        cs[rr][kk] = c < K ? centres[static_cast<int64_t>(c) * d + k0 + kk] : 0.0f;
      }
      __syncthreads();
#pragma unroll 4
      for (int kk = 0; kk < kTd; ++kk) {
        float xv[4], cv[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) xv[a] = xs[4 * tr + a][kk];
#pragma unroll
        for (int b = 0; b < 4; ++b) cv[b] = cs[4 * tc + b][kk];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const float df = xv[a] - cv[b];
            acc[a][b] = __builtin_fmaf(df, df, acc[a][b]);
          }
      }
    }
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int64_t row = r0 + 4 * tr + a;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int c = c0 + 4 * tc + b;
        if (c >= K || row >= n) continue;
        const bool use = bound == nullptr || bound[c] > 0.0f;
        if (use && (acc[a][b] < bv[a] || (acc[a][b] == bv[a] && c < bi[a]))) {
          bv[a] = acc[a][b];
          bi[a] = c;
        }
        if (mask && use) {
          const double R = static_cast<double>(bound[c]);
          if (static_cast<double>(acc[a][b]) < R * R * (1.0 + slack_rel))
            atomicOr(&mask[row * words + c / 32], 1u << (c % 32));
        }
      }
    }
  }
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    bestv[4 * tr + a][tc] = bv[a];
    besti[4 * tr + a][tc] = bi[a];
  }
  __syncthreads();
  if (t < kTq && r0 + t < n) {
    float v = bestv[t][0];
    int i = besti[t][0];
    for (int j = 1; j < 16; ++j) {
      if (bestv[t][j] < v || (bestv[t][j] == v && besti[t][j] < i)) {
        v = bestv[t][j];
        i = besti[t][j];
      }
    }
    nearest[r0 + t] = i == INT_MAX ? 0u : static_cast<uint32_t>(i);
  }
}

__global__ void fill_f64_kernel(double* __restrict__ p, int64_t n, double v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void fill_u32_kernel(uint32_t* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

__global__ void fill_u64x_kernel(unsigned long long* __restrict__ p, int64_t n, unsigned long long v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// centres[j] = row floor(j n / K) (stored values as float32).
__global__ void centre_init_kernel(const void* __restrict__ z, int store, int64_t n, int d, int K,
                                   float* __restrict__ centres) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(K) * d) return;
  const int j = static_cast<int>(t / d), k = static_cast<int>(t % d);
  const int64_t row = static_cast<int64_t>(j) * n / K;
  centres[t] = stored_value(z, store, row, d, k);
}

// sum[c][k] += z_ik, cnt[c] += 1 over live rows (thread per (row, column)).
__global__ void centre_sum_kernel(const void* __restrict__ z, int store, const float* __restrict__ r, int64_t n,
                                  int d, const uint32_t* __restrict__ assign, double* __restrict__ sum,
                                  unsigned long long* __restrict__ cnt) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= n * d) return;
  const int64_t i = t / d;
  const int k = static_cast<int>(t % d);
  if (!(r[i] > 0.0f)) return;
  const uint32_t c = assign[i];
  atomicAdd(&sum[static_cast<int64_t>(c) * d + k], static_cast<double>(stored_value(z, store, i, d, k)));
  if (k == 0) atomicAdd(&cnt[c], 1ull);
}

__global__ void centre_update_kernel(const double* __restrict__ sum, const unsigned long long* __restrict__ cnt,
                                     int K, int d, float* __restrict__ centres) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(K) * d) return;
  const unsigned long long m = cnt[t / d];
  if (m > 0) centres[t] = static_cast<float>(sum[t] / static_cast<double>(m));
}

// Keys for the stable sort of rows by cluster; dead rows go to their cluster
// too (they are kept, they just never raise R_c).
__global__ void row_keys_kernel(const uint32_t* __restrict__ assign, int64_t n, uint32_t* __restrict__ keys,
                                uint32_t* __restrict__ vals) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  keys[i] = assign[i];
  vals[i] = static_cast<uint32_t>(i);
}

__global__ void count_kernel(const uint32_t* __restrict__ assign, int64_t n, unsigned long long* __restrict__ cnt) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) atomicAdd(&cnt[assign[i]], 1ull);
}

// offsets[c] = sum of counts below c (one block, serial chunks).
__global__ void offsets_kernel(const unsigned long long* __restrict__ cnt, int K, int64_t* __restrict__ offsets) {
  if (threadIdx.x != 0) return;
  int64_t s = 0;
  for (int c = 0; c < K; ++c) {
    offsets[c] = s;
    s += static_cast<int64_t>(cnt[c]);
  }
  offsets[K] = s;
}

// Sorted row j: copy cache row perm[j]; R_c candidates from live rows.
__global__ void reorder_kernel(const lipcache_cache c, lipcache_cache out, const uint32_t* __restrict__ order,
                               int64_t n, int64_t* __restrict__ perm, const uint32_t* __restrict__ assign,
                               const float* __restrict__ centres, unsigned long long* __restrict__ rbits) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (j >= n) return;
  const int lane = lane_id();
  const int64_t src = order[j];
  const int d = c.d;
  const uint32_t cl = assign[src];
  double part = 0.0;
  for (int k = lane; k < d; k += kWave) {
    if (c.store_dtype == LIPCACHE_BF16) {
      const uint16_t h = static_cast<const uint16_t*>(c.z)[src * d + k];
      static_cast<uint16_t*>(out.z)[j * d + k] = h;
      const double diff = static_cast<double>(bf16_to_f32(h)) - static_cast<double>(centres[static_cast<int64_t>(cl) * d + k]);
      part = __builtin_fma(diff, diff, part);
    } else {
      const float v = static_cast<const float*>(c.z)[src * d + k];
      static_cast<float*>(out.z)[j * d + k] = v;
      if (out.zimg) {
        static_cast<uint16_t*>(out.zimg)[j * d + k] =
            c.zimg ? static_cast<const uint16_t*>(c.zimg)[src * d + k] : bf16_bits(v);
      }
      const double diff = static_cast<double>(v) - static_cast<double>(centres[static_cast<int64_t>(cl) * d + k]);
      part = __builtin_fma(diff, diff, part);
    }
  }
  const double d2 = wave_sum(part);
  if (lane == 0) {
    perm[j] = src;
    const float rr = c.r[src];
    out.r[j] = rr;
    out.label[j] = c.label[src];
    out.norm2[j] = c.norm2[src];
    if (rr > 0.0f) {
      // the ball widened by 2^-16 r, so every pair inside the 1e-5 r band of
      // the re-check is also reached
      const double reach = __builtin_sqrt(d2) + static_cast<double>(rr) * (1.0 + 0x1p-16);
      atomicMax(&rbits[cl], __builtin_bit_cast(unsigned long long, reach));
    }
  }
}

// R_c rounded up to float32; -inf when no live member.  The reach values are
// non-negative doubles, whose bit patterns order like the values, so the
// 64-bit atomicMax above takes the largest.
__global__ void bound_kernel(const unsigned long long* __restrict__ rbits, int K, float* __restrict__ bound) {
  const int c = static_cast<int>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (c >= K) return;
  const unsigned long long b = rbits[c];
  if (b == 0ull) {
    bound[c] = -__builtin_inff();
    return;
  }
  // 2^-40 covers the float64 rounding of the squared sum, the root and the
  // addition (d <= 1024 terms)
  const double R = __builtin_bit_cast(double, b) * (1.0 + 0x1p-40);
  float f = static_cast<float>(R);
  if (static_cast<double>(f) < R) f = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, f) + 1u);
  bound[c] = f;
}

struct BuildWs {
  uint32_t* assign;
  double* sum;
  unsigned long long* cnt;
  unsigned long long* rbits;
  uint32_t* keys[2];
  uint32_t* vals[2];
  uint32_t* hist;
  uint32_t* dsum;
  uint32_t* dbase;
  size_t total;
};

inline BuildWs build_layout(int64_t n, int d, int K, char* base) {
  BuildWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off = align_up(off + bytes, 256);
    return p;
  };
  w.assign = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(n) * 4));
  w.sum = reinterpret_cast<double*>(take(static_cast<size_t>(K) * d * 8));
  w.cnt = reinterpret_cast<unsigned long long*>(take(static_cast<size_t>(K) * 8));
  w.rbits = reinterpret_cast<unsigned long long*>(take(static_cast<size_t>(K) * 8));
  for (int s = 0; s < 2; ++s) {
    w.keys[s] = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(n) * 4));
    w.vals[s] = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(n) * 4));
  }
  w.hist = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(radix_blocks(n)) * kBins * 4));
  w.dsum = reinterpret_cast<uint32_t*>(take(kBins * 4));
  w.dbase = reinterpret_cast<uint32_t*>(take(kBins * 4));
  w.total = off;
  return w;
}

inline int sort_passes(int K) {
  int p = 1;
  while (p < 4 && (static_cast<int64_t>(1) << (8 * p)) < K) ++p;
  return p;
}

// ---------------------------------------------------------------- query plan
__global__ void plan_keys_kernel(const uint32_t* __restrict__ nearest, int64_t B, uint32_t* __restrict__ keys,
                                 uint32_t* __restrict__ vals) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= B) return;
  keys[i] = nearest[i];
  vals[i] = static_cast<uint32_t>(i);
}

// Internal query j = original query order[j]: copy its row, record the map.
__global__ void plan_gather_kernel(const float* __restrict__ zq, const uint32_t* __restrict__ order, int64_t B,
                                   int d, float* __restrict__ zs, int64_t* __restrict__ qmap) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (j >= B) return;
  const int64_t src = order[j];
  for (int k = lane_id(); k < d; k += kWave) zs[j * d + k] = zq[src * d + k];
  if (lane_id() == 0) qmap[j] = src;
}

// One block per query block: union of the candidate clusters of its
// queries, then one item per (needed cluster, chunk of <= kItemRows rows).
__global__ __launch_bounds__(256) void plan_items_kernel(const uint32_t* __restrict__ mask, int words,
                                                         const int64_t* __restrict__ qmap, int64_t B, int qblock,
                                                         const int64_t* __restrict__ offsets, int64_t* __restrict__ items,
                                                         int64_t capacity, unsigned long long* __restrict__ counters) {
  extern __shared__ uint32_t un[];  // [words]
  const int qb = static_cast<int>(blockIdx.x);
  for (int w = threadIdx.x; w < words; w += 256) un[w] = 0u;
  __syncthreads();
  const int64_t q0 = static_cast<int64_t>(qb) * qblock;
  const int64_t q1 = q0 + qblock < B ? q0 + qblock : B;
  for (int64_t q = q0 + threadIdx.x / 8; q < q1; q += 256 / 8) {
    const uint32_t* row = mask + qmap[q] * words;
    for (int w = threadIdx.x % 8; w < words; w += 8) {
      const uint32_t v = row[w];
      if (v) atomicOr(&un[w], v);
    }
  }
  __syncthreads();
  const unsigned long long nq = static_cast<unsigned long long>(q1 - q0);
  for (int w = threadIdx.x; w < words; w += 256) {
    uint32_t v = un[w];
    while (v) {
      const int b = __builtin_ctz(v);
      v &= v - 1u;
      const int c = 32 * w + b;
      const int64_t e0 = offsets[c], e1 = offsets[c + 1];
      for (int64_t s = e0; s < e1; s += kItemRows) {
        const int64_t e = s + kItemRows < e1 ? s + kItemRows : e1;
        const unsigned long long slot = atomicAdd(&counters[0], 1ull);
        atomicAdd(&counters[1], nq * static_cast<unsigned long long>(e - s));
        if (static_cast<int64_t>(slot) < capacity) {
          items[3 * slot] = qb;
          items[3 * slot + 1] = s;
          items[3 * slot + 2] = e;
        } else {
          atomicOr(&counters[2], 1ull);
        }
      }
    }
  }
}

}  // namespace lc

using namespace lc;

namespace lc {

size_t index_plan_layout(int64_t B, int d, int K, int64_t n_indexed, int qblock, IndexPlanWs* w, char* base) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off = align_up(off + bytes, 256);
    return p;
  };
  const int words = (K + 31) / 32;
  const int64_t nqb = (B + qblock - 1) / qblock;
  IndexPlanWs t{};
  t.mask = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(B) * words * 4));
  for (int s = 0; s < 2; ++s) {
    t.keys[s] = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(B) * 4));
    t.vals[s] = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(B) * 4));
  }
  t.hist = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(radix_blocks(B)) * kBins * 4));
  t.dsum = reinterpret_cast<uint32_t*>(take(kBins * 4));
  t.dbase = reinterpret_cast<uint32_t*>(take(kBins * 4));
  t.qmap = reinterpret_cast<int64_t*>(take(static_cast<size_t>(B) * 8));
  t.zq_sorted = reinterpret_cast<float*>(take(static_cast<size_t>(B) * d * 4));
  t.capacity = nqb * (K + n_indexed / kItemRows + 1);
  t.items = reinterpret_cast<int64_t*>(take(static_cast<size_t>(t.capacity) * 3 * 8));
  t.counters = reinterpret_cast<unsigned long long*>(take(64));
  if (w) *w = t;
  return off;
}

lipcache_status index_query_plan(const lipcache_index* idx, const float* zq, int64_t B, int d, int qblock,
                                 const IndexPlanWs& w, int64_t& n_items, int64_t& pairs, hipStream_t s) {
  const int K = idx->K;
  const int words = (K + 31) / 32;
  const int64_t mwords = B * words;
  hipLaunchKernelGGL(fill_u64x_kernel, dim3(1), dim3(64), 0, s, w.counters, 8, 0ull);
  LC_LAUNCHED();
  hipLaunchKernelGGL(fill_u32_kernel, dim3(static_cast<unsigned>((mwords + 255) / 256)), dim3(256), 0, s, w.mask,
                     mwords);
  LC_LAUNCHED();
  // rigorous slack of the float32 squared distance: 4 (d + 3) u, relative
  const double slack = 4.0 * (d + 3) / 16777216.0;
  hipLaunchKernelGGL(nearest_centre_kernel, dim3(static_cast<unsigned>((B + kTq - 1) / kTq)), dim3(256), 0, s, zq,
                     LIPCACHE_F32, B, d, idx->centers, K, idx->bound, slack, w.mask, w.keys[1]);
  LC_LAUNCHED();
  hipLaunchKernelGGL(plan_keys_kernel, dim3(static_cast<unsigned>((B + 255) / 256)), dim3(256), 0, s, w.keys[1], B,
                     w.keys[0], w.vals[0]);
  LC_LAUNCHED();
  uint32_t* keys[2] = {w.keys[0], w.keys[1]};
  uint32_t* vals[2] = {w.vals[0], w.vals[1]};
  int cur = 0;
  LC_HIP(radix_sort_u32(keys, vals, B, sort_passes(K), w.hist, w.dsum, w.dbase, cur, s));
  hipLaunchKernelGGL(plan_gather_kernel, dim3(static_cast<unsigned>((B + 3) / 4)), dim3(256), 0, s, zq, vals[cur], B,
                     d, w.zq_sorted, w.qmap);
  LC_LAUNCHED();
  const int64_t nqb = (B + qblock - 1) / qblock;
  hipLaunchKernelGGL(plan_items_kernel, dim3(static_cast<unsigned>(nqb)), dim3(256),
                     static_cast<size_t>(words) * 4, s, w.mask, words, w.qmap, B, qblock, idx->offsets, w.items,
                     w.capacity, w.counters);
  LC_LAUNCHED();
  unsigned long long host[3] = {0ull, 0ull, 0ull};
  LC_HIP(hipMemcpyAsync(host, w.counters, sizeof(host), hipMemcpyDeviceToHost, s));
  LC_HIP(hipStreamSynchronize(s));
  if (host[2] != 0ull) return LIPCACHE_EHIP;  // the capacity bound was wrong: never expected
  n_items = static_cast<int64_t>(host[0]);
  pairs = static_cast<int64_t>(host[1]);
  return LIPCACHE_OK;
}

}  // namespace lc

extern "C" size_t lipcache_index_build_workspace_bytes(int64_t n, int32_t d, int32_t K) {
  if (n < 0 || d < 1 || K < 1) return 0;
  return build_layout(n, d, K, nullptr).total;
}

extern "C" lipcache_status lipcache_index_build(const lipcache_cache* c, int32_t K, int32_t iters,
                                                lipcache_index* idx, void* ws, size_t ws_bytes,
                                                lipcache_stream_t stream) {
  if (!c || !idx) return LIPCACHE_EINVAL;
  if (c->d < 32 || c->d > 1024 || c->d % 32 != 0) return LIPCACHE_EINVAL;
  if (c->store_dtype != LIPCACHE_F32 && c->store_dtype != LIPCACHE_BF16) return LIPCACHE_EINVAL;
  if (c->n < 1 || c->n > c->capacity || c->n >= static_cast<int64_t>(UINT_MAX)) return LIPCACHE_EINVAL;
  if (!c->z || !c->r || !c->label || !c->norm2) return LIPCACHE_EINVAL;
  if (K < 1 || K > 65536 || K > c->n || iters < 0 || iters > 1000) return LIPCACHE_EINVAL;
  const lipcache_cache& so = idx->sorted;
  if (so.d != c->d || so.store_dtype != c->store_dtype || so.capacity < c->n) return LIPCACHE_EINVAL;
  if (!so.z || !so.r || !so.label || !so.norm2 || !idx->perm || !idx->offsets || !idx->centers || !idx->bound)
    return LIPCACHE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(so.z) & 15u) != 0 || (reinterpret_cast<uintptr_t>(so.zimg) & 15u) != 0)
    return LIPCACHE_EINVAL;
  const size_t need = lipcache_index_build_workspace_bytes(c->n, c->d, K);
  if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  BuildWs w = build_layout(c->n, c->d, K, static_cast<char*>(ws));
  const int64_t n = c->n;
  const int d = c->d;
  const int64_t kd = static_cast<int64_t>(K) * d;
  hipLaunchKernelGGL(centre_init_kernel, dim3(static_cast<unsigned>((kd + 255) / 256)), dim3(256), 0, s, c->z,
                     c->store_dtype, n, d, K, idx->centers);
  LC_LAUNCHED();
  const unsigned gq = static_cast<unsigned>((n + kTq - 1) / kTq);
  for (int it = 0; it < iters; ++it) {
    hipLaunchKernelGGL(nearest_centre_kernel, dim3(gq), dim3(256), 0, s, c->z, c->store_dtype, n, d, idx->centers,
                       K, nullptr, 0.0, nullptr, w.assign);
    LC_LAUNCHED();
    hipLaunchKernelGGL(fill_f64_kernel, dim3(static_cast<unsigned>((kd + 255) / 256)), dim3(256), 0, s, w.sum, kd,
                       0.0);
    LC_LAUNCHED();
    hipLaunchKernelGGL(fill_u64x_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0, s, w.cnt,
                       static_cast<int64_t>(K), 0ull);
    LC_LAUNCHED();
    const int64_t nd = n * d;
    hipLaunchKernelGGL(centre_sum_kernel, dim3(static_cast<unsigned>((nd + 255) / 256)), dim3(256), 0, s, c->z,
                       c->store_dtype, c->r, n, d, w.assign, w.sum, w.cnt);
    LC_LAUNCHED();
    hipLaunchKernelGGL(centre_update_kernel, dim3(static_cast<unsigned>((kd + 255) / 256)), dim3(256), 0, s, w.sum,
                       w.cnt, K, d, idx->centers);
    LC_LAUNCHED();
  }
  hipLaunchKernelGGL(nearest_centre_kernel, dim3(gq), dim3(256), 0, s, c->z, c->store_dtype, n, d, idx->centers, K,
                     nullptr, 0.0, nullptr, w.assign);
  LC_LAUNCHED();
  hipLaunchKernelGGL(row_keys_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s, w.assign, n,
                     w.keys[0], w.vals[0]);
  LC_LAUNCHED();
  int cur = 0;
  LC_HIP(radix_sort_u32(w.keys, w.vals, n, sort_passes(K), w.hist, w.dsum, w.dbase, cur, s));
  hipLaunchKernelGGL(fill_u64x_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0, s, w.cnt,
                     static_cast<int64_t>(K), 0ull);
  LC_LAUNCHED();
  hipLaunchKernelGGL(count_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s, w.assign, n, w.cnt);
  LC_LAUNCHED();
  hipLaunchKernelGGL(offsets_kernel, dim3(1), dim3(64), 0, s, w.cnt, K, idx->offsets);
  LC_LAUNCHED();
  hipLaunchKernelGGL(fill_u64x_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0, s, w.rbits,
                     static_cast<int64_t>(K), 0ull);
  LC_LAUNCHED();
  lipcache_cache out = idx->sorted;
  hipLaunchKernelGGL(reorder_kernel, dim3(static_cast<unsigned>((n + 3) / 4)), dim3(256), 0, s, *c, out, w.vals[cur],
                     n, idx->perm, w.assign, idx->centers, w.rbits);
  LC_LAUNCHED();
  hipLaunchKernelGGL(bound_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0, s, w.rbits, K,
                     idx->bound);
  LC_LAUNCHED();
  idx->K = K;
  idx->n_indexed = n;
  idx->sorted.n = n;
  return LIPCACHE_OK;
}
