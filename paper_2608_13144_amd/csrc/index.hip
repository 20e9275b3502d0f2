// Exact cluster index for a sublinear lookup.
//
// Build: K centres start at evenly spaced cache rows; `iters` Lloyd
// iterations over an evenly strided sample of the rows (about 512 per
// cluster) assign each sampled row to its nearest centre (x . mu_c on the
// matrix cores, centre_mfma_kernel) and move each centre to the float64
// mean of its live sampled rows, summed per cluster in sample order after a
// stable sort of the sample by cluster (so a build does not depend on
// scheduling); the final assignment covers every row.  After the final
// assignment a stable radix sort by cluster gives the row order, the
// cluster offsets come from the counts, and
// R_c = max over live members of ||z_i - mu_c|| + r_i (widened so that the
// re-check's boundary band is covered) is taken in float64 and rounded up to
// float32.  The indexed rows are copied into a cluster-ordered cache.  Any
// partition gives exact answers; the iterations only make the clusters
// tight.
//
// Query plan: for every query the clusters with ||q - mu_c|| < R_c (tested
// on the float16 matrix cores with a rigorous slack, so no such cluster is
// missed); for every cluster the list of queries that need it; and work
// items pairing a block of a cluster's list with a chunk of its rows, which
// the fused lookup kernel scans through the list.
#include <limits.h>

#include "lc_common.hpp"
#include "lc_index.hpp"
#include "lc_sort.hpp"

namespace lc {

constexpr int kCr = 64;              // rows per block (4 waves x 16)
constexpr int64_t kSampleRows = 512; // rows per cluster the Lloyd iterations sample
constexpr int kCc = 64;              // centres per chunk (4 column tiles of 16)
constexpr int kCk = 64;              // features per LDS stage
constexpr int kCs = kCk + 4;         // floats per LDS row (padding spreads the banks)

__device__ __forceinline__ float stored_value(const void* z, int store, int64_t i, int d, int k) {
  if (store == LIPCACHE_BF16) return bf16_to_f32(static_cast<const uint16_t*>(z)[i * d + k]);
  return static_cast<const float*>(z)[i * d + k];
}

__device__ __forceinline__ f32x4 stored_x4(const void* z, int store, int64_t i, int d, int k) {
  if (store == LIPCACHE_BF16) {
    const uint2 h = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(z) + i * d + k);
    return f32x4{bf16_to_f32(static_cast<uint16_t>(h.x & 0xffffu)), bf16_to_f32(static_cast<uint16_t>(h.x >> 16)),
                 bf16_to_f32(static_cast<uint16_t>(h.y & 0xffffu)), bf16_to_f32(static_cast<uint16_t>(h.y >> 16))};
  }
  return *reinterpret_cast<const f32x4*>(static_cast<const float*>(z) + i * d + k);
}

// ||x||^2 in float64 of n rows (one wave per row).
__global__ void row_norm_kernel(const void* __restrict__ x, int store, int64_t n, int d, double* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (i >= n) return;
  double s = 0.0;
  for (int k = lane_id(); k < d; k += kWave) {
    const double v = static_cast<double>(stored_value(x, store, i, d, k));
    s = __builtin_fma(v, v, s);
  }
  s = wave_sum(s);
  if (lane_id() == 0) out[i] = s;
}

// Rows x (n of them: rows j * stride of the array, float32 or bf16 storage)
// against K centres mu_c, on the
// matrix cores: g = x . mu_c by v_mfma_f32_16x16x4_f32 (float32 products
// and sums), then in float64 the score ||mu_c||^2 - 2 g, which orders the
// centres like ||x - mu_c||^2.
//  - nearest[r] (optional): the centre of least score (ties: lower index)
//    among the usable ones (bound[c] > 0; all when bound is null);
//  - mask (optional): bit c of row r when ||x||^2 + score < R_c^2 + slack.
//    The float32 dot product is off by at most about (d + 1) 2^-24 ||x|| ||mu||
//    <= (d + 1) 2^-24 (||x||^2 + ||mu||^2) / 2, so with
//    slack = slack_rel (||x||^2 + ||mu||^2), slack_rel = 2 (d + 2) 2^-24, and a
//    2^-50 R_c^2 term for the rounding of R_c^2, every cluster with
//    ||x - mu_c|| < R_c sets its bit.
// Block: 4 waves, 64 rows; each wave owns 16 rows and all 64 centres of a
// chunk (4 accumulator tiles); rows and centres pass through LDS in stages
// of 64 features.  blockIdx.y splits the chunks into groups (only with
// nearest == nullptr: the mask bits of different centres are independent).
__global__ __launch_bounds__(256) void centre_mfma_kernel(const void* __restrict__ rows, int store, int64_t n,
                                                          int64_t stride, int d,
                                                          const float* __restrict__ centres,
                                                          const double* __restrict__ cnorm, int K,
                                                          const double* __restrict__ rnorm,
                                                          const float* __restrict__ bound, double slack_rel,
                                                          uint32_t* __restrict__ mask,
                                                          uint32_t* __restrict__ nearest) {
  __shared__ __attribute__((aligned(16))) float xs[kCr * kCs];
  __shared__ __attribute__((aligned(16))) float cs[kCc * kCs];
  const int t = static_cast<int>(threadIdx.x);
  const int lane = lane_id(), w = t / kWave;
  const int m16 = lane & 15, g = lane >> 4;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kCr;
  const int words = (K + 31) / 32;
  double bs[4], qn[4];
  int bi[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int64_t row = r0 + w * 16 + 4 * g + v;
    bs[v] = __builtin_inf();
    bi[v] = INT_MAX;
    qn[v] = (rnorm && row < n) ? rnorm[row] : 0.0;
  }
  const int chunks = (K + kCc - 1) / kCc;
  const int per = (chunks + static_cast<int>(gridDim.y) - 1) / static_cast<int>(gridDim.y);
  const int c_begin = static_cast<int>(blockIdx.y) * per * kCc;
  const int c_end = c_begin + per * kCc < K ? c_begin + per * kCc : K;
  for (int c0 = c_begin; c0 < c_end; c0 += kCc) {
    f32x4 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < d; k0 += kCk) {
      __syncthreads();
      for (int e = t; e < kCr * kCk / 4; e += 256) {
        const int rr = e / (kCk / 4), k4 = 4 * (e % (kCk / 4));
        const bool kin = k0 + k4 < d;
        const int64_t row = r0 + rr;
        const int c = c0 + rr;
        f32x4 xv = f32x4{0.f, 0.f, 0.f, 0.f}, cv = f32x4{0.f, 0.f, 0.f, 0.f};
        if (kin && row < n) xv = stored_x4(rows, store, row * stride, d, k0 + k4);
        if (kin && c < K) cv = *reinterpret_cast<const f32x4*>(centres + static_cast<int64_t>(c) * d + k0 + k4);
        *reinterpret_cast<f32x4*>(&xs[rr * kCs + k4]) = xv;
        *reinterpret_cast<f32x4*>(&cs[rr * kCs + k4]) = cv;
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < kCk; kk += 16) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(&xs[(w * 16 + m16) * kCs + kk + 4 * g]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 b = *reinterpret_cast<const f32x4*>(&cs[(j * 16 + m16) * kCs + kk + 4 * g]);
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], acc[j], 0, 0, 0);
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], acc[j], 0, 0, 0);
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], acc[j], 0, 0, 0);
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], acc[j], 0, 0, 0);
        }
      }
    }
    // lane (m16, g) holds rows 4g + v of the wave's 16 and centre 16 j + m16
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = c0 + 16 * j + m16;
      if (c >= K) continue;
      const float R = bound ? bound[c] : 1.0f;
      if (!(R > 0.0f)) continue;
      const double cn = cnorm[c];
      const double R2 = static_cast<double>(R) * static_cast<double>(R);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const double score = cn - 2.0 * static_cast<double>(acc[j][v]);
        if (score < bs[v] || (score == bs[v] && c < bi[v])) {
          bs[v] = score;
          bi[v] = c;
        }
        if (mask) {
          const int64_t row = r0 + w * 16 + 4 * g + v;
          if (row < n && qn[v] + score < R2 * (1.0 + 0x1p-50) + slack_rel * (qn[v] + cn))
            atomicOr(&mask[row * words + c / 32], 1u << (c % 32));
        }
      }
    }
  }
  // least score over the 16 lanes that share g (same rows)
#pragma unroll
  for (int v = 0; v < 4; ++v) {
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) {
      const double os = __shfl_xor(bs[v], off, kWave);
      const int oi = __shfl_xor(bi[v], off, kWave);
      if (os < bs[v] || (os == bs[v] && oi < bi[v])) {
        bs[v] = os;
        bi[v] = oi;
      }
    }
    const int64_t row = r0 + w * 16 + 4 * g + v;
    if (nearest && m16 == 0 && row < n) nearest[row] = bi[v] == INT_MAX ? 0u : static_cast<uint32_t>(bi[v]);
  }
}

// Nearest centre of each row for the build, on the 16-bit matrix cores:
// x.mu_c by v_mfma_f32_16x16x32_f16 from the float16 image of the rows and
// float16-rounded centres (or v_mfma_f32_16x16x32_bf16 from a bf16 store
// without an image and bf16-rounded centres), then ||mu_c||^2 - 2 x.mu_c in
// float64; ties go to the lower index.  Any assignment keeps the index
// exact (R_c is taken from the rows a cluster receives), so the rounding only
// affects how tight the clusters are.  Rows are j * stride, j < n.
// Block: 4 waves x 16 rows; a wave keeps its rows' A operands for the whole
// feature range in registers (KS k-steps of 32, features past d read as 0)
// and sweeps the centres in chunks staged in LDS (rows padded by 16 bytes so
// the 16 lanes of one k-chunk read distinct banks).  Lane (m16, g) supplies
// row m16, features 32 s + 8 g .. + 7 of step s, and holds the products of
// rows 4 g .. 4 g + 3 with centre m16 of each 16-centre tile.
template <int KS>
struct AssignTraits {
  static constexpr int kChunk = KS <= 8 ? 64 : (KS <= 16 ? 32 : 16);  // centres per LDS chunk
  static constexpr int kRowBytes = KS * 64 + 16;                       // padded 16-bit row
};

__device__ __forceinline__ u32x4 load16_or_zero(const uint16_t* base, bool ok) {
  return ok ? *reinterpret_cast<const u32x4*>(base) : u32x4{0u, 0u, 0u, 0u};
}

template <int KS, bool F16>
__global__ __launch_bounds__(256) void assign16_kernel(const uint16_t* __restrict__ rows, int64_t n,
                                                          int64_t stride, int d,
                                                          const uint16_t* __restrict__ centres16,
                                                          const double* __restrict__ cnorm, int K,
                                                          uint32_t* __restrict__ nearest) {
  using T = AssignTraits<KS>;
  constexpr int kTiles = T::kChunk / 16;
  __shared__ __attribute__((aligned(16))) unsigned char cs[T::kChunk * T::kRowBytes];
  const int t = static_cast<int>(threadIdx.x);
  const int lane = lane_id(), w = t / kWave;
  const int m16 = lane & 15, g = lane >> 4;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kCr;
  // this lane's row of the wave's 16 (clamped; rows past n are never written)
  int64_t ra = r0 + w * 16 + m16;
  ra = ra < n ? ra : n - 1;
  const uint16_t* arow = rows + ra * stride * d;
  u32x4 a[KS];
#pragma unroll
  for (int st = 0; st < KS; ++st) {
    const int k0 = 32 * st + 8 * g;
    a[st] = load16_or_zero(arow + k0, k0 < d);
  }
  double bs[4];
  int bi[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    bs[v] = __builtin_inf();
    bi[v] = INT_MAX;
  }
  constexpr int kChunksPerRow = 4 * KS;  // 16-byte chunks of a row (without the padding)
  for (int c0 = 0; c0 < K; c0 += T::kChunk) {
    __syncthreads();
    for (int e = t; e < T::kChunk * kChunksPerRow; e += 256) {
      const int cr = e / kChunksPerRow, q = e % kChunksPerRow;
      const int c = c0 + cr, k0 = 8 * q;
      const u32x4 v = load16_or_zero(centres16 + static_cast<int64_t>(c < K ? c : 0) * d + k0, c < K && k0 < d);
      *reinterpret_cast<u32x4*>(cs + cr * T::kRowBytes + q * 16) = v;
    }
    __syncthreads();
    f32x4 acc[kTiles];
#pragma unroll
    for (int j = 0; j < kTiles; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < KS; ++st) {
#pragma unroll
      for (int j = 0; j < kTiles; ++j) {
        const u32x4 b = *reinterpret_cast<const u32x4*>(cs + (16 * j + m16) * T::kRowBytes + (4 * st + g) * 16);
        if constexpr (F16) {
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a[st]),
                                                          __builtin_bit_cast(f16x8, b), acc[j], 0, 0, 0);
        } else {
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[st]),
                                                           __builtin_bit_cast(bf16x8, b), acc[j], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kTiles; ++j) {
      const int c = c0 + 16 * j + m16;
      if (c >= K) continue;
      const double cn = cnorm[c];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const double score = cn - 2.0 * static_cast<double>(acc[j][v]);
        if (score < bs[v] || (score == bs[v] && c < bi[v])) {
          bs[v] = score;
          bi[v] = c;
        }
      }
    }
  }
  // least score over the 16 lanes that share g (same rows)
#pragma unroll
  for (int v = 0; v < 4; ++v) {
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) {
      const double os = __shfl_xor(bs[v], off, kWave);
      const int oi = __shfl_xor(bi[v], off, kWave);
      if (os < bs[v] || (os == bs[v] && oi < bi[v])) {
        bs[v] = os;
        bi[v] = oi;
      }
    }
    const int64_t row = r0 + w * 16 + 4 * g + v;
    if (m16 == 0 && row < n) nearest[row] = bi[v] == INT_MAX ? 0u : static_cast<uint32_t>(bi[v]);
  }
}

// 16-bit copy of the float32 centres: float16 (clamped, nearest even) or
// bf16 (nearest even), the element type of the rows they meet.
__global__ void centre16_kernel(const float* __restrict__ c, int64_t n, int f16, uint16_t* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) out[i] = f16 ? f16_bits(c[i]) : bf16_bits(c[i]);
}

// Assignment of rows j * stride (j < n) for the build: the 16-bit kernel on
// the float16 image, else on a bf16 store, else the float32 one.
inline void launch_assign(const lipcache_cache* c, int64_t n, int64_t stride, int d, const float* centres,
                          uint16_t* centres16, const double* cnorm, int K, uint32_t* nearest, hipStream_t s) {
  const bool f16 = c->zimg != nullptr;
  const uint16_t* rows16 = f16 ? static_cast<const uint16_t*>(c->zimg)
                               : (c->store_dtype == LIPCACHE_BF16 ? static_cast<const uint16_t*>(c->z) : nullptr);
  const unsigned grid = static_cast<unsigned>((n + kCr - 1) / kCr);
  if (!rows16) {
    hipLaunchKernelGGL(centre_mfma_kernel, dim3(grid), dim3(256), 0, s, c->z, c->store_dtype, n, stride, d, centres,
                       cnorm, K, nullptr, nullptr, 0.0, nullptr, nearest);
    return;
  }
  const int64_t kd = static_cast<int64_t>(K) * d;
  hipLaunchKernelGGL(centre16_kernel, dim3(static_cast<unsigned>((kd + 255) / 256)), dim3(256), 0, s, centres, kd,
                     f16 ? 1 : 0, centres16);
  int ks = 1;
  while (ks * 32 < d) ks *= 2;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), 0, s, rows16, n, stride, d, centres16, cnorm, K, nearest);
  };
#define LC_ASSIGN(KS_)                          \
  if (f16) {                                    \
    go(assign16_kernel<KS_, true>);             \
  } else {                                      \
    go(assign16_kernel<KS_, false>);            \
  }
  switch (ks) {
    case 1: LC_ASSIGN(1) break;
    case 2: LC_ASSIGN(2) break;
    case 4: LC_ASSIGN(4) break;
    case 8: LC_ASSIGN(8) break;
    case 16: LC_ASSIGN(16) break;
    default: LC_ASSIGN(32) break;
  }
#undef LC_ASSIGN
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

// Lloyd update of cluster c (one workgroup): mu_c = the float64 mean of the
// live rows among its sampled rows order[off[c] .. off[c + 1]) (sample
// index j is row j * stride), added in that order, so the centres do not
// depend on scheduling; a cluster without a live sampled row keeps its
// centre.  Thread t owns features t + 256 q, q < Q = ceil(d / 256); rows are
// taken 64 / Q at a time and their loads are unconditional (a dead or
// missing row reads row 0, a feature past d reads feature 0), so a batch's
// loads are all in flight before its sums.
template <int STORE, int Q>
__global__ __launch_bounds__(256) void centre_mean_kernel(const void* __restrict__ z, const float* __restrict__ r,
                                                          int d, int64_t stride, const uint32_t* __restrict__ order,
                                                          const int64_t* __restrict__ off,
                                                          float* __restrict__ centres) {
  constexpr int kBatch = 64 / Q;
  __shared__ int64_t rows[kBatch];
  const int c = static_cast<int>(blockIdx.x);
  const int t = static_cast<int>(threadIdx.x);
  const int64_t b = off[c], e = off[c + 1];
  double s[Q];
  int kq[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    s[q] = 0.0;
    kq[q] = t + 256 * q < d ? t + 256 * q : 0;
  }
  int64_t live = 0;
  for (int64_t j0 = b; j0 < e; j0 += kBatch) {
    const int m = e - j0 < kBatch ? static_cast<int>(e - j0) : kBatch;
    __syncthreads();  // the previous batch's row list is consumed
    if (t < kBatch) {
      int64_t i = -1;
      if (t < m) {
        i = static_cast<int64_t>(order[j0 + t]) * stride;
        if (!(r[i] > 0.0f)) i = -1;
      }
      rows[t] = i;
    }
    __syncthreads();
    float v[kBatch][Q];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int64_t i = rows[u];
      const int64_t base = (i >= 0 ? i : 0) * d;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        if constexpr (STORE == LIPCACHE_BF16) {
          v[u][q] = bf16_to_f32(static_cast<const uint16_t*>(z)[base + kq[q]]);
        } else {
          v[u][q] = static_cast<const float*>(z)[base + kq[q]];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (rows[u] >= 0) {
        ++live;
#pragma unroll
        for (int q = 0; q < Q; ++q) s[q] += static_cast<double>(v[u][q]);
      }
    }
  }
  if (live == 0) return;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int k = t + 256 * q;
    if (k < d) centres[static_cast<int64_t>(c) * d + k] = static_cast<float>(s[q] / static_cast<double>(live));
  }
}

template <int STORE>
inline void launch_centre_mean(int d, unsigned K, hipStream_t s, const void* z, const float* r, int64_t stride,
                               const uint32_t* order, const int64_t* off, float* centres) {
  const int q = (d + 255) / 256;
  if (q <= 1) {
    hipLaunchKernelGGL((centre_mean_kernel<STORE, 1>), dim3(K), dim3(256), 0, s, z, r, d, stride, order, off, centres);
  } else if (q == 2) {
    hipLaunchKernelGGL((centre_mean_kernel<STORE, 2>), dim3(K), dim3(256), 0, s, z, r, d, stride, order, off, centres);
  } else if (q == 3) {
    hipLaunchKernelGGL((centre_mean_kernel<STORE, 3>), dim3(K), dim3(256), 0, s, z, r, d, stride, order, off, centres);
  } else {
    hipLaunchKernelGGL((centre_mean_kernel<STORE, 4>), dim3(K), dim3(256), 0, s, z, r, d, stride, order, off, centres);
  }
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

// Rows per cluster: a workgroup counts 4096 rows in LDS and flushes one
// atomic per cluster it saw (clusters from kCountLds on count globally).
constexpr int kCountLds = 4096;

__global__ __launch_bounds__(256) void count_kernel(const uint32_t* __restrict__ assign, int64_t n, int K,
                                                    uint32_t* __restrict__ cnt) {
  __shared__ uint32_t h[kCountLds];
  for (int c = threadIdx.x; c < K && c < kCountLds; c += 256) h[c] = 0u;
  __syncthreads();
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * 4096;
  for (int64_t i = i0 + threadIdx.x; i < i0 + 4096 && i < n; i += 256) {
    const uint32_t c = assign[i];
    if (c < static_cast<uint32_t>(kCountLds)) {
      atomicAdd(&h[c], 1u);
    } else {
      atomicAdd(&cnt[c], 1u);
    }
  }
  __syncthreads();
  for (int c = threadIdx.x; c < K && c < kCountLds; c += 256)
    if (h[c]) atomicAdd(&cnt[c], h[c]);
}

// Sorted rows j0 .. j0+7 (one wave): copy cache rows perm[j] and raise R_c.
// Lanes 0..7 move the per-row scalars; the feature rows move as 16-byte
// (f32) or 8-byte (bf16, float16 image) vectors, the eight rows' loads issued
// before their stores.  The rows are in cluster order, so the wave keeps a
// running max of ||z_j - mu_c|| + r_j and flushes one atomic per cluster
// it covers instead of one per row.
constexpr int kReorderRows = 8;

__device__ __forceinline__ double diff2_4(float4 v, float4 m) {
  double p = static_cast<double>(v.x) - static_cast<double>(m.x);
  double acc = p * p;
  p = static_cast<double>(v.y) - static_cast<double>(m.y);
  acc = __builtin_fma(p, p, acc);
  p = static_cast<double>(v.z) - static_cast<double>(m.z);
  acc = __builtin_fma(p, p, acc);
  p = static_cast<double>(v.w) - static_cast<double>(m.w);
  return __builtin_fma(p, p, acc);
}

__device__ __forceinline__ float4 bf16x4_to_f32(uint2 h) {
  return make_float4(bf16_to_f32(static_cast<uint16_t>(h.x)), bf16_to_f32(static_cast<uint16_t>(h.x >> 16)),
                     bf16_to_f32(static_cast<uint16_t>(h.y)), bf16_to_f32(static_cast<uint16_t>(h.y >> 16)));
}

__device__ __forceinline__ uint2 f32x4_to_f16(float4 v) {
  return make_uint2(static_cast<uint32_t>(f16_bits(v.x)) | (static_cast<uint32_t>(f16_bits(v.y)) << 16),
                    static_cast<uint32_t>(f16_bits(v.z)) | (static_cast<uint32_t>(f16_bits(v.w)) << 16));
}

__global__ __launch_bounds__(256) void reorder_kernel(const lipcache_cache c, lipcache_cache out,
                                                      const uint32_t* __restrict__ order, int64_t n,
                                                      int64_t* __restrict__ perm,
                                                      const uint32_t* __restrict__ assign,
                                                      const float* __restrict__ centres,
                                                      unsigned long long* __restrict__ rbits) {
  constexpr int R = kReorderRows;
  const int64_t j0 = (static_cast<int64_t>(blockIdx.x) * (blockDim.x / kWave) + threadIdx.x / kWave) * R;
  if (j0 >= n) return;
  const int lane = lane_id();
  const int rows = n - j0 < R ? static_cast<int>(n - j0) : R;
  int64_t src_l = 0;
  uint32_t cl_l = 0;
  float r_l = 0.0f;
  if (lane < rows) {
    src_l = order[j0 + lane];
    cl_l = assign[src_l];
    r_l = c.r[src_l];
    perm[j0 + lane] = src_l;
    out.r[j0 + lane] = r_l;
    out.label[j0 + lane] = c.label[src_l];
    out.norm2[j0 + lane] = c.norm2[src_l];
  }
  int64_t src[R];
  uint32_t cl[R];
#pragma unroll
  for (int t = 0; t < R; ++t) {
    // rows past the end repeat the last row's loads; their stores are skipped
    const int u = t < rows ? t : rows - 1;
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(src_l)), u);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(src_l >> 32)), u);
    src[t] = static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
    cl[t] = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(cl_l), u));
  }
  const int d = c.d;
  const int d4 = d >> 2;
  const float4* __restrict__ mu4 = reinterpret_cast<const float4*>(centres);
  double part[R];
#pragma unroll
  for (int t = 0; t < R; ++t) part[t] = 0.0;
  const uint2* __restrict__ is = static_cast<const uint2*>(c.zimg);
  uint2* __restrict__ io = static_cast<uint2*>(out.zimg);
  for (int k4 = lane; k4 < d4; k4 += kWave) {
    if (c.store_dtype == LIPCACHE_BF16) {
      const uint2* __restrict__ zs = static_cast<const uint2*>(c.z);
      uint2* __restrict__ zo = static_cast<uint2*>(out.z);
      uint2 v[R];
      uint2 im[R];
#pragma unroll
      for (int t = 0; t < R; ++t) v[t] = zs[src[t] * d4 + k4];
      if (io && is) {
#pragma unroll
        for (int t = 0; t < R; ++t) im[t] = is[src[t] * d4 + k4];
      } else if (io) {
#pragma unroll
        for (int t = 0; t < R; ++t) im[t] = f32x4_to_f16(bf16x4_to_f32(v[t]));
      }
#pragma unroll
      for (int t = 0; t < R; ++t) {
        if (t < rows) {
          zo[(j0 + t) * d4 + k4] = v[t];
          if (io) io[(j0 + t) * d4 + k4] = im[t];
          part[t] += diff2_4(bf16x4_to_f32(v[t]), mu4[static_cast<int64_t>(cl[t]) * d4 + k4]);
        }
      }
    } else {
      const float4* __restrict__ zs = static_cast<const float4*>(c.z);
      float4* __restrict__ zo = static_cast<float4*>(out.z);
      float4 v[R];
      uint2 im[R];
#pragma unroll
      for (int t = 0; t < R; ++t) v[t] = zs[src[t] * d4 + k4];
      if (io && is) {
#pragma unroll
        for (int t = 0; t < R; ++t) im[t] = is[src[t] * d4 + k4];
      } else if (io) {
#pragma unroll
        for (int t = 0; t < R; ++t) im[t] = f32x4_to_f16(v[t]);
      }
#pragma unroll
      for (int t = 0; t < R; ++t) {
        if (t < rows) {
          zo[(j0 + t) * d4 + k4] = v[t];
          if (io) io[(j0 + t) * d4 + k4] = im[t];
          part[t] += diff2_4(v[t], mu4[static_cast<int64_t>(cl[t]) * d4 + k4]);
        }
      }
    }
  }
  // per-row reach, folded into a running max per cluster (negative: none yet)
  double run = -1.0;
  uint32_t run_cl = cl[0];
#pragma unroll
  for (int t = 0; t < R; ++t) {
    if (t < rows) {
      const double d2 = wave_sum_dpp(part[t]);
      const float rr = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, r_l), t));
      if (cl[t] != run_cl) {
        if (run >= 0.0 && lane == 0) atomicMax(&rbits[run_cl], __builtin_bit_cast(unsigned long long, run));
        run = -1.0;
        run_cl = cl[t];
      }
      if (rr > 0.0f) {
        // the ball widened by 2^-16 r, so every pair inside the 1e-5 r band
        // of the re-check is also reached
        const double reach = __builtin_sqrt(d2) + static_cast<double>(rr) * (1.0 + 0x1p-16);
        run = reach > run ? reach : run;
      }
    }
  }
  if (run >= 0.0 && lane == 0) atomicMax(&rbits[run_cl], __builtin_bit_cast(unsigned long long, run));
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
  uint32_t* cnt;
  int64_t* coff;
  uint16_t* c16;  // 16-bit copy of the centres (16-bit assignment)
  unsigned long long* rbits;
  double* cnorm;
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
  w.cnt = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(K) * 4));
  w.coff = reinterpret_cast<int64_t*>(take(static_cast<size_t>(K + 1) * 8));
  w.c16 = reinterpret_cast<uint16_t*>(take(static_cast<size_t>(K) * d * 2));
  w.rbits = reinterpret_cast<unsigned long long*>(take(static_cast<size_t>(K) * 8));
  w.cnorm = reinterpret_cast<double*>(take(static_cast<size_t>(K) * 8));
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
// The per-cluster query lists.  A workgroup takes kPlanRows consecutive
// queries, whose mask words are contiguous: its threads read them coalesced
// (thread i takes words i, i + 256, ...), first summing each query's
// candidate count in LDS.  A query with more than kMaxCand candidate
// clusters joins list K, otherwise every candidate cluster's list.  Counts
// are gathered in LDS and flushed with one global atomic per list and
// workgroup (lists above kPlanLds fall back to global atomics).
constexpr int kPlanLds = 4096;
constexpr int kPlanRows = 128;

// Candidate counts of the workgroup's rows q0 .. q0 + rows - 1 into rc.
__device__ __forceinline__ void plan_row_counts(const uint32_t* __restrict__ mask, int words, int64_t q0, int rows,
                                                uint32_t* rc) {
  for (int i = threadIdx.x; i < rows; i += blockDim.x) rc[i] = 0u;
  __syncthreads();
  const uint32_t* base = mask + q0 * words;
  const int nw = rows * words;
  for (int i = threadIdx.x; i < nw; i += blockDim.x) {
    const uint32_t v = base[i];
    if (v) atomicAdd(&rc[i / words], static_cast<uint32_t>(__builtin_popcount(v)));
  }
  __syncthreads();
}

// Calls f(list, row) for every list entry of the workgroup's rows (any order).
template <typename F>
__device__ __forceinline__ void plan_entries(const uint32_t* __restrict__ mask, int words, int64_t q0, int rows,
                                             int K, const uint32_t* rc, F&& f) {
  const uint32_t* base = mask + q0 * words;
  const int nw = rows * words;
  for (int i = threadIdx.x; i < nw; i += blockDim.x) {
    const int row = i / words, wd = i - row * words;
    if (rc[row] > static_cast<uint32_t>(kMaxCand)) {
      if (wd == 0) f(K, row);
      continue;
    }
    uint32_t v = base[i];
    while (v) {
      f(32 * wd + __builtin_ctz(v), row);
      v &= v - 1u;
    }
  }
}

__global__ __launch_bounds__(256) void plan_count_kernel(const uint32_t* __restrict__ mask, int words, int64_t B,
                                                         int K, uint32_t* __restrict__ ccount) {
  __shared__ uint32_t h[kPlanLds];
  __shared__ uint32_t rc[kPlanRows];
  const int lists = K + 1;
  for (int c = threadIdx.x; c < lists && c < kPlanLds; c += 256) h[c] = 0u;
  const int64_t q0 = static_cast<int64_t>(blockIdx.x) * kPlanRows;
  const int rows = static_cast<int>(B - q0 < kPlanRows ? B - q0 : kPlanRows);
  plan_row_counts(mask, words, q0, rows, rc);  // (its barrier also publishes h)
  plan_entries(mask, words, q0, rows, K, rc, [&](int c, int) {
    if (c < kPlanLds) {
      atomicAdd(&h[c], 1u);
    } else {
      atomicAdd(&ccount[c], 1u);
    }
  });
  __syncthreads();
  for (int c = threadIdx.x; c < lists && c < kPlanLds; c += 256)
    if (h[c]) atomicAdd(&ccount[c], h[c]);
}

// Each workgroup reserves, per list, a range for its queries (one global
// atomic per list) and places them with LDS cursors.
__global__ __launch_bounds__(256) void plan_fill_kernel(const uint32_t* __restrict__ mask, int words, int64_t B,
                                                        int K, const int64_t* __restrict__ coff,
                                                        uint32_t* __restrict__ cfill, int32_t* __restrict__ qlist) {
  __shared__ uint32_t h[kPlanLds];
  __shared__ uint32_t base[kPlanLds];
  __shared__ uint32_t rc[kPlanRows];
  const int lists = K + 1;
  for (int c = threadIdx.x; c < lists && c < kPlanLds; c += 256) h[c] = 0u;
  const int64_t q0 = static_cast<int64_t>(blockIdx.x) * kPlanRows;
  const int rows = static_cast<int>(B - q0 < kPlanRows ? B - q0 : kPlanRows);
  plan_row_counts(mask, words, q0, rows, rc);
  plan_entries(mask, words, q0, rows, K, rc, [&](int c, int) {
    if (c < kPlanLds) atomicAdd(&h[c], 1u);
  });
  __syncthreads();
  for (int c = threadIdx.x; c < lists && c < kPlanLds; c += 256) {
    base[c] = h[c] ? atomicAdd(&cfill[c], h[c]) : 0u;
    h[c] = 0u;  // becomes the workgroup's cursor
  }
  __syncthreads();
  plan_entries(mask, words, q0, rows, K, rc, [&](int c, int row) {
    const uint32_t slot = c < kPlanLds ? base[c] + atomicAdd(&h[c], 1u) : atomicAdd(&cfill[c], 1u);
    qlist[coff[c] + slot] = static_cast<int32_t>(q0 + row);
  });
}

// Rows of list c: cluster c, or every indexed row for list K; cut into
// nearly equal chunks of at most item_rows (<= kItemRowsMax).
__device__ __forceinline__ void list_rows(const int64_t* offsets, int K, int64_t n_indexed, int c, int64_t item_rows,
                                          int64_t& e0, int64_t& e1, int64_t& chunks, int64_t& step) {
  e0 = c < K ? offsets[c] : 0;
  e1 = c < K ? offsets[c + 1] : n_indexed;
  chunks = e1 > e0 ? (e1 - e0 + item_rows - 1) / item_rows : 0;
  step = chunks ? (e1 - e0 + chunks - 1) / chunks : 1;
}

// Work-item shape: lists of 512 queries or more on average (over the K + 1
// lists) take the long shape (query blocks of qb_long, row chunks of at
// most kItemRowsMax), others the short one (qb_short, kItemRows).  Every
// kernel that cuts items takes the same decision from coff.
__device__ __forceinline__ bool plan_long(const int64_t* __restrict__ coff, int K) {
  return coff[K + 1] >= 512 * static_cast<int64_t>(K + 1);
}

// Items per list: (query blocks) x (row chunks); one thread per list.
__global__ void plan_item_count_kernel(const int64_t* __restrict__ coff, const int64_t* __restrict__ offsets, int K,
                                       int64_t n_indexed, int qb_short, int qb_long, uint32_t* __restrict__ icount,
                                       unsigned long long* __restrict__ counters) {
  const int c = static_cast<int>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (c > K) return;
  const bool lng = plan_long(coff, K);
  const int qblock = lng ? qb_long : qb_short;
  const int64_t nq = coff[c + 1] - coff[c];
  int64_t e0, e1, chunks, step;
  list_rows(offsets, K, n_indexed, c, lng ? kItemRowsMax : kItemRows, e0, e1, chunks, step);
  const int64_t qb = (nq + qblock - 1) / qblock;
  icount[c] = static_cast<uint32_t>(qb * chunks);
  if (nq > 0 && e1 > e0) atomicAdd(&counters[1], static_cast<unsigned long long>(nq * (e1 - e0)));
}

// Item i of the work list (list order; within a list, query blocks outer
// and row chunks inner), one thread per item over a grid-stride loop: its
// list is the last c with ioff[c] <= i.  counters[0] = the number of items,
// counters[3] = 1 for the long shape.
__global__ __launch_bounds__(256) void plan_items_kernel(const int64_t* __restrict__ coff,
                                                         const int64_t* __restrict__ offsets, int K, int64_t n_indexed,
                                                         int qb_short, int qb_long, const int64_t* __restrict__ ioff,
                                                         int64_t* __restrict__ items, int64_t capacity,
                                                         unsigned long long* __restrict__ counters) {
  const int64_t total = ioff[K + 1];
  const bool lng = plan_long(coff, K);
  const int qblock = lng ? qb_long : qb_short;
  const int64_t item_rows = lng ? kItemRowsMax : kItemRows;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    counters[0] = static_cast<unsigned long long>(total);
    counters[3] = lng ? 1ull : 0ull;
    if (total > capacity) counters[2] = 1ull;
  }
  if (total > capacity) return;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total; i += stride) {
    int lo = 0, hi = K;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (ioff[mid] <= i) {
        lo = mid;
      } else {
        hi = mid - 1;
      }
    }
    const int c = lo;
    int64_t e0, e1, chunks, step;
    list_rows(offsets, K, n_indexed, c, item_rows, e0, e1, chunks, step);
    const int64_t local = i - ioff[c];
    const int64_t qa = coff[c] + (local / chunks) * qblock;
    const int64_t qend = coff[c + 1];
    const int64_t ea = e0 + (local % chunks) * step;
    int64_t* it = items + 4 * i;
    it[0] = qa;
    it[1] = qa + qblock < qend ? qa + qblock : qend;
    it[2] = ea;
    it[3] = ea + step < e1 ? ea + step : e1;
  }
}

}  // namespace lc

using namespace lc;

namespace lc {

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }


size_t index_plan_layout(int64_t B, int d, int K, int64_t n_indexed, int qblock, IndexPlanWs* w, char* base) {
  (void)d;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off = align_up(off + bytes, 256);
    return p;
  };
  const int words = (K + 31) / 32;
  const int64_t maxc = K < kMaxCand ? K : kMaxCand;
  IndexPlanWs t{};
  t.mask = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(B) * words * 4));
  t.ccount = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(K + 1) * 4));
  t.cfill = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(K + 1) * 4));
  t.coff = reinterpret_cast<int64_t*>(take(static_cast<size_t>(K + 2) * 8));
  // every query sits in at most maxc lists, or in list K alone
  t.qcap = B * maxc;
  t.qlist = reinterpret_cast<int32_t*>(take(static_cast<size_t>(t.qcap > 0 ? t.qcap : 1) * 4));
  // sum over lists c of ceil(cnt_c / qblock) ceil(rows_c / R), with
  // sum cnt_c <= B maxc, cnt_c <= B, sum rows_c <= 2 n (list K holds all n)
  const int64_t R = kItemRows;
  t.capacity = cdiv(2 * B, qblock) * cdiv(n_indexed, R) + cdiv(B * maxc, qblock) + 2 * cdiv(n_indexed, R) + K + 4;
  t.items = reinterpret_cast<int64_t*>(take(static_cast<size_t>(t.capacity) * 4 * 8));
  t.icount = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(K + 1) * 4));
  t.ioff = reinterpret_cast<int64_t*>(take(static_cast<size_t>(K + 2) * 8));
  t.counters = reinterpret_cast<unsigned long long*>(take(64));
  t.qnorm = reinterpret_cast<double*>(take(static_cast<size_t>(B) * 8));
  t.cterm = reinterpret_cast<double*>(take(static_cast<size_t>(K) * 8));
  t.c16 = reinterpret_cast<uint16_t*>(take(static_cast<size_t>(K) * d * 2));
  if (w) *w = t;
  return off;
}

// Candidate test of the query plan.  The float16 dot product g_hat of a
// query and a centre, both rounded (u = 2^-11, sub-normal error eta =
// 2^-14, float32 accumulation gamma over d_pad + 2 terms), is within
//   E = k (||q||^2 + ||mu||^2) / 2 + e1 (||q|| + ||mu||) + e0,
//   k = 2u + u^2 + gamma (1 + u)^2, e1 = eta (1 + u)(1 + gamma) sqrt(d_pad),
//   e0 = (1 + gamma) d_pad eta^2,
// of q . mu, so ||q - mu_c|| < R_c implies ||q||^2 + ||mu||^2 - 2 g_hat <
// R_c^2 + 2E.  The test allows 4E, split into a query term and a centre term
//   X_q = (1 - 2k) ||q||^2 - 4 e1 ||q|| - 2 e0,
//   Y_c = (1 - 2k) ||mu||^2 - 4 e1 ||mu|| - 2 e0 - R_c^2 (1 + 2^-50),
// and c is a candidate of q iff X_q + Y_c < 2 g_hat (splitting the sum moves
// its float64 rounding by a few units in the last place of ||q||^2 +
// ||mu||^2, far inside the second 2E).  A query or centre of squared norm
// >= 2^30 (its float16 copy may not hold it) is a candidate of every live
// cluster (Y_c = -inf marks such a centre); a cluster with R_c <= 0 is
// nobody's (Y_c = NaN).
struct CandSlack {
  double k2;    // 2k
  double e1x4;  // 4 e1
  double e0x2;  // 2 e0
};

inline CandSlack cand_slack(int d) {
  int ks = 1;
  while (ks * 32 < d) ks *= 2;
  const double u = 1.0 / 2048.0, eta = 1.0 / 16384.0;
  const double dp = 32.0 * ks;
  const double nn = dp + 2.0;
  const double gam = nn / 16777216.0 / (1.0 - nn / 16777216.0);
  const double k = 2.0 * u + u * u + gam * (1.0 + u) * (1.0 + u);
  const double e1 = eta * (1.0 + u) * (1.0 + gam) * __builtin_sqrt(dp);
  const double e0 = (1.0 + gam) * dp * eta * eta;
  return CandSlack{2.0 * k, 4.0 * e1, 2.0 * e0};
}

// Plan set-up in one launch: blocks [0, zblocks) zero the list counts and
// cursors and the counters; the others take four centres each (one wave per
// centre): the float16 copy of the centre and its term Y_c.
__global__ __launch_bounds__(256) void plan_init_kernel(uint32_t* __restrict__ ccount, uint32_t* __restrict__ cfill,
                                                        int K, unsigned long long* __restrict__ counters,
                                                        unsigned zblocks, const float* __restrict__ centres,
                                                        const float* __restrict__ bound, int d, CandSlack sl,
                                                        double* __restrict__ cterm, uint16_t* __restrict__ c16) {
  if (blockIdx.x < zblocks) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i <= K) {
      ccount[i] = 0u;
      cfill[i] = 0u;
    }
    if (i < 8) counters[i] = 0ull;
    return;
  }
  const int64_t c = static_cast<int64_t>(blockIdx.x - zblocks) * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (c >= K) return;
  double s = 0.0;
  for (int k = lane_id(); k < d; k += kWave) {
    const float x = centres[c * d + k];
    s = __builtin_fma(static_cast<double>(x), static_cast<double>(x), s);
    c16[c * d + k] = f16_bits(x);
  }
  s = wave_sum(s);
  if (lane_id() == 0) {
    const float R = bound[c];
    double y = __builtin_nan("");
    if (R > 0.0f) {
      const double R2 = static_cast<double>(R) * static_cast<double>(R) * (1.0 + 0x1p-50);
      y = s >= kF16Range2 ? -__builtin_inf() : s - sl.k2 * s - sl.e1x4 * __builtin_sqrt(s) - sl.e0x2 - R2;
    }
    cterm[c] = y;
  }
}

// Candidate masks of the queries: bit c of word c / 32 of row r is set iff
// cluster c passes the test above for query r.  Block: 4 waves x kRT row
// tiles of 16 queries, their A operands in registers for the whole feature
// range; blockIdx.y takes a range of `cspan` centres (a multiple of 64, so
// no mask word is shared by two blocks), staged through LDS in chunks
// (padded rows, as in assign16_kernel), double-buffered: the next chunk's
// loads are in flight while the current one is multiplied.  Every word of
// every row is written once (no clearing, no atomics): for each 16-centre
// tile and each of its four rows a lane's pass bits are gathered by a wave
// ballot, and lane (v, g) keeps the half-words of row 4 g + v until its
// word is complete.
template <int KS>
struct CandTraits {
  static constexpr int kRT = KS <= 8 ? 2 : 1;                              // row tiles per wave
  static constexpr int kRows = 4 * kRT * 16;                               // queries per block
  static constexpr int kChunk = AssignTraits<KS>::kChunk;                  // centres per LDS chunk
  static constexpr int kRowBytes = AssignTraits<KS>::kRowBytes;
  static constexpr int kCPR = 4 * KS;                                      // 16-byte chunks per row
  static constexpr int kStage = kChunk * kCPR / 256;                       // loads per thread per chunk
};

template <int KS>
__global__ __launch_bounds__(256) void cand16_kernel(const uint16_t* __restrict__ zq16, const double* __restrict__ qnorm,
                                                     int64_t B, int d, const uint16_t* __restrict__ centres16,
                                                     const double* __restrict__ cterm, int K, int cspan, int words,
                                                     CandSlack sl, uint32_t* __restrict__ mask) {
  using T = CandTraits<KS>;
  constexpr int RT = T::kRT;
  constexpr int kTiles = T::kChunk / 16;
  static_assert(T::kStage >= 1 && T::kStage * 256 == T::kChunk * T::kCPR, "whole loads per thread");
  __shared__ __attribute__((aligned(16))) unsigned char cs[2][T::kChunk * T::kRowBytes];
  const int t = static_cast<int>(threadIdx.x);
  const int lane = lane_id(), w = t / kWave;
  const int m16 = lane & 15, g = lane >> 4;
  const int c_begin = static_cast<int>(blockIdx.y) * cspan;
  const int c_end = c_begin + cspan < K ? c_begin + cspan : K;
  if (c_begin >= c_end) return;  // whole block
  const int64_t rw = static_cast<int64_t>(blockIdx.x) * T::kRows + w * (RT * 16);  // the wave's first row
  u32x4 a[RT][KS];
  double X[RT][4];
  bool big[RT][4];
  uint32_t word[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    int64_t ra = rw + rt * 16 + m16;
    ra = ra < B ? ra : B - 1;
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      const int k0 = 32 * st + 8 * g;
      a[rt][st] = load16_or_zero(zq16 + ra * d + k0, k0 < d);
    }
    // query terms of this lane's accumulator rows 4 g + v
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t row = rw + rt * 16 + 4 * g + v;
      const double qn = row < B ? qnorm[row] : __builtin_nan("");
      X[rt][v] = qn - sl.k2 * qn - sl.e1x4 * __builtin_sqrt(qn) - sl.e0x2;
      big[rt][v] = qn >= kF16Range2 && qn < __builtin_inf();
    }
    word[rt] = 0u;
  }
  u32x4 stage[T::kStage];
  auto load_chunk16 = [&](int c0) {
#pragma unroll
    for (int i = 0; i < T::kStage; ++i) {
      const int e = t + 256 * i;
      const int c = c0 + e / T::kCPR, k0 = 8 * (e % T::kCPR);
      stage[i] = load16_or_zero(centres16 + static_cast<int64_t>(c < c_end ? c : 0) * d + k0, c < c_end && k0 < d);
    }
  };
  auto store_chunk16 = [&](unsigned char* buf) {
#pragma unroll
    for (int i = 0; i < T::kStage; ++i) {
      const int e = t + 256 * i;
      *reinterpret_cast<u32x4*>(buf + (e / T::kCPR) * T::kRowBytes + (e % T::kCPR) * 16) = stage[i];
    }
  };
  load_chunk16(c_begin);
  store_chunk16(cs[0]);
  __syncthreads();
  int cur = 0;
  for (int c0 = c_begin; c0 < c_end; c0 += T::kChunk) {
    const bool more = c0 + T::kChunk < c_end;
    if (more) load_chunk16(c0 + T::kChunk);  // in flight while this chunk is multiplied
    const unsigned char* buf = cs[cur];
#pragma unroll
    for (int j = 0; j < kTiles; ++j) {
      const int cbase = c0 + 16 * j;  // block-uniform
      if (cbase >= c_end) break;
      f32x4 acc[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < KS; ++st) {
        const u32x4 b = *reinterpret_cast<const u32x4*>(buf + (16 * j + m16) * T::kRowBytes + (4 * st + g) * 16);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a[rt][st]),
                                                           __builtin_bit_cast(f16x8, b), acc[rt], 0, 0, 0);
      }
      const int c = cbase + m16;
      const double Y = c < c_end ? cterm[c] : __builtin_nan("");
      const bool live = Y == Y;  // not NaN: a live cluster
      const bool ybig = Y == -__builtin_inf();
      const int sh = 16 * ((cbase >> 4) & 1);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const bool pass = live && (big[rt][v] || ybig || X[rt][v] + Y < 2.0 * static_cast<double>(acc[rt][v]));
          const unsigned long long bal = __ballot(pass);
          const uint32_t half = static_cast<uint32_t>(bal >> (16 * g)) & 0xFFFFu;
          if ((m16 & 3) == v) word[rt] |= half << sh;
        }
      }
      if (sh || cbase + 16 >= c_end) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const int64_t row = rw + rt * 16 + 4 * g + (m16 & 3);
          if (m16 < 4 && row < B) mask[row * words + (cbase >> 5)] = word[rt];
          word[rt] = 0u;
        }
      }
    }
    if (more) store_chunk16(cs[cur ^ 1]);  // that buffer was last read before the previous barrier
    __syncthreads();
    cur ^= 1;
  }
}

lipcache_status index_query_plan(const lipcache_index* idx, const uint16_t* zq16, int64_t B, int d, int qb_short,
                                 int qb_long, const IndexPlanWs& w, int64_t& n_items, int64_t& pairs, bool& long_items,
                                 hipStream_t s) {
  const int K = idx->K;
  const int words = (K + 31) / 32;
  const CandSlack sl = cand_slack(d);
  const int64_t zn = K + 1 > 8 ? K + 1 : 8;
  const int64_t zblocks = (zn + 255) / 256;
  const int64_t cblocks = (K + 3) / 4;
  hipLaunchKernelGGL(plan_init_kernel, dim3(static_cast<unsigned>(zblocks + cblocks)), dim3(256), 0, s, w.ccount,
                     w.cfill, K, w.counters, static_cast<unsigned>(zblocks), idx->centers, idx->bound, d, sl, w.cterm,
                     w.c16);
  LC_LAUNCHED();
  int ks = 1;
  while (ks * 32 < d) ks *= 2;
  auto go = [&](auto kern, int rows) {
    // about two blocks per CU: split the centres when the queries alone
    // give fewer
    const int64_t gx = (B + rows - 1) / rows;
    const int64_t chunks64 = (K + 63) / 64;
    int64_t gy = (512 + gx - 1) / gx;
    gy = gy < 1 ? 1 : (gy > chunks64 ? chunks64 : gy);
    const int cspan = static_cast<int>(((K + gy - 1) / gy + 63) / 64 * 64);
    gy = (K + cspan - 1) / cspan;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(gy)), dim3(256), 0, s, zq16,
                       w.qnorm, B, d, w.c16, w.cterm, K, cspan, words, sl, w.mask);
  };
#define LC_CAND(KS_) go(cand16_kernel<KS_>, CandTraits<KS_>::kRows)
  switch (ks) {
    case 1: LC_CAND(1); break;
    case 2: LC_CAND(2); break;
    case 4: LC_CAND(4); break;
    case 8: LC_CAND(8); break;
    case 16: LC_CAND(16); break;
    default: LC_CAND(32); break;
  }
#undef LC_CAND
  LC_LAUNCHED();
  const unsigned gq = static_cast<unsigned>((B + kPlanRows - 1) / kPlanRows);
  const unsigned gl = static_cast<unsigned>((K + 1 + 255) / 256);
  hipLaunchKernelGGL(plan_count_kernel, dim3(gq), dim3(256), 0, s, w.mask, words, B, K, w.ccount);
  LC_LAUNCHED();
  hipLaunchKernelGGL(exclusive_scan_kernel, dim3(1), dim3(1024), 0, s, w.ccount, K + 1, w.coff);
  LC_LAUNCHED();
  hipLaunchKernelGGL(plan_fill_kernel, dim3(gq), dim3(256), 0, s, w.mask, words, B, K, w.coff, w.cfill, w.qlist);
  LC_LAUNCHED();
  hipLaunchKernelGGL(plan_item_count_kernel, dim3(gl), dim3(256), 0, s, w.coff, idx->offsets, K, idx->n_indexed,
                     qb_short, qb_long, w.icount, w.counters);
  LC_LAUNCHED();
  hipLaunchKernelGGL(exclusive_scan_kernel, dim3(1), dim3(1024), 0, s, w.icount, K + 1, w.ioff);
  LC_LAUNCHED();
  hipLaunchKernelGGL(plan_items_kernel, dim3(256), dim3(256), 0, s, w.coff, idx->offsets, K, idx->n_indexed, qb_short,
                     qb_long, w.ioff, w.items, w.capacity, w.counters);
  LC_LAUNCHED();
  unsigned long long host[4] = {0ull, 0ull, 0ull, 0ull};
  LC_HIP(read_back(host, w.counters, sizeof(host), s));
  if (host[2] != 0ull) return LIPCACHE_EHIP;  // the capacity bound was wrong: never expected
  n_items = static_cast<int64_t>(host[0]);
  pairs = static_cast<int64_t>(host[1]);
  long_items = host[3] != 0ull;
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
  if ((reinterpret_cast<uintptr_t>(so.z) & 15u) != 0 || (reinterpret_cast<uintptr_t>(so.zimg) & 15u) != 0 ||
      (reinterpret_cast<uintptr_t>(c->z) & 15u) != 0 || (reinterpret_cast<uintptr_t>(c->zimg) & 7u) != 0 ||
      (reinterpret_cast<uintptr_t>(idx->centers) & 15u) != 0)
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
  const unsigned gk = static_cast<unsigned>((K + 3) / 4);
  // The iterations see every stride-th row (about kSampleRows per cluster);
  // the final assignment sees every row.
  const int64_t stride = n / (static_cast<int64_t>(K) * kSampleRows) > 1 ? n / (static_cast<int64_t>(K) * kSampleRows) : 1;
  const int64_t ns = (n + stride - 1) / stride;
  for (int it = 0; it < iters; ++it) {
    hipLaunchKernelGGL(row_norm_kernel, dim3(gk), dim3(256), 0, s, idx->centers, LIPCACHE_F32,
                       static_cast<int64_t>(K), d, w.cnorm);
    LC_LAUNCHED();
    launch_assign(c, ns, stride, d, idx->centers, w.c16, w.cnorm, K, w.assign, s);
    LC_LAUNCHED();
    // the sample in cluster order, then one workgroup per cluster
    hipLaunchKernelGGL(row_keys_kernel, dim3(static_cast<unsigned>((ns + 255) / 256)), dim3(256), 0, s, w.assign,
                       ns, w.keys[0], w.vals[0]);
    LC_LAUNCHED();
    int scur = 0;
    LC_HIP(radix_sort_u32(w.keys, w.vals, ns, sort_passes(K), w.hist, w.dsum, w.dbase, scur, s));
    hipLaunchKernelGGL(fill_u32_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0, s, w.cnt,
                       static_cast<int64_t>(K));
    LC_LAUNCHED();
    hipLaunchKernelGGL(count_kernel, dim3(static_cast<unsigned>((ns + 4095) / 4096)), dim3(256), 0, s, w.assign, ns,
                       K, w.cnt);
    LC_LAUNCHED();
    hipLaunchKernelGGL(exclusive_scan_kernel, dim3(1), dim3(1024), 0, s, w.cnt, K, w.coff);
    LC_LAUNCHED();
    if (c->store_dtype == LIPCACHE_BF16) {
      launch_centre_mean<LIPCACHE_BF16>(d, static_cast<unsigned>(K), s, c->z, c->r, stride, w.vals[scur], w.coff,
                                        idx->centers);
    } else {
      launch_centre_mean<LIPCACHE_F32>(d, static_cast<unsigned>(K), s, c->z, c->r, stride, w.vals[scur], w.coff,
                                       idx->centers);
    }
    LC_LAUNCHED();
  }
  hipLaunchKernelGGL(row_norm_kernel, dim3(gk), dim3(256), 0, s, idx->centers, LIPCACHE_F32, static_cast<int64_t>(K),
                     d, w.cnorm);
  LC_LAUNCHED();
  launch_assign(c, n, 1, d, idx->centers, w.c16, w.cnorm, K, w.assign, s);
  LC_LAUNCHED();
  hipLaunchKernelGGL(row_keys_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s, w.assign, n,
                     w.keys[0], w.vals[0]);
  LC_LAUNCHED();
  int cur = 0;
  LC_HIP(radix_sort_u32(w.keys, w.vals, n, sort_passes(K), w.hist, w.dsum, w.dbase, cur, s));
  hipLaunchKernelGGL(fill_u32_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0, s, w.cnt,
                     static_cast<int64_t>(K));
  LC_LAUNCHED();
  hipLaunchKernelGGL(count_kernel, dim3(static_cast<unsigned>((n + 4095) / 4096)), dim3(256), 0, s, w.assign, n, K,
                     w.cnt);
  LC_LAUNCHED();
  hipLaunchKernelGGL(exclusive_scan_kernel, dim3(1), dim3(1024), 0, s, w.cnt, K, idx->offsets);
  LC_LAUNCHED();
  hipLaunchKernelGGL(fill_u64x_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0, s, w.rbits,
                     static_cast<int64_t>(K), 0ull);
  LC_LAUNCHED();
  lipcache_cache out = idx->sorted;
  const int64_t rpb = 4 * kReorderRows;  // rows per 256-thread workgroup
  hipLaunchKernelGGL(reorder_kernel, dim3(static_cast<unsigned>((n + rpb - 1) / rpb)), dim3(256), 0, s, *c, out,
                     w.vals[cur], n, idx->perm, w.assign, idx->centers, w.rbits);
  LC_LAUNCHED();
  hipLaunchKernelGGL(bound_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0, s, w.rbits, K,
                     idx->bound);
  LC_LAUNCHED();
  idx->K = K;
  idx->n_indexed = n;
  idx->sorted.n = n;
  return LIPCACHE_OK;
}
