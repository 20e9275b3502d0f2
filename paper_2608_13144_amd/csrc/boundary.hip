// Reuse boundaries compared with the certified radius (Sec. 6) and the
// certified-consistency count.
//
// lipcache_boundary_radius writes a per-entry radius for one of
//   scaled     - factor * r_i (radius tightening keeps every hit inside the
//                certified ball when factor <= 1);
//   global     - factor for every entry (one nearest-neighbour threshold);
//   interclass - factor * 1/2 * min_{c != y_i} ||mu_{y_i} - mu_c||, with mu_c
//                the float64 mean of the cached features of label c (an
//                empirical radius from inter-class distance statistics).
// Entries whose certified radius is not positive get 0 (never hit).  The
// result is meant for lipcache_lookup on a copy of the cache descriptor whose
// `r` points at it: the features, labels and norms are shared.
//
// The class means are accumulated per workgroup in LDS (a slice of 64
// feature columns for up to 256 labels) and flushed with float64 atomics, so
// their last bits depend on the flush order (~1e-16 relative).
#include "lc_common.hpp"

namespace lc {

constexpr int kBndThreads = 256;
constexpr int kBndCols = 64;            // feature columns per workgroup
constexpr int kBndRows = 4096;          // entries per workgroup
constexpr int kBndLdsClasses = 192;     // LDS partial sums up to this many labels (96 KiB)

__global__ void bnd_fill_kernel(double* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.0;
}

__global__ void bnd_fill_u64_kernel(unsigned long long* __restrict__ p, int64_t n, unsigned long long v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void bnd_simple_kernel(const float* __restrict__ r, int64_t n, int mode, double factor,
                                  float* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float ri = r[i];
  const double v = mode == LIPCACHE_BOUNDARY_SCALED ? factor * static_cast<double>(ri) : factor;
  out[i] = ri > 0.0f ? static_cast<float>(v) : 0.0f;
}

__device__ __forceinline__ double feature(const void* z, int store, int64_t i, int d, int k) {
  if (store == LIPCACHE_BF16) return static_cast<double>(bf16_to_f32(static_cast<const uint16_t*>(z)[i * d + k]));
  return static_cast<double>(static_cast<const float*>(z)[i * d + k]);
}

// sum[c][k] += features of live entries with label c; cnt[c] += 1 (column
// slice 0 only).  Block (x = row range, y = column slice).
template <bool LDS>
__global__ __launch_bounds__(kBndThreads) void bnd_class_sum_kernel(const void* __restrict__ z, int store,
                                                                    const float* __restrict__ r,
                                                                    const int32_t* __restrict__ label, int64_t n,
                                                                    int d, int n_classes, double* __restrict__ sum,
                                                                    unsigned long long* __restrict__ cnt) {
  __shared__ double part[LDS ? kBndLdsClasses * kBndCols : 1];
  const int col = static_cast<int>(threadIdx.x) % kBndCols;
  const int sub = static_cast<int>(threadIdx.x) / kBndCols;  // 4 row lanes
  const int k = static_cast<int>(blockIdx.y) * kBndCols + col;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kBndRows;
  const int64_t r1 = r0 + kBndRows < n ? r0 + kBndRows : n;
  if constexpr (LDS) {
    for (int e = threadIdx.x; e < n_classes * kBndCols; e += kBndThreads) part[e] = 0.0;
    __syncthreads();
  }
  for (int64_t i = r0 + sub; i < r1; i += kBndThreads / kBndCols) {
    const int c = label[i];
    if (!(r[i] > 0.0f) || c < 0 || c >= n_classes) continue;
    if (k < d) {
      const double v = feature(z, store, i, d, k);
      if constexpr (LDS) {
        atomicAdd(&part[c * kBndCols + col], v);
      } else {
        atomicAdd(&sum[static_cast<int64_t>(c) * d + k], v);
      }
    }
    if (blockIdx.y == 0 && col == 0) atomicAdd(&cnt[c], 1ull);
  }
  if constexpr (LDS) {
    __syncthreads();
    for (int e = threadIdx.x; e < n_classes * kBndCols; e += kBndThreads) {
      const int c = e / kBndCols, cc = e % kBndCols;
      const int kk = static_cast<int>(blockIdx.y) * kBndCols + cc;
      if (kk < d && part[e] != 0.0) atomicAdd(&sum[static_cast<int64_t>(c) * d + kk], part[e]);
    }
  }
}

// half[c] bits (atomic min over o of ||mu_c - mu_o||^2 as float64 bits, >= 0);
// one thread per ordered pair (c, o), c != o, both present.
__global__ void bnd_pair_kernel(const double* __restrict__ sum, const unsigned long long* __restrict__ cnt,
                                int n_classes, int d, unsigned long long* __restrict__ best) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(n_classes) * n_classes) return;
  const int c = static_cast<int>(t / n_classes), o = static_cast<int>(t % n_classes);
  if (c == o || cnt[c] == 0 || cnt[o] == 0) return;
  const double nc = static_cast<double>(cnt[c]), no = static_cast<double>(cnt[o]);
  double acc = 0.0;
  for (int k = 0; k < d; ++k) {
    const double diff = sum[static_cast<int64_t>(c) * d + k] / nc - sum[static_cast<int64_t>(o) * d + k] / no;
    acc = __builtin_fma(diff, diff, acc);
  }
  atomicMin(&best[c], __builtin_bit_cast(unsigned long long, acc));
}

__global__ void bnd_interclass_kernel(const float* __restrict__ r, const int32_t* __restrict__ label, int64_t n,
                                      int n_classes, double factor, const unsigned long long* __restrict__ best,
                                      float* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int c = label[i];
  float v = 0.0f;
  if (r[i] > 0.0f && c >= 0 && c < n_classes) {
    const unsigned long long b = best[c];
    v = b == ~0ull ? __builtin_inff()
                   : static_cast<float>(factor * (0.5 * __builtin_sqrt(__builtin_bit_cast(double, b))));
  }
  out[i] = v;
}

// counts[0] += hits (lookup label != MISS), counts[1] += hits whose label is
// the head's own label at the query.
__global__ __launch_bounds__(256) void consistency_kernel(const int32_t* __restrict__ lk,
                                                          const int32_t* __restrict__ head, int64_t B,
                                                          unsigned long long* __restrict__ counts) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const bool hit = i < B && lk[i] != LIPCACHE_MISS;
  const bool ok = hit && lk[i] == head[i];
  const unsigned long long bh = __ballot(hit), bo = __ballot(ok);
  if (lane_id() == 0) {
    if (bh) atomicAdd(&counts[0], static_cast<unsigned long long>(__builtin_popcountll(bh)));
    if (bo) atomicAdd(&counts[1], static_cast<unsigned long long>(__builtin_popcountll(bo)));
  }
}

}  // namespace lc

using namespace lc;

extern "C" size_t lipcache_boundary_radius_workspace_bytes(int32_t d, int32_t n_classes) {
  if (d < 1 || n_classes < 0) return 0;
  const size_t c = static_cast<size_t>(n_classes > 0 ? n_classes : 1);
  return align_up(c * static_cast<size_t>(d) * 8, 256) + 2 * align_up(c * 8, 256);
}

extern "C" lipcache_status lipcache_boundary_radius(const lipcache_cache* c, int32_t mode, double factor,
                                                    int32_t n_classes, float* r_out, void* ws, size_t ws_bytes,
                                                    lipcache_stream_t stream) {
  if (!c || !r_out) return LIPCACHE_EINVAL;
  if (c->d < 32 || c->d > 1024 || c->d % 32 != 0) return LIPCACHE_EINVAL;
  if (c->store_dtype != LIPCACHE_F32 && c->store_dtype != LIPCACHE_BF16) return LIPCACHE_EINVAL;
  if (c->n < 0 || c->n > c->capacity) return LIPCACHE_EINVAL;
  if (c->n > 0 && (!c->z || !c->r || !c->label)) return LIPCACHE_EINVAL;
  if (mode != LIPCACHE_BOUNDARY_SCALED && mode != LIPCACHE_BOUNDARY_GLOBAL && mode != LIPCACHE_BOUNDARY_INTERCLASS)
    return LIPCACHE_EINVAL;
  if (!(factor >= 0.0) || factor == __builtin_inf()) return LIPCACHE_EINVAL;
  if (mode == LIPCACHE_BOUNDARY_INTERCLASS && (n_classes < 1 || n_classes > 65536)) return LIPCACHE_EINVAL;
  if (mode == LIPCACHE_BOUNDARY_INTERCLASS) {
    const size_t need = lipcache_boundary_radius_workspace_bytes(c->d, n_classes);
    if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;
  }
  if (c->n == 0) return LIPCACHE_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int64_t n = c->n;
  const unsigned g = static_cast<unsigned>((n + 255) / 256);
  if (mode != LIPCACHE_BOUNDARY_INTERCLASS) {
    hipLaunchKernelGGL(bnd_simple_kernel, dim3(g), dim3(256), 0, s, c->r, n, mode, factor, r_out);
    LC_LAUNCHED();
    return LIPCACHE_OK;
  }
  const int d = c->d;
  char* base = static_cast<char*>(ws);
  const size_t sum_bytes = align_up(static_cast<size_t>(n_classes) * d * 8, 256);
  double* sum = reinterpret_cast<double*>(base);
  unsigned long long* cnt = reinterpret_cast<unsigned long long*>(base + sum_bytes);
  unsigned long long* best = reinterpret_cast<unsigned long long*>(base + sum_bytes +
                                                                   align_up(static_cast<size_t>(n_classes) * 8, 256));
  const int64_t cd = static_cast<int64_t>(n_classes) * d;
  hipLaunchKernelGGL(bnd_fill_kernel, dim3(static_cast<unsigned>((cd + 255) / 256)), dim3(256), 0, s, sum, cd);
  LC_LAUNCHED();
  const unsigned gc = static_cast<unsigned>((n_classes + 255) / 256);
  hipLaunchKernelGGL(bnd_fill_u64_kernel, dim3(gc), dim3(256), 0, s, cnt, static_cast<int64_t>(n_classes), 0ull);
  LC_LAUNCHED();
  hipLaunchKernelGGL(bnd_fill_u64_kernel, dim3(gc), dim3(256), 0, s, best, static_cast<int64_t>(n_classes), ~0ull);
  LC_LAUNCHED();
  const dim3 sg(static_cast<unsigned>((n + kBndRows - 1) / kBndRows), static_cast<unsigned>((d + kBndCols - 1) / kBndCols));
  if (n_classes <= kBndLdsClasses) {
    hipLaunchKernelGGL(bnd_class_sum_kernel<true>, sg, dim3(kBndThreads), 0, s, c->z, c->store_dtype, c->r, c->label,
                       n, d, n_classes, sum, cnt);
  } else {
    hipLaunchKernelGGL(bnd_class_sum_kernel<false>, sg, dim3(kBndThreads), 0, s, c->z, c->store_dtype, c->r, c->label,
                       n, d, n_classes, sum, cnt);
  }
  LC_LAUNCHED();
  const int64_t pairs = static_cast<int64_t>(n_classes) * n_classes;
  hipLaunchKernelGGL(bnd_pair_kernel, dim3(static_cast<unsigned>((pairs + 255) / 256)), dim3(256), 0, s, sum, cnt,
                     n_classes, d, best);
  LC_LAUNCHED();
  hipLaunchKernelGGL(bnd_interclass_kernel, dim3(g), dim3(256), 0, s, c->r, c->label, n, n_classes, factor, best,
                     r_out);
  LC_LAUNCHED();
  return LIPCACHE_OK;
}

extern "C" lipcache_status lipcache_consistency(const int32_t* lookup_label, const int32_t* head_label, int64_t B,
                                                uint64_t* counts, lipcache_stream_t stream) {
  if (B < 0 || !counts || (B > 0 && (!lookup_label || !head_label))) return LIPCACHE_EINVAL;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  unsigned long long* cc = reinterpret_cast<unsigned long long*>(counts);
  hipLaunchKernelGGL(bnd_fill_u64_kernel, dim3(1), dim3(64), 0, s, cc, 2, 0ull);
  LC_LAUNCHED();
  if (B == 0) return LIPCACHE_OK;
  hipLaunchKernelGGL(consistency_kernel, dim3(static_cast<unsigned>((B + 255) / 256)), dim3(256), 0, s, lookup_label,
                     head_label, B, cc);
  LC_LAUNCHED();
  return LIPCACHE_OK;
}
