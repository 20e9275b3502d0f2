// Write-back of missed samples into the feature cache (Sec. 4.4, Alg. 2;
// construction, Alg. 1).
//
// Rows are taken in ascending order (a stable compaction), so the same input
// always produces the same cache rows.  Three kernels:
//   count   - per 1024-row block, how many rows are selected;
//   scan    - one workgroup turns the block counts into block offsets and the
//             total (read back by the host for the all-or-nothing capacity
//             check: nothing is written to the cache before it passes);
//   scatter - each block ranks its selected rows with wave ballots and copies
//             them, one wave per row (coalesced), casting to the store dtype
//             and recomputing ||z||^2 of the stored values in float64.
#include "lc_common.hpp"

namespace lc {

constexpr int kInsBlock = 1024;
constexpr int kInsWaves = kInsBlock / kWave;

__device__ __forceinline__ bool selected(int64_t j, int64_t k, const float* r_src, const int32_t* sel) {
  if (j >= k) return false;
  const float r = r_src[j];
  if (!(r > 0.0f)) return false;
  return sel == nullptr || sel[j] == LIPCACHE_MISS;
}

__global__ __launch_bounds__(kInsBlock) void insert_count_kernel(const float* __restrict__ r_src,
                                                                 const int32_t* __restrict__ sel, int64_t k,
                                                                 int64_t* __restrict__ counts) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * kInsBlock + threadIdx.x;
  const int c = __syncthreads_count(selected(j, k, r_src, sel) ? 1 : 0);
  if (threadIdx.x == 0) counts[blockIdx.x] = c;
}

// Exclusive scan of the block counts (one workgroup, any number of blocks).
__global__ __launch_bounds__(kInsBlock) void insert_scan_kernel(const int64_t* __restrict__ counts, int64_t nblocks,
                                                                int64_t* __restrict__ offsets,
                                                                int64_t* __restrict__ total) {
  __shared__ int64_t buf[kInsBlock];
  int64_t running = 0;
  for (int64_t base = 0; base < nblocks; base += kInsBlock) {
    const int64_t i = base + threadIdx.x;
    const int64_t v = i < nblocks ? counts[i] : 0;
    buf[threadIdx.x] = v;
    __syncthreads();
    for (int off = 1; off < kInsBlock; off <<= 1) {  // Hillis-Steele inclusive scan
      const int64_t add = threadIdx.x >= static_cast<unsigned>(off) ? buf[threadIdx.x - off] : 0;
      __syncthreads();
      buf[threadIdx.x] += add;
      __syncthreads();
    }
    if (i < nblocks) offsets[i] = running + buf[threadIdx.x] - v;
    running += buf[kInsBlock - 1];
    __syncthreads();
  }
  if (threadIdx.x == 0) *total = running;
}

struct InsertParams {
  const float* z_src;
  const int32_t* label_src;
  const float* r_src;
  const int32_t* sel;
  int64_t k;
  const int64_t* offsets;
  void* cz;
  uint16_t* cimg;
  float* cr;
  int32_t* clabel;
  float* cnorm2;
  int64_t n0;
  int d;
  int store;
};

__global__ __launch_bounds__(kInsBlock) void insert_scatter_kernel(const InsertParams p) {
  __shared__ int wave_count[kInsWaves];
  __shared__ int src_local[kInsBlock];
  const int64_t j = static_cast<int64_t>(blockIdx.x) * kInsBlock + threadIdx.x;
  const bool take = selected(j, p.k, p.r_src, p.sel);
  const int lane = lane_id();
  const int wave = static_cast<int>(threadIdx.x) / kWave;
  const unsigned long long bal = __ballot(take);
  const int below = __builtin_popcountll(bal & ((1ull << lane) - 1ull));
  if (lane == 0) wave_count[wave] = __builtin_popcountll(bal);
  __syncthreads();
  int before = 0, total = 0;
  for (int w = 0; w < kInsWaves; ++w) {
    before += w < wave ? wave_count[w] : 0;
    total += wave_count[w];
  }
  if (take) src_local[before + below] = static_cast<int>(threadIdx.x);
  __syncthreads();

  const int64_t dst0 = p.n0 + p.offsets[blockIdx.x];
  for (int t = wave; t < total; t += kInsWaves) {
    const int64_t src = static_cast<int64_t>(blockIdx.x) * kInsBlock + src_local[t];
    const int64_t dst = dst0 + t;
    const float* zr = p.z_src + src * p.d;
    double s = 0.0;
    if (p.store == LIPCACHE_BF16) {
      uint16_t* out = static_cast<uint16_t*>(p.cz) + dst * p.d;
      for (int k = lane; k < p.d; k += kWave) {
        const uint16_t h = bf16_bits(zr[k]);
        out[k] = h;
        const double v = static_cast<double>(bf16_to_f32(h));
        s = __builtin_fma(v, v, s);
      }
    } else {
      float* out = static_cast<float*>(p.cz) + dst * p.d;
      uint16_t* img = p.cimg ? p.cimg + dst * p.d : nullptr;
      for (int k = lane; k < p.d; k += kWave) {
        const float f = zr[k];
        out[k] = f;
        if (img) img[k] = bf16_bits(f);
        s = __builtin_fma(static_cast<double>(f), static_cast<double>(f), s);
      }
    }
    s = wave_sum(s);
    if (lane == 0) {
      p.cnorm2[dst] = static_cast<float>(s);
      p.cr[dst] = p.r_src[src];
      p.clabel[dst] = p.label_src[src];
    }
  }
}

}  // namespace lc

using namespace lc;

extern "C" size_t lipcache_insert_workspace_bytes(int64_t k) {
  const int64_t nb = k > 0 ? (k + kInsBlock - 1) / kInsBlock : 1;
  return 2 * align_up(static_cast<size_t>(nb) * sizeof(int64_t), 256) + 256;
}

extern "C" lipcache_status lipcache_insert(lipcache_cache* c, const float* z_src, const int32_t* label_src,
                                           const float* r_src, const int32_t* miss_selector, int64_t k,
                                           int64_t* inserted, void* ws, size_t ws_bytes,
                                           lipcache_stream_t stream) {
  if (!c || k < 0) return LIPCACHE_EINVAL;
  if (c->d < 32 || c->d > 1024 || c->d % 32 != 0) return LIPCACHE_EINVAL;
  if (c->store_dtype != LIPCACHE_F32 && c->store_dtype != LIPCACHE_BF16) return LIPCACHE_EINVAL;
  if (c->n < 0 || c->capacity < 0 || c->n > c->capacity) return LIPCACHE_EINVAL;
  if (c->capacity > 0 && (!c->z || !c->r || !c->label || !c->norm2)) return LIPCACHE_EINVAL;
  if (k > 0 && (!z_src || !label_src || !r_src)) return LIPCACHE_EINVAL;
  if (k > (static_cast<int64_t>(1) << 40)) return LIPCACHE_EINVAL;
  const size_t need = lipcache_insert_workspace_bytes(k);
  if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;
  if (inserted) *inserted = 0;
  if (k == 0) return LIPCACHE_OK;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int64_t nb = (k + kInsBlock - 1) / kInsBlock;
  char* base = static_cast<char*>(ws);
  int64_t* counts = reinterpret_cast<int64_t*>(base);
  int64_t* offsets = reinterpret_cast<int64_t*>(base + align_up(static_cast<size_t>(nb) * 8, 256));
  int64_t* total = reinterpret_cast<int64_t*>(base + 2 * align_up(static_cast<size_t>(nb) * 8, 256));

  hipLaunchKernelGGL(insert_count_kernel, dim3(static_cast<unsigned>(nb)), dim3(kInsBlock), 0, s, r_src,
                     miss_selector, k, counts);
  LC_LAUNCHED();
  hipLaunchKernelGGL(insert_scan_kernel, dim3(1), dim3(kInsBlock), 0, s, counts, nb, offsets, total);
  LC_LAUNCHED();
  int64_t host_total = 0;
  LC_HIP(hipMemcpyAsync(&host_total, total, sizeof(host_total), hipMemcpyDeviceToHost, s));
  LC_HIP(hipStreamSynchronize(s));
  if (host_total < 0 || host_total > k) return LIPCACHE_EHIP;
  if (c->n + host_total > c->capacity) return LIPCACHE_ECAPACITY;
  if (host_total == 0) return LIPCACHE_OK;

  InsertParams p;
  p.z_src = z_src;
  p.label_src = label_src;
  p.r_src = r_src;
  p.sel = miss_selector;
  p.k = k;
  p.offsets = offsets;
  p.cz = c->z;
  p.cimg = c->store_dtype == LIPCACHE_F32 ? static_cast<uint16_t*>(c->zimg) : nullptr;
  p.cr = c->r;
  p.clabel = c->label;
  p.cnorm2 = c->norm2;
  p.n0 = c->n;
  p.d = c->d;
  p.store = c->store_dtype;
  hipLaunchKernelGGL(insert_scatter_kernel, dim3(static_cast<unsigned>(nb)), dim3(kInsBlock), 0, s, p);
  LC_LAUNCHED();
  c->n += host_total;
  if (inserted) *inserted = host_total;
  return LIPCACHE_OK;
}
