// Write-back of missed samples into the feature cache (Sec. 4.4, Alg. 2;
// construction, Alg. 1).
//
// Rows are taken in ascending order (a stable compaction), so the same input
// always produces the same cache rows.  Four kernels (a batch of at most
// 1024 rows runs count, scan and rank as one):
//   count   - per 1024-row block, how many rows are selected;
//   scan    - one workgroup turns the block counts into block offsets and the
//             total (read back by the host for the all-or-nothing capacity
//             check: nothing is written to the cache before it passes);
//   rank    - each block ranks its selected rows with wave ballots and writes
//             the source row of every destination row;
//   copy    - one wave per destination row over the whole chip, 16-byte
//             loads and stores, casting to the store dtype, writing the
//             float16 image of the stored values (when the cache keeps one)
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

// The block's selected rows in order: src_of[offset + t] = the t-th; returns
// how many the block selected (in every thread).
__device__ __forceinline__ int rank_block(int64_t j, bool take, int64_t offset, int64_t* __restrict__ src_of,
                                          int* wave_count) {
  const int lane = lane_id();
  const int wave = static_cast<int>(threadIdx.x) / kWave;
  const unsigned long long bal = __ballot(take);
  const int below = __builtin_popcountll(bal & ((1ull << lane) - 1ull));
  if (lane == 0) wave_count[wave] = __builtin_popcountll(bal);
  __syncthreads();
  int before = 0, all = 0;
  for (int w = 0; w < kInsWaves; ++w) {
    if (w < wave) before += wave_count[w];
    all += wave_count[w];
  }
  if (take) src_of[offset + before + below] = j;
  return all;
}

// src_of[offsets[block] + t] = the t-th selected row of the block.
__global__ __launch_bounds__(kInsBlock) void insert_rank_kernel(const float* __restrict__ r_src,
                                                                const int32_t* __restrict__ sel, int64_t k,
                                                                const int64_t* __restrict__ offsets,
                                                                int64_t* __restrict__ src_of) {
  __shared__ int wave_count[kInsWaves];
  const int64_t j = static_cast<int64_t>(blockIdx.x) * kInsBlock + threadIdx.x;
  rank_block(j, selected(j, k, r_src, sel), offsets[blockIdx.x], src_of, wave_count);
}

// k <= kInsBlock: count, scan and rank in one workgroup (its offset is 0,
// the total is its own count).
__global__ __launch_bounds__(kInsBlock) void insert_rank_one_kernel(const float* __restrict__ r_src,
                                                                    const int32_t* __restrict__ sel, int64_t k,
                                                                    int64_t* __restrict__ src_of,
                                                                    int64_t* __restrict__ total) {
  __shared__ int wave_count[kInsWaves];
  const int64_t j = threadIdx.x;
  const int all = rank_block(j, selected(j, k, r_src, sel), 0, src_of, wave_count);
  if (threadIdx.x == 0) *total = all;
}

struct InsertParams {
  const float* z_src;
  const int32_t* label_src;
  const float* r_src;
  const int64_t* src_of;
  int64_t count;
  void* cz;
  uint16_t* cimg;
  float* cr;
  int32_t* clabel;
  float* cnorm2;
  int64_t n0;
  int d;
  int store;
};

constexpr int kCopyThreads = 256;
constexpr int kCopyWaves = kCopyThreads / kWave;

// One wave per destination row t: lane l moves elements 4 l .. 4 l + 3 of
// each 256-element stretch of the row.
__global__ __launch_bounds__(kCopyThreads) void insert_copy_kernel(const InsertParams p) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * kCopyWaves + threadIdx.x / kWave;
  if (t >= p.count) return;
  const int lane = lane_id();
  const int64_t src = p.src_of[t];
  const int64_t dst = p.n0 + t;
  const float* zr = p.z_src + src * p.d;
  double s = 0.0;
  for (int k = 4 * lane; k < p.d; k += 4 * kWave) {
    f32x4 v = *reinterpret_cast<const f32x4*>(zr + k);
    if (p.store == LIPCACHE_BF16) {
      uint16_t h[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        h[i] = bf16_bits(v[i]);
        v[i] = bf16_to_f32(h[i]);  // the stored value
      }
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.cz) + dst * p.d + k) =
          uint2{static_cast<uint32_t>(h[0]) | (static_cast<uint32_t>(h[1]) << 16),
                static_cast<uint32_t>(h[2]) | (static_cast<uint32_t>(h[3]) << 16)};
    } else {
      *reinterpret_cast<f32x4*>(static_cast<float*>(p.cz) + dst * p.d + k) = v;
    }
    if (p.cimg)
      *reinterpret_cast<uint2*>(p.cimg + dst * p.d + k) =
          uint2{static_cast<uint32_t>(f16_bits(v[0])) | (static_cast<uint32_t>(f16_bits(v[1])) << 16),
                static_cast<uint32_t>(f16_bits(v[2])) | (static_cast<uint32_t>(f16_bits(v[3])) << 16)};
#pragma unroll
    for (int i = 0; i < 4; ++i) s = __builtin_fma(static_cast<double>(v[i]), static_cast<double>(v[i]), s);
  }
  s = wave_sum(s);
  if (lane == 0) {
    p.cnorm2[dst] = static_cast<float>(s);
    p.cr[dst] = p.r_src[src];
    p.clabel[dst] = p.label_src[src];
  }
}

}  // namespace lc

using namespace lc;

extern "C" size_t lipcache_insert_workspace_bytes(int64_t k) {
  const int64_t nb = k > 0 ? (k + kInsBlock - 1) / kInsBlock : 1;
  return 2 * align_up(static_cast<size_t>(nb) * sizeof(int64_t), 256) + 256 +
         align_up(static_cast<size_t>(k > 0 ? k : 1) * sizeof(int64_t), 256);
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
  // rows move as 16-byte vectors
  if (k > 0 && (reinterpret_cast<uintptr_t>(z_src) & 15u) != 0) return LIPCACHE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(c->z) & 15u) != 0 || (reinterpret_cast<uintptr_t>(c->zimg) & 7u) != 0)
    return LIPCACHE_EINVAL;
  if ((k + kCopyWaves - 1) / kCopyWaves > static_cast<int64_t>(UINT32_MAX)) return LIPCACHE_EUNSUPPORTED;
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
  int64_t* src_of = reinterpret_cast<int64_t*>(base + 2 * align_up(static_cast<size_t>(nb) * 8, 256) + 256);

  if (nb == 1) {
    // one block: its ranks are final, one launch before the read-back
    hipLaunchKernelGGL(insert_rank_one_kernel, dim3(1), dim3(kInsBlock), 0, s, r_src, miss_selector, k, src_of,
                       total);
    LC_LAUNCHED();
  } else {
    hipLaunchKernelGGL(insert_count_kernel, dim3(static_cast<unsigned>(nb)), dim3(kInsBlock), 0, s, r_src,
                       miss_selector, k, counts);
    LC_LAUNCHED();
    hipLaunchKernelGGL(insert_scan_kernel, dim3(1), dim3(kInsBlock), 0, s, counts, nb, offsets, total);
    LC_LAUNCHED();
  }
  int64_t host_total = 0;
  LC_HIP(read_back(&host_total, total, sizeof(host_total), s));
  if (host_total < 0 || host_total > k) return LIPCACHE_EHIP;
  if (c->n + host_total > c->capacity) return LIPCACHE_ECAPACITY;
  if (host_total == 0) return LIPCACHE_OK;

  if (nb > 1) {
    hipLaunchKernelGGL(insert_rank_kernel, dim3(static_cast<unsigned>(nb)), dim3(kInsBlock), 0, s, r_src,
                       miss_selector, k, offsets, src_of);
    LC_LAUNCHED();
  }
  InsertParams p;
  p.z_src = z_src;
  p.label_src = label_src;
  p.r_src = r_src;
  p.src_of = src_of;
  p.count = host_total;
  p.cz = c->z;
  p.cimg = static_cast<uint16_t*>(c->zimg);
  p.cr = c->r;
  p.clabel = c->label;
  p.cnorm2 = c->norm2;
  p.n0 = c->n;
  p.d = c->d;
  p.store = c->store_dtype;
  hipLaunchKernelGGL(insert_copy_kernel, dim3(static_cast<unsigned>((host_total + kCopyWaves - 1) / kCopyWaves)),
                     dim3(kCopyThreads), 0, s, p);
  LC_LAUNCHED();
  c->n += host_total;
  if (inserted) *inserted = host_total;
  return LIPCACHE_OK;
}
