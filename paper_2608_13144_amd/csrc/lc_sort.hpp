// Stable LSD radix sort of (32-bit key, 32-bit value) pairs, 8 bits per
// pass: per-block digit histograms, a per-digit scan over blocks, digit
// bases, and a scatter that keeps the order of equal digits inside a block
// (rank in the wave from eight digit-bit ballots, then the counts of the
// same digit in the block's earlier waves); and a one-block exclusive scan of
// counts.  The kernels are file-local so that every translation unit that
// uses them carries its own copy.
#pragma once

#include "lc_common.hpp"

namespace lc {
namespace {

constexpr int kSortThreads = 1024;  // one item per thread
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kBins = 256;

// hist[d * nb + b] = number of items of block b whose digit is d.
__global__ __launch_bounds__(kSortThreads) void radix_hist_kernel(const uint32_t* __restrict__ keys, int64_t n,
                                                                  int shift, int64_t nb, uint32_t* __restrict__ hist) {
  __shared__ uint32_t h[kBins];
  if (threadIdx.x < kBins) h[threadIdx.x] = 0u;
  __syncthreads();
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kSortThreads + threadIdx.x;
  if (i < n) atomicAdd(&h[(keys[i] >> shift) & (kBins - 1)], 1u);
  __syncthreads();
  if (threadIdx.x < kBins) hist[static_cast<int64_t>(threadIdx.x) * nb + blockIdx.x] = h[threadIdx.x];
}

// Inclusive prefix sum over the 1024 threads of the block (wave shuffles,
// then the 16 wave totals).
__device__ __forceinline__ uint32_t block_inclusive_scan(uint32_t v, uint32_t* wave_tot, uint32_t& block_total) {
  const int lane = lane_id();
  const int wave = static_cast<int>(threadIdx.x) / kWave;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t o = static_cast<uint32_t>(__shfl_up(static_cast<int>(v), off, kWave));
    if (lane >= off) v += o;
  }
  if (lane == kWave - 1) wave_tot[wave] = v;
  __syncthreads();
  uint32_t before = 0, total = 0;
  for (int w = 0; w < kSortWaves; ++w) {
    const uint32_t t = wave_tot[w];
    before += w < wave ? t : 0u;
    total += t;
  }
  __syncthreads();
  block_total = total;
  return before + v;
}

// Block d: exclusive scan of hist[d * nb .. d * nb + nb) in place; the digit
// total goes to dsum[d].
__global__ __launch_bounds__(kSortThreads) void radix_digit_scan_kernel(uint32_t* __restrict__ hist, int64_t nb,
                                                                        uint32_t* __restrict__ dsum) {
  __shared__ uint32_t wave_tot[kSortWaves];
  uint32_t* row = hist + static_cast<int64_t>(blockIdx.x) * nb;
  uint32_t running = 0;
  for (int64_t base = 0; base < nb; base += kSortThreads) {
    const int64_t j = base + threadIdx.x;
    const uint32_t v = j < nb ? row[j] : 0u;
    uint32_t tot = 0;
    const uint32_t incl = block_inclusive_scan(v, wave_tot, tot);
    if (j < nb) row[j] = running + incl - v;
    running += tot;
  }
  if (threadIdx.x == 0) dsum[blockIdx.x] = running;
}

// dbase[d] = sum of dsum[0 .. d) (one block of 256 threads, serial is fine).
__global__ void radix_base_kernel(const uint32_t* __restrict__ dsum, uint32_t* __restrict__ dbase) {
  if (threadIdx.x == 0) {
    uint32_t s = 0;
    for (int d = 0; d < kBins; ++d) {
      dbase[d] = s;
      s += dsum[d];
    }
  }
}

// Stable scatter: within a block, items keep their order among equal digits
// (rank inside the wave from eight digit-bit ballots, then the counts of the
// same digit in the block's earlier waves).
__global__ __launch_bounds__(kSortThreads) void radix_scatter_kernel(
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in, int64_t n, int shift, int64_t nb,
    const uint32_t* __restrict__ hist, const uint32_t* __restrict__ dbase, uint32_t* __restrict__ keys_out,
    uint32_t* __restrict__ vals_out) {
  __shared__ uint32_t wcount[kSortWaves][kBins];
  for (int t = threadIdx.x; t < kSortWaves * kBins; t += kSortThreads) (&wcount[0][0])[t] = 0u;
  __syncthreads();
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kSortThreads + threadIdx.x;
  const bool valid = i < n;
  const uint32_t key = valid ? keys_in[i] : 0u;
  const int dig = static_cast<int>((key >> shift) & (kBins - 1));
  const int lane = lane_id();
  const int wave = static_cast<int>(threadIdx.x) / kWave;
  unsigned long long same = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (dig >> b) & 1;
    const unsigned long long bal = __ballot(bit);
    same &= bit ? bal : ~bal;
  }
  const int rank = __builtin_popcountll(same & ((1ull << lane) - 1ull));
  if (valid && rank == 0) wcount[wave][dig] = static_cast<uint32_t>(__builtin_popcountll(same));
  __syncthreads();
  if (valid) {
    uint32_t before = 0;
    for (int w = 0; w < wave; ++w) before += wcount[w][dig];
    const uint32_t pos = dbase[dig] + hist[static_cast<int64_t>(dig) * nb + blockIdx.x] + before + rank;
    keys_out[pos] = key;
    vals_out[pos] = vals_in[i];
  }
}

// out[i] = sum of cnt below i for i = 0 .. m (out[m] is the total); one
// block of 1024 threads, each owning a contiguous run of counts.
__global__ __launch_bounds__(1024) void exclusive_scan_kernel(const uint32_t* __restrict__ cnt, int m,
                                                              int64_t* __restrict__ out) {
  __shared__ int64_t wsum[16];
  const int t = static_cast<int>(threadIdx.x);
  const int lane = t & 63, w = t >> 6;
  const int per = (m + 1023) / 1024;
  const int b0 = t * per, b1 = b0 + per < m ? b0 + per : m;
  int64_t sum = 0;
  for (int i = b0; i < b1; ++i) sum += cnt[i];
  // inclusive scan of the thread sums inside each wave, then of the wave totals
  int64_t x = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  if (w == 0) {
    int64_t v = lane < 16 ? wsum[lane] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int64_t y = __shfl_up(v, o, 64);
      if (lane >= o) v += y;
    }
    if (lane < 16) wsum[lane] = v;
  }
  __syncthreads();
  int64_t run = x - sum + (w > 0 ? wsum[w - 1] : 0);
  if (t == 1023) out[m] = run + sum;
  for (int i = b0; i < b1; ++i) {
    out[i] = run;
    run += cnt[i];
  }
}

inline int64_t radix_blocks(int64_t n) { return (n + kSortThreads - 1) / kSortThreads; }

// Sorts keys[cur]/vals[cur] (n items) by the low 8 * passes bits of the key;
// the result is in keys[cur']/vals[cur'] with cur' returned through `cur`.
// hist needs radix_blocks(n) * 256 words, dsum and dbase 256 each.
inline hipError_t radix_sort_u32(uint32_t* keys[2], uint32_t* vals[2], int64_t n, int passes, uint32_t* hist,
                                 uint32_t* dsum, uint32_t* dbase, int& cur, hipStream_t s) {
  const int64_t nb = radix_blocks(n);
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = 8 * pass;
    hipLaunchKernelGGL(radix_hist_kernel, dim3(static_cast<unsigned>(nb)), dim3(kSortThreads), 0, s, keys[cur], n,
                       shift, nb, hist);
    hipLaunchKernelGGL(radix_digit_scan_kernel, dim3(kBins), dim3(kSortThreads), 0, s, hist, nb, dsum);
    hipLaunchKernelGGL(radix_base_kernel, dim3(1), dim3(64), 0, s, dsum, dbase);
    hipLaunchKernelGGL(radix_scatter_kernel, dim3(static_cast<unsigned>(nb)), dim3(kSortThreads), 0, s, keys[cur],
                       vals[cur], n, shift, nb, hist, dbase, keys[cur ^ 1], vals[cur ^ 1]);
    cur ^= 1;
  }
  return hipGetLastError();
}

}  // namespace
}  // namespace lc
