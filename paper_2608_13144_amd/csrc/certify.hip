// Certification of candidate features (Sec. 4.3, Alg. 1; Sec. 5.2).
//
// For each feature z_i: logits s = W z_i + b in float64 (Eq. (5)), label
// y = argmax (Eq. (6)), margin m = s_y - max_{j != y} s_j (Eq. (20)) and the
// conservative radius r = m / (sigma_max(W) sqrt 2) (Eq. (21)), or the tight
// radius r* = min_{j != y} (s_y - s_j) / ||W_y - W_j|| of Remark 5.1, where
// a competitor with W_j = W_y sets no finite constraint.  The margin is a
// difference of two logits of similar size, so the logits are accumulated
// in float64; float32 accumulation would move a large share of the radii by
// more than 1e-5 relative.
//
// Layout: a workgroup of four waves owns a tile of E features (E = 64 for
// d <= 512, else 32), staged once in LDS.  Lane e of every wave works on
// feature e; wave w runs over the class chunks w, w+4, w+8, ... (eight classes
// per chunk), so the head row it reads is the same in all 64 lanes and comes
// through scalar loads of a float64 copy of W.  Each lane keeps a running
// (top-1 value, top-1 class, top-2 value); the four waves' candidates are
// merged in wave order through LDS.  For the tight radius the label is
// broadcast back to the four waves, which recompute their classes' logits
// with the same arithmetic (so s_y comes out bit-identical) and keep the
// least (s_y - s_j) / ||W_y - W_j||, read from a C x C table of row
// distances built once per call.
#include <limits.h>

#include "lc_common.hpp"

namespace lc {

constexpr int kCertThreads = 256;
constexpr int kCertWaves = kCertThreads / kWave;
constexpr int kCertChunk = 8;
constexpr double kSqrt2 = 1.4142135623730951;  // float64 nearest to sqrt(2)

__global__ void widen_kernel(const float* __restrict__ src, int64_t n, double* __restrict__ dst) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = static_cast<double>(src[i]);
}

__device__ __forceinline__ void top2_push(double s, int c, double& v1, int& i1, double& v2) {
  if (s > v1) {
    v2 = v1;
    v1 = s;
    i1 = c;
  } else if (s > v2) {
    v2 = s;
  }
}

// dist[y * C + j] = ||W_y - W_j||_2 in float64 (the denominator of the
// per-pair radius of Remark 5.1).
__global__ void row_distance_kernel(const double* __restrict__ W64, int C, int d, double* __restrict__ dist) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(C) * C) return;
  const int y = static_cast<int>(t / C);
  const int j = static_cast<int>(t % C);
  const double* a = W64 + static_cast<int64_t>(y) * d;
  const double* b = W64 + static_cast<int64_t>(j) * d;
  double acc = 0.0;
  for (int k = 0; k < d; ++k) {
    const double diff = a[k] - b[k];
    acc = __builtin_fma(diff, diff, acc);
  }
  dist[t] = __builtin_sqrt(acc);
}

// W z (no bias) for the classes c0 .. c0 + 7 below C, from the lane's feature
// row zr in LDS and the float64 head (rows read through scalar loads).
__device__ __forceinline__ void chunk_logits(const float* zr, const double* __restrict__ W64, int c0, int C, int d,
                                             double (&acc)[kCertChunk]) {
#pragma unroll
  for (int j = 0; j < kCertChunk; ++j) acc[j] = 0.0;
  if (c0 + kCertChunk <= C) {
    const double* w0 = W64 + static_cast<int64_t>(c0) * d;
    for (int k = 0; k < d; k += 4) {
      const f32x4 zv = *reinterpret_cast<const f32x4*>(zr + k);
      const double z0 = zv[0], z1 = zv[1], z2 = zv[2], z3 = zv[3];
#pragma unroll
      for (int j = 0; j < kCertChunk; ++j) {
        const double* w = w0 + static_cast<int64_t>(j) * d + k;
        double a = acc[j];
        a = __builtin_fma(w[0], z0, a);
        a = __builtin_fma(w[1], z1, a);
        a = __builtin_fma(w[2], z2, a);
        a = __builtin_fma(w[3], z3, a);
        acc[j] = a;
      }
    }
  } else {
    for (int j = 0; j < C - c0; ++j) {
      const double* w = W64 + static_cast<int64_t>(c0 + j) * d;
      double a = 0.0;
      for (int k = 0; k < d; k += 4) {
        const f32x4 zv = *reinterpret_cast<const f32x4*>(zr + k);
        a = __builtin_fma(w[k], static_cast<double>(zv[0]), a);
        a = __builtin_fma(w[k + 1], static_cast<double>(zv[1]), a);
        a = __builtin_fma(w[k + 2], static_cast<double>(zv[2]), a);
        a = __builtin_fma(w[k + 3], static_cast<double>(zv[3]), a);
      }
      acc[j] = a;
    }
  }
}

template <bool BF16_STORE, bool TIGHT>
__global__ __launch_bounds__(kCertThreads) void certify_kernel(
    const float* __restrict__ z, int64_t N, int d, int E, const double* __restrict__ W64,
    const float* __restrict__ b, int C, double sigma, const double* __restrict__ row_dist,
    int32_t* __restrict__ label_out, float* __restrict__ r_out, float* __restrict__ margin_out,
    float* __restrict__ norm2_out) {
  extern __shared__ float zs[];  // E rows of stride d + 4 floats
  __shared__ double s_v1[kCertWaves][kWave];
  __shared__ double s_v2[kCertWaves][kWave];
  __shared__ int s_i1[kCertWaves][kWave];
  __shared__ int s_label[kWave];
  __shared__ double s_top[kWave];

  const int stride = d + 4;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * E;
  const int q4 = d / 4;
  for (int c = threadIdx.x; c < E * q4; c += kCertThreads) {
    const int row = c / q4;
    const int col = (c % q4) * 4;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (base + row < N) v = *reinterpret_cast<const f32x4*>(z + (base + row) * d + col);
    if constexpr (BF16_STORE) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = bf16_round_f32(v[i]);
    }
    *reinterpret_cast<f32x4*>(zs + row * stride + col) = v;
  }
  __syncthreads();

  const int lane = lane_id();
  const int wave = uniform(static_cast<int>(threadIdx.x) / kWave);
  const float* zr = zs + (lane < E ? lane : E - 1) * stride;
  const bool valid = lane < E && base + lane < N;

  double v1 = -__builtin_inf(), v2 = -__builtin_inf();
  int i1 = INT_MAX;
  const int nchunks = (C + kCertChunk - 1) / kCertChunk;
  for (int t = wave; t < nchunks; t += kCertWaves) {
    const int c0 = t * kCertChunk;
    double acc[kCertChunk];
    chunk_logits(zr, W64, c0, C, d, acc);
#pragma unroll
    for (int j = 0; j < kCertChunk; ++j) {
      const int c = c0 + j;
      if (c < C) {
        const double s = acc[j] + (b ? static_cast<double>(b[c]) : 0.0);
        top2_push(s, c, v1, i1, v2);
      }
    }
  }
  s_v1[wave][lane] = v1;
  s_v2[wave][lane] = v2;
  s_i1[wave][lane] = i1;

  double nrm = 0.0;
  if (wave == 0) {
    for (int k = 0; k < d; ++k) nrm = __builtin_fma(static_cast<double>(zr[k]), static_cast<double>(zr[k]), nrm);
  }
  __syncthreads();

  // Merge in wave order: the largest top-1 wins, the lower class on equal
  // values; everything else competes for top-2.
  double V1 = -__builtin_inf(), V2 = -__builtin_inf();
  int I1 = INT_MAX;
  if (wave == 0) {
#pragma unroll
    for (int w = 0; w < kCertWaves; ++w) {
      const double a1 = s_v1[w][lane];
      const int ai = s_i1[w][lane];
      if (a1 > V1 || (a1 == V1 && ai < I1)) {
        V2 = V1 > V2 ? V1 : V2;
        V1 = a1;
        I1 = ai;
      } else {
        V2 = a1 > V2 ? a1 : V2;
      }
      const double a2 = s_v2[w][lane];
      V2 = a2 > V2 ? a2 : V2;
    }
  }
  const double m = V1 - V2;
  double r = m / (sigma * kSqrt2);
  if constexpr (TIGHT) {
    if (wave == 0) {
      s_label[lane] = I1;
      s_top[lane] = V1;
    }
    __syncthreads();
    const int y = s_label[lane];
    const double sy = s_top[lane];
    double best = __builtin_inf();
    if (y >= 0 && y < C) {  // no label when the feature is not finite
      const double* dy = row_dist + static_cast<int64_t>(y) * C;
      for (int t = wave; t < nchunks; t += kCertWaves) {
        const int c0 = t * kCertChunk;
        double acc[kCertChunk];
        chunk_logits(zr, W64, c0, C, d, acc);
#pragma unroll
        for (int j = 0; j < kCertChunk; ++j) {
          const int c = c0 + j;
          if (c < C && c != y) {
            const double den = dy[c];
            if (den > 0.0) {
              const double rij = (sy - (acc[j] + (b ? static_cast<double>(b[c]) : 0.0))) / den;
              best = rij < best ? rij : best;
            }
          }
        }
      }
    } else {
      best = __builtin_nan("");
    }
    s_v1[wave][lane] = best;  // every wave has read its merge inputs above
    __syncthreads();
    if (wave == 0) {
      r = s_v1[0][lane];
#pragma unroll
      for (int w = 1; w < kCertWaves; ++w) r = s_v1[w][lane] < r ? s_v1[w][lane] : r;
    }
  }
  if (wave != 0 || !valid) return;
  const int64_t i = base + lane;
  label_out[i] = I1;
  r_out[i] = static_cast<float>(r);
  if (margin_out) margin_out[i] = static_cast<float>(m);
  if (norm2_out) norm2_out[i] = static_cast<float>(nrm);
}

}  // namespace lc

using namespace lc;

namespace {

size_t head_bytes(int32_t C, int32_t d) { return align_up(static_cast<size_t>(C) * d * sizeof(double), 256); }

template <bool BF16_STORE, bool TIGHT>
hipError_t launch_certify(unsigned grid, size_t lds, hipStream_t s, const float* z, int64_t N, int d, int E,
                          const double* W64, const float* b, int C, double sigma, const double* row_dist,
                          int32_t* label_out, float* r_out, float* margin_out, float* norm2_out) {
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(certify_kernel<BF16_STORE, TIGHT>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((certify_kernel<BF16_STORE, TIGHT>), dim3(grid), dim3(kCertThreads), lds, s, z, N, d, E, W64, b,
                     C, sigma, row_dist, label_out, r_out, margin_out, norm2_out);
  return hipGetLastError();
}

}  // namespace

extern "C" size_t lipcache_certify_workspace_bytes(int32_t C, int32_t d, int32_t radius_mode) {
  if (C < 1 || d < 1) return 0;
  size_t n = head_bytes(C, d);
  if (radius_mode == LIPCACHE_RADIUS_TIGHT) n += align_up(static_cast<size_t>(C) * C * sizeof(double), 256);
  return n;
}

extern "C" lipcache_status lipcache_certify(const float* z, int64_t N, int32_t d, const float* W,
                                            const float* b, int32_t C, double sigma,
                                            int32_t radius_mode, int32_t store_dtype,
                                            int32_t* label_out, float* r_out, float* margin_out,
                                            float* norm2_out, void* ws, size_t ws_bytes,
                                            lipcache_stream_t stream) {
  if (N < 0 || d < 32 || d > 1024 || d % 32 != 0 || C < 2) return LIPCACHE_EINVAL;
  if (!W || (N > 0 && (!z || !label_out || !r_out))) return LIPCACHE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(z) & 15u) != 0) return LIPCACHE_EINVAL;
  if (!(sigma > 0.0) || sigma == __builtin_inf()) return LIPCACHE_EINVAL;
  if (store_dtype != LIPCACHE_F32 && store_dtype != LIPCACHE_BF16) return LIPCACHE_EINVAL;
  if (radius_mode != LIPCACHE_RADIUS_CONSERVATIVE && radius_mode != LIPCACHE_RADIUS_TIGHT)
    return LIPCACHE_EINVAL;
  const size_t need = lipcache_certify_workspace_bytes(C, d, radius_mode);
  if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;
  if (N == 0) return LIPCACHE_OK;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  double* W64 = static_cast<double*>(ws);
  const int64_t cd = static_cast<int64_t>(C) * d;
  hipLaunchKernelGGL(widen_kernel, dim3(static_cast<unsigned>((cd + 255) / 256)), dim3(256), 0, s, W, cd, W64);
  LC_LAUNCHED();
  const bool tight = radius_mode == LIPCACHE_RADIUS_TIGHT;
  double* row_dist = nullptr;
  if (tight) {
    row_dist = reinterpret_cast<double*>(static_cast<unsigned char*>(ws) + head_bytes(C, d));
    const int64_t cc = static_cast<int64_t>(C) * C;
    hipLaunchKernelGGL(row_distance_kernel, dim3(static_cast<unsigned>((cc + 255) / 256)), dim3(256), 0, s, W64, C, d,
                       row_dist);
    LC_LAUNCHED();
  }

  const int E = d <= 512 ? 64 : 32;
  const size_t lds = static_cast<size_t>(E) * (d + 4) * sizeof(float);
  const unsigned grid = static_cast<unsigned>((N + E - 1) / E);
  const bool bf16 = store_dtype == LIPCACHE_BF16;
  hipError_t e;
  if (bf16 && tight)
    e = launch_certify<true, true>(grid, lds, s, z, N, d, E, W64, b, C, sigma, row_dist, label_out, r_out, margin_out,
                                   norm2_out);
  else if (bf16)
    e = launch_certify<true, false>(grid, lds, s, z, N, d, E, W64, b, C, sigma, row_dist, label_out, r_out,
                                    margin_out, norm2_out);
  else if (tight)
    e = launch_certify<false, true>(grid, lds, s, z, N, d, E, W64, b, C, sigma, row_dist, label_out, r_out,
                                    margin_out, norm2_out);
  else
    e = launch_certify<false, false>(grid, lds, s, z, N, d, E, W64, b, C, sigma, row_dist, label_out, r_out,
                                     margin_out, norm2_out);
  return e == hipSuccess ? LIPCACHE_OK : LIPCACHE_EHIP;
}
