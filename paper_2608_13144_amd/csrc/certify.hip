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
// Two kernels.  For d <= 512 the logits run on the float64 matrix cores
// (certify_mfma_kernel, below).  For wider features a vector kernel is used:
// a workgroup of four waves owns a tile of E = 32 features, staged once in
// LDS.  Lane e of every wave works on feature e; wave w runs over the class
// chunks w, w+4, w+8, ... (eight classes per chunk), so the head row it
// reads is the same in all 64 lanes and comes through scalar loads of a
// float64 copy of W.  Each lane keeps a running
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

// dmax[y] = max over j with dist[y * C + j] > 0 of that distance (0 when
// every other row equals W_y): bounds every denominator of row y.
__global__ void row_dmax_kernel(const double* __restrict__ dist, int C, double* __restrict__ dmax) {
  const int y = static_cast<int>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (y >= C) return;
  double m = 0.0;
  for (int j = 0; j < C; ++j) {
    const double v = dist[static_cast<int64_t>(y) * C + j];
    m = v > m ? v : m;
  }
  dmax[y] = m;
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
  r_out[i] = f32_round_down(r);  // toward zero (r >= 0): never above the certificate
  if (margin_out) margin_out[i] = static_cast<float>(m);
  if (norm2_out) norm2_out[i] = static_cast<float>(nrm);
}

// ------------------------------------------------------------ matrix cores
// The same certification with the logits on the matrix cores (d <= 512):
// s = Z W^T by v_mfma_f64_16x16x4_f64 (float64 products of float32 values
// are exact; sums in float64).  A workgroup of four waves owns 64 features,
// 16 per wave, held as A operands in registers (lane (m, g) keeps feature m's
// k = 16 kq + 4 g + j); the head's rows pass through LDS 32 classes at a
// time (two 16-class B tiles, shared by the four waves).  Lane (m, g) ends a
// tile holding s for features g + 4 v of its wave and class c0 + m (the
// float64 instruction interleaves its output rows); it keeps
// a running (top-1, class, top-2) per feature over its classes in increasing
// order, and a butterfly over the 16 lanes of its row group merges them (the
// larger top-1 wins, the lower class on equal values, the rest competes for
// top-2): the same result as one pass over the classes in order.  For the
// tight radius each lane also keeps the classes of its own two largest
// logits and its third largest value; the minimum of (s_y - s_j) /
// ||W_y - W_j|| over the listed classes is the tight radius whenever a bound
// through the third values and the largest row distance of y shows that no
// unlisted class goes below it, and a workgroup with any row it cannot
// settle evaluates all logits a second time.
constexpr int kCmThreads = 256;
constexpr int kCmRows = 64;        // features per workgroup
constexpr int kCmClasses = 32;     // head rows per LDS stage

typedef double f64x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void top2_merge(double w1, int j1, double w2, double& v1, int& i1, double& v2) {
  if (w1 > v1 || (w1 == v1 && j1 < i1)) {
    v2 = v1 > v2 ? v1 : v2;
    v1 = w1;
    i1 = j1;
  } else {
    v2 = w1 > v2 ? w1 : v2;
  }
  v2 = w2 > v2 ? w2 : v2;
}

// Features past d are zero on both sides (registers and LDS), so every
// k-group runs and adds exact zeros there.
template <int KQ>
__device__ __forceinline__ void tile_logits(const f32x4 (&za)[KQ], const float* wl, int stride, int m16, int g,
                                            f64x4& acc0, f64x4& acc1) {
  acc0 = f64x4{0.0, 0.0, 0.0, 0.0};
  acc1 = f64x4{0.0, 0.0, 0.0, 0.0};
  const float* r0 = wl + m16 * stride + 4 * g;
  const float* r1 = wl + (16 + m16) * stride + 4 * g;
#pragma unroll
  for (int kq = 0; kq < KQ; ++kq) {
    const f32x4 b0 = *reinterpret_cast<const f32x4*>(r0 + 16 * kq);
    const f32x4 b1 = *reinterpret_cast<const f32x4*>(r1 + 16 * kq);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const double a = static_cast<double>(za[kq][j]);
      acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64(a, static_cast<double>(b0[j]), acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64(a, static_cast<double>(b1[j]), acc1, 0, 0, 0);
    }
  }
}

// Head rows c0 .. c0 + 31 into LDS, float32 as given; zeros past C and in
// the columns from d to the padded width `width`.
__device__ __forceinline__ void stage_head(const float* __restrict__ W, int C, int d, int width, int c0, float* wl,
                                           int stride) {
  const int q4 = width / 4;
  for (int t = static_cast<int>(threadIdx.x); t < kCmClasses * q4; t += kCmThreads) {
    const int row = t / q4, col = 4 * (t % q4);
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (c0 + row < C && col < d) v = *reinterpret_cast<const f32x4*>(W + static_cast<int64_t>(c0 + row) * d + col);
    *reinterpret_cast<f32x4*>(wl + row * stride + col) = v;
  }
}

template <bool BF16_STORE, bool TIGHT, int KQ>
__global__ __launch_bounds__(kCmThreads) void certify_mfma_kernel(
    const float* __restrict__ z, int64_t N, int d, const float* __restrict__ W, const float* __restrict__ b, int C,
    double sigma, const double* __restrict__ row_dist, const double* __restrict__ dmax, int32_t* __restrict__ label_out,
    float* __restrict__ r_out, float* __restrict__ margin_out, float* __restrict__ norm2_out) {
  extern __shared__ float wl[];  // kCmClasses rows of stride 16 KQ + 4 floats
  constexpr int kWidth = 16 * KQ;
  constexpr int stride = kWidth + 4;
  const int lane = lane_id();
  const int wave = uniform(static_cast<int>(threadIdx.x) / kWave);
  const int m16 = lane & 15, g = lane >> 4;
  const int nk = d / 16;
  const int64_t row0 = static_cast<int64_t>(blockIdx.x) * kCmRows + wave * 16;

  // A operands: feature row0 + m16, k = 16 kq + 4 g + j (stored values)
  f32x4 za[KQ];
  double nrm = 0.0;
  {
    const int64_t e = row0 + m16;
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      if (kq < nk && e < N) v = *reinterpret_cast<const f32x4*>(z + e * d + 16 * kq + 4 * g);
      if constexpr (BF16_STORE) {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = bf16_round_f32(v[j]);
      }
      za[kq] = v;
#pragma unroll
      for (int j = 0; j < 4; ++j) nrm = __builtin_fma(static_cast<double>(v[j]), static_cast<double>(v[j]), nrm);
    }
  }
  // ||z||^2 of feature m16: the four lanes g = 0..3 hold a quarter each
  nrm += __shfl_xor(nrm, 16, kWave);
  nrm += __shfl_xor(nrm, 32, kWave);

  double v1[4], v2[4];
  int i1[4];
  // tight radius: the lane's own two largest logits with their classes and
  // its third largest value, per feature
  double a1[4], a2[4], a3[4];
  int c1[4], c2[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    v1[v] = -__builtin_inf();
    v2[v] = -__builtin_inf();
    i1[v] = INT_MAX;
    a1[v] = a2[v] = a3[v] = -__builtin_inf();
    c1[v] = c2[v] = -1;
  }
  for (int c0 = 0; c0 < C; c0 += kCmClasses) {
    __syncthreads();
    stage_head(W, C, d, kWidth, c0, wl, stride);
    __syncthreads();
    f64x4 acc[2];
    tile_logits<KQ>(za, wl, stride, m16, g, acc[0], acc[1]);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int c = c0 + 16 * t + m16;
      if (c < C) {
        const double bc = b ? static_cast<double>(b[c]) : 0.0;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const double sv = acc[t][v] + bc;
          if constexpr (TIGHT) {
            if (sv > a1[v]) {
              a3[v] = a2[v];
              a2[v] = a1[v];
              c2[v] = c1[v];
              a1[v] = sv;
              c1[v] = c;
            } else if (sv > a2[v]) {
              a3[v] = a2[v];
              a2[v] = sv;
              c2[v] = c;
            } else if (sv > a3[v]) {
              a3[v] = sv;
            }
          } else {
            top2_push(sv, c, v1[v], i1[v], v2[v]);
          }
        }
      }
    }
  }
  if constexpr (TIGHT) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      v1[v] = a1[v];
      i1[v] = c1[v] < 0 ? INT_MAX : c1[v];
      v2[v] = a2[v];
    }
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const double w1 = __shfl_xor(v1[v], off, kWave);
      const int j1 = __shfl_xor(i1[v], off, kWave);
      const double w2 = __shfl_xor(v2[v], off, kWave);
      top2_merge(w1, j1, w2, v1[v], i1[v], v2[v]);
    }
  }

  double r[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = (v1[v] - v2[v]) / (sigma * kSqrt2);
  if constexpr (TIGHT) {
    // r* = min over j != y of (s_y - s_j) / ||W_y - W_j||.  First from the
    // lanes' lists: rl = the least ratio over every listed class.  A class a
    // lane did not list has s_j <= a3 of that lane and a denominator <=
    // dmax[y], so (rounding being monotone) its computed ratio is at least
    // fl(fl(s_y - a3) / dmax[y]); when that is >= rl on all 16 lanes, rl is
    // the minimum over all classes.  Otherwise the workgroup recomputes
    // every logit (same arithmetic, so the same values) and takes the
    // minimum over all of them; the result is the same number either way.
    double best[4];
    bool ok = true;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int y = i1[v];
      double rl = __builtin_inf();
      bool lane_ok = true;
      if (y >= 0 && y < C) {
        if (c1[v] >= 0 && c1[v] != y) {
          const double den = row_dist[static_cast<int64_t>(y) * C + c1[v]];
          if (den > 0.0) {
            const double q = (v1[v] - a1[v]) / den;
            rl = q < rl ? q : rl;
          }
        }
        if (c2[v] >= 0 && c2[v] != y) {
          const double den = row_dist[static_cast<int64_t>(y) * C + c2[v]];
          if (den > 0.0) {
            const double q = (v1[v] - a2[v]) / den;
            rl = q < rl ? q : rl;
          }
        }
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const double o = __shfl_xor(rl, off, kWave);
        rl = o < rl ? o : rl;
      }
      if (y >= 0 && y < C && a3[v] > -__builtin_inf()) {
        const double dm = dmax[y];
        if (dm > 0.0) lane_ok = (v1[v] - a3[v]) / dm >= rl;
      }
      ok = ok && lane_ok;
      best[v] = rl;
    }
    if (__syncthreads_or(ok ? 0 : 1)) {
#pragma unroll
    for (int v = 0; v < 4; ++v) best[v] = __builtin_inf();
    for (int c0 = 0; c0 < C; c0 += kCmClasses) {
      __syncthreads();
      stage_head(W, C, d, kWidth, c0, wl, stride);
      __syncthreads();
      f64x4 acc[2];
      tile_logits<KQ>(za, wl, stride, m16, g, acc[0], acc[1]);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int c = c0 + 16 * t + m16;
        if (c < C) {
          const double bc = b ? static_cast<double>(b[c]) : 0.0;
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int y = i1[v];
            if (y >= 0 && y < C && c != y) {
              const double den = row_dist[static_cast<int64_t>(y) * C + c];
              if (den > 0.0) {
                const double rij = (v1[v] - (acc[t][v] + bc)) / den;
                best[v] = rij < best[v] ? rij : best[v];
              }
            }
          }
        }
      }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const double o = __shfl_xor(best[v], off, kWave);
        best[v] = o < best[v] ? o : best[v];
      }
    }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      // no label when the feature is not finite
      r[v] = (i1[v] >= 0 && i1[v] < C) ? best[v] : __builtin_nan("");
    }
  }
  // lane (m16 < 4, g) writes feature g + 4 m16 of the wave (its v = m16)
  const double n_out = __shfl(nrm, g + 4 * (m16 & 3), kWave);
  if (m16 < 4) {
    const int64_t i = row0 + g + 4 * m16;
    if (i < N) {
      double rv = r[0], mv = v1[0] - v2[0];
      int lab = i1[0];
#pragma unroll
      for (int v = 1; v < 4; ++v) {
        if (m16 == v) {
          rv = r[v];
          mv = v1[v] - v2[v];
          lab = i1[v];
        }
      }
      label_out[i] = lab;
      r_out[i] = f32_round_down(rv);  // toward zero (r >= 0): never above the certificate
      if (margin_out) margin_out[i] = static_cast<float>(mv);
      if (norm2_out) norm2_out[i] = static_cast<float>(n_out);
    }
  }
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

template <bool BF16_STORE, bool TIGHT, int KQ>
hipError_t launch_mfma_kq(unsigned grid, size_t lds, hipStream_t s, const float* z, int64_t N, int d, const float* W,
                          const float* b, int C, double sigma, const double* row_dist, const double* dmax, int32_t* label_out,
                          float* r_out, float* margin_out, float* norm2_out) {
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(certify_mfma_kernel<BF16_STORE, TIGHT, KQ>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((certify_mfma_kernel<BF16_STORE, TIGHT, KQ>), dim3(grid), dim3(kCmThreads), lds, s, z, N, d, W,
                     b, C, sigma, row_dist, dmax, label_out, r_out, margin_out, norm2_out);
  return hipGetLastError();
}

template <bool BF16_STORE, bool TIGHT>
hipError_t launch_mfma_d(int d, unsigned grid, size_t lds, hipStream_t s, const float* z, int64_t N, const float* W,
                         const float* b, int C, double sigma, const double* row_dist, const double* dmax, int32_t* label_out,
                         float* r_out, float* margin_out, float* norm2_out) {
  // registers for d / 16 k-groups, rounded up to a power of two
  const int nk = d / 16;
  if (nk <= 2)
    return launch_mfma_kq<BF16_STORE, TIGHT, 2>(grid, lds, s, z, N, d, W, b, C, sigma, row_dist, dmax, label_out, r_out,
                                                margin_out, norm2_out);
  if (nk <= 4)
    return launch_mfma_kq<BF16_STORE, TIGHT, 4>(grid, lds, s, z, N, d, W, b, C, sigma, row_dist, dmax, label_out, r_out,
                                                margin_out, norm2_out);
  if (nk <= 8)
    return launch_mfma_kq<BF16_STORE, TIGHT, 8>(grid, lds, s, z, N, d, W, b, C, sigma, row_dist, dmax, label_out, r_out,
                                                margin_out, norm2_out);
  if (nk <= 16)
    return launch_mfma_kq<BF16_STORE, TIGHT, 16>(grid, lds, s, z, N, d, W, b, C, sigma, row_dist, dmax, label_out, r_out,
                                                 margin_out, norm2_out);
  return launch_mfma_kq<BF16_STORE, TIGHT, 32>(grid, lds, s, z, N, d, W, b, C, sigma, row_dist, dmax, label_out, r_out,
                                               margin_out, norm2_out);
}

hipError_t launch_certify_mfma(bool bf16, bool tight, int d, unsigned grid, size_t lds, hipStream_t s, const float* z,
                               int64_t N, const float* W, const float* b, int C, double sigma,
                               const double* row_dist, const double* dmax, int32_t* label_out, float* r_out, float* margin_out,
                               float* norm2_out) {
  if (bf16 && tight)
    return launch_mfma_d<true, true>(d, grid, lds, s, z, N, W, b, C, sigma, row_dist, dmax, label_out, r_out, margin_out,
                                     norm2_out);
  if (bf16)
    return launch_mfma_d<true, false>(d, grid, lds, s, z, N, W, b, C, sigma, row_dist, dmax, label_out, r_out, margin_out,
                                      norm2_out);
  if (tight)
    return launch_mfma_d<false, true>(d, grid, lds, s, z, N, W, b, C, sigma, row_dist, dmax, label_out, r_out, margin_out,
                                      norm2_out);
  return launch_mfma_d<false, false>(d, grid, lds, s, z, N, W, b, C, sigma, row_dist, dmax, label_out, r_out, margin_out,
                                     norm2_out);
}

}  // namespace

extern "C" size_t lipcache_certify_workspace_bytes(int32_t C, int32_t d, int32_t radius_mode) {
  if (C < 1 || d < 1) return 0;
  size_t n = head_bytes(C, d);
  if (radius_mode == LIPCACHE_RADIUS_TIGHT)
    n += align_up(static_cast<size_t>(C) * C * sizeof(double), 256) + align_up(static_cast<size_t>(C) * sizeof(double), 256);
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
  const bool tight = radius_mode == LIPCACHE_RADIUS_TIGHT;
  // the float64 copy of W feeds the row distances and the vector kernel
  if (tight || d > 512) {
    hipLaunchKernelGGL(widen_kernel, dim3(static_cast<unsigned>((cd + 255) / 256)), dim3(256), 0, s, W, cd, W64);
    LC_LAUNCHED();
  }
  double* row_dist = nullptr;
  double* dmax = nullptr;
  if (tight) {
    row_dist = reinterpret_cast<double*>(static_cast<unsigned char*>(ws) + head_bytes(C, d));
    dmax = reinterpret_cast<double*>(reinterpret_cast<unsigned char*>(row_dist) +
                                     align_up(static_cast<size_t>(C) * C * sizeof(double), 256));
    const int64_t cc = static_cast<int64_t>(C) * C;
    hipLaunchKernelGGL(row_distance_kernel, dim3(static_cast<unsigned>((cc + 255) / 256)), dim3(256), 0, s, W64, C, d,
                       row_dist);
    LC_LAUNCHED();
    hipLaunchKernelGGL(row_dmax_kernel, dim3(static_cast<unsigned>((C + 255) / 256)), dim3(256), 0, s, row_dist, C,
                       dmax);
    LC_LAUNCHED();
  }

  if (d <= 512) {
    int kq = 2;
    while (16 * kq < d) kq *= 2;
    const size_t lds_m = static_cast<size_t>(kCmClasses) * (16 * kq + 4) * sizeof(float);
    const unsigned grid_m = static_cast<unsigned>((N + kCmRows - 1) / kCmRows);
    const hipError_t em = launch_certify_mfma(store_dtype == LIPCACHE_BF16, radius_mode == LIPCACHE_RADIUS_TIGHT, d,
                                              grid_m, lds_m, s, z, N, W, b, C, sigma, row_dist, dmax, label_out, r_out,
                                              margin_out, norm2_out);
    return em == hipSuccess ? LIPCACHE_OK : LIPCACHE_EHIP;
  }
  const int E = 32;  // features per workgroup of the vector kernel (d > 512)
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
