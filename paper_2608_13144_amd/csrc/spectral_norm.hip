// sigma_max(W) by float64 power iteration (Sec. 5.1, Eq. (18); Alg. 1).
//
// The head W is C x d.  The iteration runs on the smaller Gram matrix G
// (W W^T when C <= d, else W^T W), which has the same non-zero eigenvalues;
// sigma_max(W)^2 is G's largest eigenvalue.  G is formed in float64 (every
// product of two floats is exact in float64).  Power iteration on G alone
// converges like (lambda_2 / lambda_1)^k, about 400 dependent matrix-vector
// products for the heads of interest (sigma_2 / sigma_1 ~ 0.98), each bound
// by latency.  Instead G is scaled by a power of two and squared
// kSquarings times on the whole chip (P = (G 2^-e)^64, a few parallel
// products), power iteration runs on P, whose eigenvalue ratio is the 64th
// power of G's (a dozen steps), and sigma_max^2 is the Rayleigh quotient of
// G itself at P's converged vector.  The iteration runs inside one
// 512-thread workgroup: the matrix stays in registers (m <= 208) or L2
// (m <= 1024), the iterate in LDS, reductions use DPP lane exchanges, and
// each step has one barrier.
#include "lc_common.hpp"

namespace lc {

constexpr int kPowThreads = 512;
constexpr int kPowWaves = kPowThreads / kWave;
constexpr int kPowTPR = 2;                                  // threads per row of G
constexpr int kPowRowsPerPass = kPowThreads / kPowTPR;      // 256
constexpr int kPowMaxM = 1024;
constexpr int kPowRegMaxM = 208;                            // matrix held in registers up to here
constexpr int kSquarings = 6;                               // P = (G 2^-e)^(2^6)

typedef double f64x4 __attribute__((ext_vector_type(4)));

enum { kGramRows = 0, kGramCols = 1, kGramSym = 2 };

// Entry (a, k) of the factor X in Out = X X^T: W's row a (W W^T), W's column
// a (W^T W), or row a of a symmetric float64 matrix times an exact power of
// two; zero outside the m x L range.
template <int MODE>
__device__ __forceinline__ double gram_x(const void* __restrict__ X, int ld, int m, int L, int a, int k, double s) {
  if (a >= m || k >= L) return 0.0;
  if constexpr (MODE == kGramRows) return static_cast<double>(static_cast<const float*>(X)[static_cast<int64_t>(a) * ld + k]);
  if constexpr (MODE == kGramCols) return static_cast<double>(static_cast<const float*>(X)[static_cast<int64_t>(k) * ld + a]);
  return static_cast<const double*>(X)[static_cast<int64_t>(a) * ld + k] * s;
}

// Out[a][b] = sum_k X(a, k) X(b, k) for a, b < m on the float64 matrix cores
// (v_mfma_f64_16x16x4_f64; products of floats are exact, sums in float64):
// one workgroup per 16 x 16 output tile.  Wave w takes the k-steps w, w + 4,
// w + 8, ... (so each dependent chain is a quarter of the k range and the
// four waves' loads overlap); lane (r, q) feeds X(i0 + r, k + q) and
// X(j0 + r, k + q) and ends holding rows i0 + q + 4v of column j0 + r.  The
// four partial tiles are added in wave order through LDS.
template <int MODE>
__global__ __launch_bounds__(256) void gram_mfma_kernel(const void* __restrict__ X, int ld, int m, int L,
                                                        const double* __restrict__ scale, double* __restrict__ Out) {
  __shared__ double part[4][4][kWave];
  const int lane = lane_id();
  const int w = static_cast<int>(threadIdx.x) / kWave;
  const int r = lane & 15, q = lane >> 4;
  const int tiles = (m + 15) / 16;
  const int t = static_cast<int>(blockIdx.x);
  const int i0 = (t / tiles) * 16, j0 = (t % tiles) * 16;
  const double s = (MODE == kGramSym && scale) ? scale[0] : 1.0;
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
  for (int k0 = 4 * w; k0 < L; k0 += 16) {
    const double a = gram_x<MODE>(X, ld, m, L, i0 + r, k0 + q, s);
    const double b = gram_x<MODE>(X, ld, m, L, j0 + r, k0 + q, s);
    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) part[w][v][lane] = acc[v];
  __syncthreads();
  if (w != 0) return;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const double sum = ((part[0][v][lane] + part[1][v][lane]) + part[2][v][lane]) + part[3][v][lane];
    const int row = i0 + q + 4 * v, col = j0 + r;
    if (row < m && col < m) Out[static_cast<int64_t>(row) * m + col] = sum;
  }
}

// scale[0] = 2^-e with 2^e > trace(A) >= lambda_max (0 for a zero trace):
// after this scaling every eigenvalue is at most 1, so 64th powers neither
// overflow nor, for the top eigenvalue (>= trace / m), underflow.
__global__ __launch_bounds__(256) void gram_scale_kernel(const double* __restrict__ A, int m,
                                                         double* __restrict__ scale) {
  __shared__ double part[256 / kWave];
  double tr = 0.0;
  for (int i = threadIdx.x; i < m; i += 256) tr += A[static_cast<int64_t>(i) * m + i];
  tr = wave_sum_dpp(tr);
  if (lane_id() == 0) part[threadIdx.x / kWave] = tr;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < 256 / kWave; ++w) t += part[w];
    scale[0] = t > 0.0 ? ldexp(1.0, -(ilogb(t) + 1)) : 0.0;
  }
}

// Start vector: SplitMix64 of the component index mapped to [-1, 1).
__device__ __forceinline__ double start_component(int i) {
  uint64_t x = (static_cast<uint64_t>(i) + 1u) * 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  x ^= x >> 31;
  return static_cast<double>(x >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}

// Power iteration on the symmetric m x m matrix M (a power of G), then
// sigma = sqrt of G's Rayleigh quotient at the final vector.
// out[0] = sigma, out[1] = iterations on M, out[2] = 1 if converged.
//
// Layout: two adjacent lanes share a row a of M (columns of one parity each),
// rows a, a + 256, ... per lane pair.  With NC > 0 the lane keeps its NC
// columns of M in registers (m <= 2 NC); with NC = 0 it re-reads them from
// global memory every iteration.  M is first scaled by an exact power of two
// (so its largest eigenvalue is at most 1).  The iterate x_k lives in LDS
// unnormalised (x_{k+1} = M x_k); the normalisation 1/||M x_k|| is applied as
// a scalar when x_{k+1} is read.  Each step therefore needs one barrier: it
// publishes the new vector and the per-wave partial sums of x.w, x.x and w.w,
// which give the Rayleigh quotient lambda_k = x_k.M x_k / x_k.x_k and the
// next normalisation.  The iteration stops when lambda_k changes by at most
// rel_tol relative on two consecutive steps.
template <int NC>
__global__ __launch_bounds__(kPowThreads) void power_kernel(const double* __restrict__ G,
                                                            const double* __restrict__ Gram, int m,
                                                            int max_iters, double rel_tol,
                                                            double* __restrict__ out) {
  __shared__ double xbuf[2][kPowMaxM];
  __shared__ double red[2][3][kPowWaves];
  __shared__ double tr_part[kPowWaves];
  __shared__ double fin[2][kPowWaves];

  const int t = threadIdx.x;
  const int g = t / kPowTPR;
  const int p = t % kPowTPR;
  const int lane = lane_id();
  const int wave = t / kWave;
  const int passes = (m + kPowRowsPerPass - 1) / kPowRowsPerPass;

  for (int i = t; i < kPowMaxM; i += kPowThreads) {
    xbuf[0][i] = i < m ? start_component(i) : 0.0;
    xbuf[1][i] = 0.0;
  }
  // trace(G) >= lambda_max > 0 fixes the power-of-two scale
  double tr = 0.0;
  for (int a = t; a < m; a += kPowThreads) tr += G[static_cast<int64_t>(a) * m + a];
  tr = wave_sum_dpp(tr);
  if (lane == 0) tr_part[wave] = tr;
  __syncthreads();
  tr = 0.0;
#pragma unroll
  for (int w = 0; w < kPowWaves; ++w) tr += tr_part[w];
  if (!(tr > 0.0)) {  // W = 0: degenerate head
    if (t == 0) {
      out[0] = 0.0;
      out[1] = 0.0;
      out[2] = 0.0;
    }
    return;
  }
  const int e = ilogb(tr) + 1;                       // 2^e > trace
  const double gscale = ldexp(1.0, -e);              // exact

  double greg[NC > 0 ? NC : 1];
  if constexpr (NC > 0) {
#pragma unroll
    for (int s = 0; s < NC; ++s) {
      const int j = p + kPowTPR * s;
      greg[s] = (g < m && j < m) ? G[static_cast<int64_t>(g) * m + j] * gscale : 0.0;
    }
  }

  int cur = 0, stable = 0, it = 0, converged = 0, last = -1;
  double prev = -1.0, invn = 1.0;
  for (it = 1; it <= max_iters; ++it) {
    const double* x = xbuf[cur];
    double lxw = 0.0, lxx = 0.0, lww = 0.0;
    for (int rr = 0; rr < passes; ++rr) {  // passes == 1 whenever NC > 0
      const int a = g + kPowRowsPerPass * rr;
      double acc0 = 0.0, acc1 = 0.0, acc2 = 0.0, acc3 = 0.0;
      if constexpr (NC > 0) {
#pragma unroll
        for (int s = 0; s < NC; s += 4) {
          acc0 = __builtin_fma(greg[s], x[p + kPowTPR * s], acc0);
          if (s + 1 < NC) acc1 = __builtin_fma(greg[s + 1], x[p + kPowTPR * (s + 1)], acc1);
          if (s + 2 < NC) acc2 = __builtin_fma(greg[s + 2], x[p + kPowTPR * (s + 2)], acc2);
          if (s + 3 < NC) acc3 = __builtin_fma(greg[s + 3], x[p + kPowTPR * (s + 3)], acc3);
        }
      } else if (a < m) {
        const double* ga = G + static_cast<int64_t>(a) * m;
        int j = p;
        for (; j + 3 * kPowTPR < m; j += 4 * kPowTPR) {
          acc0 = __builtin_fma(ga[j], x[j], acc0);
          acc1 = __builtin_fma(ga[j + kPowTPR], x[j + kPowTPR], acc1);
          acc2 = __builtin_fma(ga[j + 2 * kPowTPR], x[j + 2 * kPowTPR], acc2);
          acc3 = __builtin_fma(ga[j + 3 * kPowTPR], x[j + 3 * kPowTPR], acc3);
        }
        for (; j < m; j += kPowTPR) acc0 = __builtin_fma(ga[j], x[j], acc0);
        acc0 *= gscale;
        acc1 *= gscale;
        acc2 *= gscale;
        acc3 *= gscale;
      }
      double row = (acc0 + acc1) + (acc2 + acc3);
      row += dpp_f64<kDppQuadXor1>(row);  // the two lanes of the row
      if (p == 0 && a < m) {
        const double xa = invn * x[a];
        const double wa = invn * row;   // (G x)_a with x = invn * stored vector
        xbuf[cur ^ 1][a] = wa;
        lxw = __builtin_fma(xa, wa, lxw);
        lxx = __builtin_fma(xa, xa, lxx);
        lww = __builtin_fma(wa, wa, lww);
      }
    }
    lxw = wave_sum_dpp(lxw);
    lxx = wave_sum_dpp(lxx);
    lww = wave_sum_dpp(lww);
    if (lane == 0) {
      red[cur][0][wave] = lxw;
      red[cur][1][wave] = lxx;
      red[cur][2][wave] = lww;
    }
    __syncthreads();
    double XW = 0.0, XX = 0.0, WW = 0.0;
#pragma unroll
    for (int w = 0; w < kPowWaves; ++w) {
      XW += red[cur][0][w];
      XX += red[cur][1][w];
      WW += red[cur][2][w];
    }
    if (!(WW > 0.0) || !(XX > 0.0)) {  // M x = 0
      last = -1;
      break;
    }
    last = cur ^ 1;                // M x_k, the newest vector
    const double lam = XW / XX;    // Rayleigh quotient of the scaled M
    invn = 1.0 / __builtin_sqrt(WW);
    if (it > 1 && __builtin_fabs(lam - prev) <= rel_tol * lam) {
      ++stable;
    } else {
      stable = 0;
    }
    prev = lam;
    if (stable >= 2) {
      converged = 1;
      break;
    }
    cur ^= 1;
  }

  // sigma^2 = y.G y / y.y at the newest vector y (G unscaled, from memory).
  double sigma = 0.0;
  if (last >= 0) {
    const double* y = xbuf[last];
    double lyg = 0.0, lyy = 0.0;
    for (int rr = 0; rr < passes; ++rr) {
      const int a = g + kPowRowsPerPass * rr;
      double acc0 = 0.0, acc1 = 0.0;
      if (a < m) {
        const double* ga = Gram + static_cast<int64_t>(a) * m;
        int j = p;
        for (; j + kPowTPR < m; j += 2 * kPowTPR) {
          acc0 = __builtin_fma(ga[j], y[j], acc0);
          acc1 = __builtin_fma(ga[j + kPowTPR], y[j + kPowTPR], acc1);
        }
        for (; j < m; j += kPowTPR) acc0 = __builtin_fma(ga[j], y[j], acc0);
      }
      double row = acc0 + acc1;
      row += dpp_f64<kDppQuadXor1>(row);
      if (p == 0 && a < m) {
        lyg = __builtin_fma(y[a], row, lyg);
        lyy = __builtin_fma(y[a], y[a], lyy);
      }
    }
    lyg = wave_sum_dpp(lyg);
    lyy = wave_sum_dpp(lyy);
    if (lane == 0) {
      fin[0][wave] = lyg;
      fin[1][wave] = lyy;
    }
    __syncthreads();
    double YG = 0.0, YY = 0.0;
#pragma unroll
    for (int w = 0; w < kPowWaves; ++w) {
      YG += fin[0][w];
      YY += fin[1][w];
    }
    const double rho = YY > 0.0 ? YG / YY : 0.0;
    sigma = __builtin_sqrt(rho > 0.0 ? rho : 0.0);
  }
  if (t == 0) {
    out[0] = sigma;
    out[1] = static_cast<double>(it > max_iters ? max_iters : it);
    out[2] = static_cast<double>(converged);
  }
}

// Small heads (m = min(C, d) <= kSmallM): everything after G in one launch
// instead of a launch per squaring.  The scale and the kSquarings squarings
// run on LDS copies (all four waves, each entry a sum over k in ascending
// order); the iteration runs in wave 0 alone: lane a holds row a of the
// power and of G in registers and the iterate's entry a, reaches the other
// entries by lane shuffles and needs no barrier.  Same method and stopping
// rule as the chip-wide path: P = (G 2^-e)^(2^kSquarings) with 2^e >
// trace(G), P scaled by 2^-e' with 2^e' > trace(P), the same start vector,
// and sigma^2 the Rayleigh quotient of G at the last iterate.
constexpr int kSmallM = 32;

__global__ __launch_bounds__(256) void small_power_kernel(const double* __restrict__ G, int m, int max_iters,
                                                          double rel_tol, double* __restrict__ out) {
  __shared__ double gs[kSmallM * kSmallM];
  __shared__ double pbuf[2][kSmallM * kSmallM];
  const int t = static_cast<int>(threadIdx.x);
  const int lane = lane_id();
  const int mm = m * m;
  for (int i = t; i < mm; i += 256) gs[i] = G[i];
  __syncthreads();
  double tr = 0.0;  // every thread, the same order: the same value everywhere
  for (int a = 0; a < m; ++a) tr += gs[a * m + a];
  if (!(tr > 0.0)) {  // W = 0: degenerate head
    if (t == 0) {
      out[0] = 0.0;
      out[1] = 0.0;
      out[2] = 0.0;
    }
    return;
  }
  const double sg = ldexp(1.0, -(ilogb(tr) + 1));  // exact
  // P_1 = (s G)(s G), P_{i+1} = P_i P_i.  The factors are symmetric, so
  // entry (a, b) is taken as the dot product of columns a and b: the lanes
  // of a wave read consecutive words of one row (b varies fastest) and a
  // common word (a), without bank conflicts; the result is exactly symmetric.
  for (int i = t; i < mm; i += 256) {
    const int a = i / m, b = i % m;
    double acc = 0.0;
    for (int k = 0; k < m; ++k) acc = __builtin_fma(gs[k * m + a] * sg, gs[k * m + b] * sg, acc);
    pbuf[0][i] = acc;
  }
  __syncthreads();
  int cur = 0;
  for (int q = 1; q < kSquarings; ++q) {
    for (int i = t; i < mm; i += 256) {
      const int a = i / m, b = i % m;
      double acc = 0.0;
      for (int k = 0; k < m; ++k) acc = __builtin_fma(pbuf[cur][k * m + a], pbuf[cur][k * m + b], acc);
      pbuf[cur ^ 1][i] = acc;
    }
    __syncthreads();
    cur ^= 1;
  }
  if (t >= kWave) return;  // the iteration is wave 0's

  const double* M = pbuf[cur];
  double trm = 0.0;
  for (int a = 0; a < m; ++a) trm += M[a * m + a];
  double mrow[kSmallM], grow[kSmallM];
  const double ms = trm > 0.0 ? ldexp(1.0, -(ilogb(trm) + 1)) : 0.0;
#pragma unroll
  for (int k = 0; k < kSmallM; ++k) {
    const bool in = lane < m && k < m;
    mrow[k] = in ? M[lane * m + k] * ms : 0.0;
    grow[k] = in ? gs[lane * m + k] : 0.0;
  }
  double x = lane < m ? start_component(lane) : 0.0;
  int it = 0, stable = 0, converged = 0;
  bool have = false;
  double prev = -1.0;
  for (it = 1; it <= max_iters; ++it) {
    double w = 0.0;
#pragma unroll
    for (int k = 0; k < kSmallM; ++k) w = __builtin_fma(mrow[k], __shfl(x, k, kWave), w);
    const double XW = wave_sum_dpp(x * w);
    const double XX = wave_sum_dpp(x * x);
    const double WW = wave_sum_dpp(w * w);
    if (!(WW > 0.0) || !(XX > 0.0)) {  // M x = 0
      have = false;
      break;
    }
    have = true;
    const double lam = XW / XX;  // Rayleigh quotient of the scaled M
    x = w / __builtin_sqrt(WW);  // the newest vector, normalised
    if (it > 1 && __builtin_fabs(lam - prev) <= rel_tol * lam) {
      ++stable;
    } else {
      stable = 0;
    }
    prev = lam;
    if (stable >= 2) {
      converged = 1;
      break;
    }
  }
  // sigma^2 = y.G y / y.y at the newest vector y
  double sigma = 0.0;
  if (have) {
    double gy = 0.0;
#pragma unroll
    for (int k = 0; k < kSmallM; ++k) gy = __builtin_fma(grow[k], __shfl(x, k, kWave), gy);
    const double YG = wave_sum_dpp(x * gy);
    const double YY = wave_sum_dpp(x * x);
    const double rho = YY > 0.0 ? YG / YY : 0.0;
    sigma = __builtin_sqrt(rho > 0.0 ? rho : 0.0);
  }
  if (lane == 0) {
    out[0] = sigma;
    out[1] = static_cast<double>(it > max_iters ? max_iters : it);
    out[2] = static_cast<double>(converged);
  }
}

}  // namespace lc

using namespace lc;

extern "C" size_t lipcache_spectral_norm_workspace_bytes(int32_t C, int32_t d) {
  if (C < 1 || d < 1) return 0;
  const int64_t m = C <= d ? C : d;
  // G and two buffers for the squarings, then the 3 result words
  return 3 * align_up(static_cast<size_t>(m * m) * sizeof(double), 256) + 256;
}

extern "C" lipcache_status lipcache_spectral_norm(const float* W, int32_t C, int32_t d,
                                                  int32_t max_iters, double rel_tol,
                                                  double* sigma, int32_t* iterations,
                                                  void* ws, size_t ws_bytes,
                                                  lipcache_stream_t stream) {
  if (!W || !sigma || C < 1 || d < 1 || max_iters < 1) return LIPCACHE_EINVAL;
  if (!(rel_tol > 0.0) || !(rel_tol < 1.0)) return LIPCACHE_EINVAL;
  const int side = C <= d ? 0 : 1;
  const int m = side == 0 ? C : d;
  if (m > kPowMaxM) return LIPCACHE_EUNSUPPORTED;
  const size_t need = lipcache_spectral_norm_workspace_bytes(C, d);
  if (!ws || ws_bytes < need || !aligned256(ws)) return LIPCACHE_EWORKSPACE;

  const size_t mat = align_up(static_cast<size_t>(m) * m * sizeof(double), 256);
  double* G = static_cast<double*>(ws);
  double* P[2] = {reinterpret_cast<double*>(static_cast<char*>(ws) + mat),
                  reinterpret_cast<double*>(static_cast<char*>(ws) + 2 * mat)};
  double* out = reinterpret_cast<double*>(static_cast<char*>(ws) + 3 * mat);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int tiles = (m + 15) / 16;
  const dim3 tgrid(static_cast<unsigned>(tiles * tiles));
  if (side == 0) {
    hipLaunchKernelGGL(gram_mfma_kernel<kGramRows>, tgrid, dim3(256), 0, s, W, d, m, d, nullptr, G);
  } else {
    hipLaunchKernelGGL(gram_mfma_kernel<kGramCols>, tgrid, dim3(256), 0, s, W, d, m, C, nullptr, G);
  }
  LC_LAUNCHED();
  if (m <= kSmallM) {
    hipLaunchKernelGGL(small_power_kernel, dim3(1), dim3(256), 0, s, G, m, max_iters, rel_tol, out);
    LC_LAUNCHED();
    double host[3] = {0.0, 0.0, 0.0};
    LC_HIP(read_back(host, out, sizeof(host), s));
    *sigma = host[0];
    if (iterations) *iterations = static_cast<int32_t>(host[1]);
    if (!(host[0] > 0.0)) return LIPCACHE_EDEGENERATE;
    if (host[2] == 0.0) return LIPCACHE_ENOCONV;
    return LIPCACHE_OK;
  }
  double* scale = out + 4;
  hipLaunchKernelGGL(gram_scale_kernel, dim3(1), dim3(256), 0, s, G, m, scale);
  LC_LAUNCHED();
  // P_1 = (s G)(s G), then P_{i+1} = P_i P_i (G and its powers are symmetric)
  hipLaunchKernelGGL(gram_mfma_kernel<kGramSym>, tgrid, dim3(256), 0, s, G, m, m, m, scale, P[0]);
  LC_LAUNCHED();
  for (int i = 1; i < kSquarings; ++i) {
    hipLaunchKernelGGL(gram_mfma_kernel<kGramSym>, tgrid, dim3(256), 0, s, P[(i + 1) & 1], m, m, m, nullptr, P[i & 1]);
    LC_LAUNCHED();
  }
  const double* M = P[(kSquarings + 1) & 1];
  const int nc = (m + kPowTPR - 1) / kPowTPR;
  auto launch = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(1), dim3(kPowThreads), 0, s, M, G, m, max_iters, rel_tol, out);
  };
  if (m > kPowRegMaxM) {
    launch(power_kernel<0>);
  } else if (nc <= 16) {
    launch(power_kernel<16>);
  } else if (nc <= 32) {
    launch(power_kernel<32>);
  } else if (nc <= 48) {
    launch(power_kernel<48>);
  } else if (nc <= 64) {
    launch(power_kernel<64>);
  } else if (nc <= 80) {
    launch(power_kernel<80>);
  } else if (nc <= 96) {
    launch(power_kernel<96>);
  } else if (nc <= 100) {
    launch(power_kernel<100>);
  } else {
    launch(power_kernel<104>);
  }
  LC_LAUNCHED();
  double host[3] = {0.0, 0.0, 0.0};
  LC_HIP(read_back(host, out, sizeof(host), s));
  *sigma = host[0];
  if (iterations) *iterations = static_cast<int32_t>(host[1]);
  if (!(host[0] > 0.0)) return LIPCACHE_EDEGENERATE;
  if (host[2] == 0.0) return LIPCACHE_ENOCONV;
  return LIPCACHE_OK;
}
