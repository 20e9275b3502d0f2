// sigma_max(W) by float64 power iteration (Sec. 5.1, Eq. (18); Alg. 1).
//
// The head W is C x d.  The iteration v <- W^T W v / ||.|| is run on the
// smaller Gram matrix G (W W^T when C <= d, else W^T W), which has the same
// non-zero eigenvalues; sigma_max(W)^2 is G's largest eigenvalue.  One
// kernel forms G in float64 (every product of two floats is exact in float64),
// a second runs the whole iteration inside one 1024-thread workgroup: the
// iteration is a chain of dependent matrix-vector products, so it is bound by
// latency, and keeping G in registers (m <= 256) or L2 (m <= 1024) and the
// iterate in LDS leaves two workgroup barriers per step.
#include "lc_common.hpp"

namespace lc {

constexpr int kPowThreads = 1024;
constexpr int kPowTPR = 4;                                  // threads per row of G
constexpr int kPowRowsPerPass = kPowThreads / kPowTPR;      // 256
constexpr int kPowRegCols = 64;                             // columns per thread (m <= 256)
constexpr int kPowMaxM = 1024;

// G[a][b] = sum over the long side of W of products of W's entries.
__global__ void gram_kernel(const float* __restrict__ W, int C, int d, int side,
                            double* __restrict__ G) {
  const int m = side == 0 ? C : d;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(m) * m) return;
  const int a = static_cast<int>(idx / m);
  const int b = static_cast<int>(idx % m);
  double s = 0.0;
  if (side == 0) {  // (W W^T)_ab = sum_k W_ak W_bk
    const float* wa = W + static_cast<int64_t>(a) * d;
    const float* wb = W + static_cast<int64_t>(b) * d;
    for (int k = 0; k < d; ++k) s = __builtin_fma(static_cast<double>(wa[k]), static_cast<double>(wb[k]), s);
  } else {          // (W^T W)_ab = sum_c W_ca W_cb
    for (int c = 0; c < C; ++c) {
      const float* wc = W + static_cast<int64_t>(c) * d;
      s = __builtin_fma(static_cast<double>(wc[a]), static_cast<double>(wc[b]), s);
    }
  }
  G[idx] = s;
}

// Start vector: SplitMix64 of the component index mapped to [-1, 1).
__device__ __forceinline__ double start_component(int i) {
  uint64_t x = (static_cast<uint64_t>(i) + 1u) * 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  x ^= x >> 31;
  return static_cast<double>(x >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}

// out[0] = sigma, out[1] = iterations, out[2] = 1 if converged.
template <bool REG>
__global__ __launch_bounds__(kPowThreads) void power_kernel(const double* __restrict__ G, int m,
                                                            int max_iters, double rel_tol,
                                                            double* __restrict__ out) {
  __shared__ double vbuf[2][kPowMaxM];
  __shared__ double red[3][kPowThreads / kWave];

  const int t = threadIdx.x;
  const int g = t / kPowTPR;
  const int p = t % kPowTPR;
  const int lane = lane_id();
  const int wave = t / kWave;
  const int passes = (m + kPowRowsPerPass - 1) / kPowRowsPerPass;

  for (int i = t; i < kPowMaxM; i += kPowThreads) {
    vbuf[0][i] = i < m ? start_component(i) : 0.0;
    vbuf[1][i] = 0.0;
  }
  double greg[REG ? kPowRegCols : 1];
  if constexpr (REG) {
#pragma unroll
    for (int s = 0; s < kPowRegCols; ++s) {
      const int j = p + kPowTPR * s;
      greg[s] = (g < m && j < m) ? G[static_cast<int64_t>(g) * m + j] : 0.0;
    }
  }
  __syncthreads();

  int cur = 0, stable = 0, it = 0, converged = 0;
  double sigma = 0.0, prev = -1.0;
  for (it = 1; it <= max_iters; ++it) {
    const double* v = vbuf[cur];
    double ww = 0.0, vw = 0.0, vv = 0.0;
    double wrow[kPowMaxM / kPowRowsPerPass];
#pragma unroll
    for (int rr = 0; rr < kPowMaxM / kPowRowsPerPass; ++rr) {
      wrow[rr] = 0.0;
      if (rr >= passes) continue;
      const int a = g + kPowRowsPerPass * rr;
      double part = 0.0;
      if constexpr (REG) {
#pragma unroll
        for (int s = 0; s < kPowRegCols; ++s) part = __builtin_fma(greg[s], v[p + kPowTPR * s], part);
      } else {
        if (a < m) {
          const double* ga = G + static_cast<int64_t>(a) * m;
          for (int j = p; j < m; j += kPowTPR) part = __builtin_fma(ga[j], v[j], part);
        }
      }
      // The four partial sums of a row sit in adjacent lanes; after the two
      // exchanges every one of them holds the same row sum.
      part += __shfl_xor(part, 1, kWave);
      part += __shfl_xor(part, 2, kWave);
      if (a < m && p == 0) {
        wrow[rr] = part;
        ww = __builtin_fma(part, part, ww);
        vw = __builtin_fma(v[a], part, vw);
        vv = __builtin_fma(v[a], v[a], vv);
      }
    }
    ww = wave_sum(ww);
    vw = wave_sum(vw);
    vv = wave_sum(vv);
    if (lane == 0) {
      red[0][wave] = ww;
      red[1][wave] = vw;
      red[2][wave] = vv;
    }
    __syncthreads();
    double WW = 0.0, VW = 0.0, VV = 0.0;
#pragma unroll
    for (int w = 0; w < kPowThreads / kWave; ++w) {
      WW += red[0][w];
      VW += red[1][w];
      VV += red[2][w];
    }
    const double nrm = __builtin_sqrt(WW);
    if (!(nrm > 0.0) || !(VV > 0.0)) {  // G v = 0: W = 0, degenerate head
      sigma = 0.0;
      break;
    }
    const double lam = VW / VV;             // Rayleigh quotient v^T G v / v^T v
    const double sk = __builtin_sqrt(lam > 0.0 ? lam : 0.0);
    if (p == 0) {
#pragma unroll
      for (int rr = 0; rr < kPowMaxM / kPowRowsPerPass; ++rr) {
        const int a = g + kPowRowsPerPass * rr;
        if (rr < passes && a < m) vbuf[cur ^ 1][a] = wrow[rr] / nrm;
      }
    }
    if (it > 1 && __builtin_fabs(sk - prev) <= rel_tol * sk) {
      ++stable;
    } else {
      stable = 0;
    }
    prev = sk;
    sigma = sk;
    if (stable >= 2) {
      converged = 1;
      break;
    }
    __syncthreads();
    cur ^= 1;
  }
  if (t == 0) {
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
  return align_up(static_cast<size_t>(m * m) * sizeof(double), 256) + 256;
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

  double* G = static_cast<double*>(ws);
  double* out = reinterpret_cast<double*>(static_cast<char*>(ws) +
                                          align_up(static_cast<size_t>(m) * m * sizeof(double), 256));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int64_t cells = static_cast<int64_t>(m) * m;
  hipLaunchKernelGGL(gram_kernel, dim3(static_cast<unsigned>((cells + 255) / 256)), dim3(256), 0, s,
                     W, C, d, side, G);
  LC_LAUNCHED();
  if (m <= kPowRowsPerPass) {
    hipLaunchKernelGGL(power_kernel<true>, dim3(1), dim3(kPowThreads), 0, s, G, m, max_iters, rel_tol, out);
  } else {
    hipLaunchKernelGGL(power_kernel<false>, dim3(1), dim3(kPowThreads), 0, s, G, m, max_iters, rel_tol, out);
  }
  LC_LAUNCHED();
  double host[3] = {0.0, 0.0, 0.0};
  LC_HIP(hipMemcpyAsync(host, out, sizeof(host), hipMemcpyDeviceToHost, s));
  LC_HIP(hipStreamSynchronize(s));
  *sigma = host[0];
  if (iterations) *iterations = static_cast<int32_t>(host[1]);
  if (!(host[0] > 0.0)) return LIPCACHE_EDEGENERATE;
  if (host[2] == 0.0) return LIPCACHE_ENOCONV;
  return LIPCACHE_OK;
}
