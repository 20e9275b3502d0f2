// Internal helpers shared by the HIP sources of liblipcache (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>

#include "lipcache.h"

namespace lc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ------------------------------------------------------------------ status
#define LC_HIP(call)                                  \
  do {                                                \
    hipError_t lc_e_ = (call);                        \
    if (lc_e_ != hipSuccess) return LIPCACHE_EHIP;    \
  } while (0)

#define LC_LAUNCHED()                                          \
  do {                                                         \
    if (hipGetLastError() != hipSuccess) return LIPCACHE_EHIP; \
  } while (0)

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }

// ------------------------------------------------------------ read-backs
// The synchronous calls read a few bytes back (sigma, a count).  A copy into
// pageable memory is staged by the runtime, so these go through one of 64
// slots of 64 bytes in a pinned buffer, allocated on the first read-back and
// held until the process ends.  A slot is taken with an atomic bitmap, so
// concurrent calls from several host threads each use their own; with every
// slot taken (or no pinned buffer) the copy goes to `dst` directly.
constexpr size_t kReadSlotBytes = 64;
constexpr int kReadSlots = 64;
inline std::atomic<uint64_t> g_read_taken{0};
inline unsigned char* g_read_buf = nullptr;
inline std::once_flag g_read_once;

inline hipError_t read_back(void* dst, const void* src, size_t bytes, hipStream_t s) {
  std::call_once(g_read_once, [] {
    void* p = nullptr;
    if (hipHostMalloc(&p, kReadSlotBytes * kReadSlots, hipHostMallocPortable) == hipSuccess)
      g_read_buf = static_cast<unsigned char*>(p);
    else
      (void)hipGetLastError();
  });
  int slot = -1;
  if (g_read_buf && bytes <= kReadSlotBytes) {
    uint64_t m = g_read_taken.load(std::memory_order_relaxed);
    while (m != ~0ull) {
      const int i = __builtin_ctzll(~m);
      if (g_read_taken.compare_exchange_weak(m, m | (1ull << i), std::memory_order_acquire)) {
        slot = i;
        break;
      }
    }
  }
  void* to = slot >= 0 ? static_cast<void*>(g_read_buf + slot * kReadSlotBytes) : dst;
  hipError_t e = hipMemcpyAsync(to, src, bytes, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (slot >= 0) {
    if (e == hipSuccess) memcpy(dst, to, bytes);
    g_read_taken.fetch_and(~(1ull << slot), std::memory_order_release);
  }
  return e;
}

// ------------------------------------------------------------- bfloat16
// Round to nearest even via the hardware conversion (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint16_t bf16_bits(float x) {
  __bf16 h = static_cast<__bf16>(x);
  return __builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}
__device__ __forceinline__ float bf16_round_f32(float x) { return bf16_to_f32(bf16_bits(x)); }

// Pack 8 floats into 8 bf16 (one 16-byte MFMA operand chunk).
__device__ __forceinline__ u32x4 pack_bf16x8(const float* v) {
  u32x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    o[i] = static_cast<uint32_t>(bf16_bits(v[2 * i])) |
           (static_cast<uint32_t>(bf16_bits(v[2 * i + 1])) << 16);
  return o;
}

// ------------------------------------------------------------- float16
// Round to nearest even (v_cvt_f16_f32 in the default rounding mode) after
// clamping to the finite range, so every image value is finite: a value
// whose magnitude the clamp changes only occurs in rows with ||x|| >= 2^15,
// which the distance filter never trusts (see kF16Range2).  NaN becomes a
// finite value; a NaN row or query has a NaN threshold and never passes.
__device__ __forceinline__ uint16_t f16_bits(float x) {
  const _Float16 h = static_cast<_Float16>(__builtin_fminf(__builtin_fmaxf(x, -65504.0f), 65504.0f));
  return __builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ float f16_to_f32(uint16_t b) {
  return static_cast<float>(__builtin_bit_cast(_Float16, b));
}

// Pack 8 floats into 8 float16 (one 16-byte MFMA operand chunk).
__device__ __forceinline__ u32x4 pack_f16x8(const float* v) {
  u32x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    o[i] = static_cast<uint32_t>(f16_bits(v[2 * i])) | (static_cast<uint32_t>(f16_bits(v[2 * i + 1])) << 16);
  return o;
}

// ------------------------------------------------------------- reductions
// Butterfly sum over the 64 lanes of a wave; fixed order, so bitwise
// reproducible from run to run.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// DPP lane exchange of a float64 (two 32-bit moves).  CTRL is the DPP
// control: quad_perm patterns and row rotations stay inside 4- and 16-lane
// groups, so every source lane exists and the exchange has no LDS latency.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(b)), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(b >> 32)), CTRL, 0xF, 0xF, false);
  return __builtin_bit_cast(double, (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) |
                                        static_cast<uint64_t>(static_cast<uint32_t>(lo)));
}
constexpr int kDppQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kDppRowRor4 = 0x124;  // row_ror:4
constexpr int kDppRowRor8 = 0x128;  // row_ror:8

__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(b)), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(b >> 32)), lane);
  return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
}

// Sum over the 64 lanes of a wave with DPP inside each 16-lane row and four
// read-lanes across rows (fixed order): the result is the same in every lane
// and bitwise reproducible.  Call from wave-uniform control flow.
__device__ __forceinline__ double wave_sum_dpp(double v) {
  v += dpp_f64<kDppQuadXor1>(v);
  v += dpp_f64<kDppQuadXor2>(v);
  v += dpp_f64<kDppRowRor4>(v);
  v += dpp_f64<kDppRowRor8>(v);
  return ((readlane_f64(v, 0) + readlane_f64(v, 16)) + readlane_f64(v, 32)) + readlane_f64(v, 48);
}

__device__ __forceinline__ int lane_id() { return static_cast<int>(threadIdx.x) & (kWave - 1); }

// Wave-uniform value (lets the compiler keep it in a scalar register).
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Next float towards -infinity (finite input).
__device__ __forceinline__ float f32_step_down(float f) {
  const uint32_t b = __builtin_bit_cast(uint32_t, f);
  if (f > 0.0f) return __builtin_bit_cast(float, b - 1u);
  if (f < 0.0f) return __builtin_bit_cast(float, b + 1u);
  return __builtin_bit_cast(float, 0x80000001u);  // below +-0: the negative sub-normal of least magnitude
}

// Largest float <= x (x in float64; +-inf and NaN pass through the conversion).
__device__ __forceinline__ float f32_round_down(double x) {
  float f = static_cast<float>(x);
  if (static_cast<double>(f) > x) f = f32_step_down(f);
  return f;
}

// --------------------------------------------------------- filter slack
// Absolute slack that covers flushed sub-normal products.
constexpr double kFilterAbsSlack = 1e-25;

// ||x||^2 at or above which the float16 operands cannot be trusted to hold x
// (some |x_k| may reach the float16 range): such a query or entry passes the
// filter against everything, so the exact re-check decides all its pairs.
constexpr double kF16Range2 = 1073741824.0;  // (2^15)^2

// Constants of the matrix-core distance filter.  With u the unit roundoff of
// the operand type, every component is rounded to x_k (1 + e) + t with
// |e| <= u and |t| <= eta (eta covers results in the sub-normal range and
// sub-normal inputs the matrix core may flush); the products (exact in
// float32 for float16 operands) and the float32 additions add at most
// gamma = n u32 / (1 - n u32), n = d_pad + 2, of the absolute terms.  Hence
//   |g_hat - q.z| <= k sum_k |q_k z_k| + eta (1 + u)(1 + gamma)(|q|_1 + |z|_1)
//                    + (1 + gamma) d_pad eta^2,
// with k = 2u + u^2 + gamma (1 + u)^2 when both operands are rounded, u +
// gamma (1 + u) when the cache values are already exact (a bf16 store in a
// float16 image), gamma for float32 operands.  Using sum |q_k z_k| <=
// (||q||^2 + ||z||^2) / 2 and |x|_1 <= sqrt(d_pad) ||x||, the filter takes
// twice each term (the order of the additions inside the matrix core is not
// specified):
//   kappa = 2 k                      (relative, on (||q||^2 + ||z||^2) / 2)
//   eta1  = 2 eta (1 + u)(1 + gamma) sqrt(d_pad)   (per ||q|| and per ||z||)
//   eta0  = 2 (1 + gamma) d_pad eta^2 + kFilterAbsSlack / 2  (per query)
struct FilterSlack {
  double kappa;
  double eta1;
  double eta0;
  double range2;  // kF16Range2 for float16 operands, +inf for float32
};

inline FilterSlack filter_slack(int precision, int store_dtype, int d_pad) {
  const double u32 = 1.0 / 16777216.0;  // 2^-24
  const double n = static_cast<double>(d_pad) + 2.0;
  const double gam = n * u32 / (1.0 - n * u32);
  double u, eta, k;
  FilterSlack f;
  if (precision == LIPCACHE_F32) {
    u = 0.0;
    eta = 1.1754943508222875e-38;  // 2^-126: a flushed float32 sub-normal
    k = gam;
    f.range2 = __builtin_inf();
  } else {
    u = 1.0 / 2048.0;              // 2^-11, float16 unit roundoff
    eta = 1.0 / 16384.0;           // 2^-14: float16 sub-normals, or flushed ones
    k = store_dtype == LIPCACHE_BF16 ? u + gam * (1.0 + u) : 2.0 * u + u * u + gam * (1.0 + u) * (1.0 + u);
    f.range2 = kF16Range2;
  }
  f.kappa = 2.0 * k;
  f.eta1 = 2.0 * eta * (1.0 + u) * (1.0 + gam) * __builtin_sqrt(static_cast<double>(d_pad));
  f.eta0 = 2.0 * (1.0 + gam) * d_pad * eta * eta + 0.5 * kFilterAbsSlack;
  return f;
}

// Largest finite float: the threshold of a query or entry that passes the
// filter against everything (-FLT_MAX) while +inf still marks rows that can
// never be hit.
constexpr float kPassAll = -3.4028234663852886e38f;

}  // namespace lc
