// Incoherence pre-rotation of rows (the "+H" preprocessing of Sec. 5): y = R x or y = R^T x,
// R = (H_{2^a} / sqrt(2^a) kron C_b) diag(s) for n = 2^a b, b odd, H the Sylvester Hadamard
// matrix, C_b the orthonormal DCT-II of length b, s_i = -1 when the top bit of the i-th
// splitmix64 output of the seed is set (the generator of the plan's sign mask).
//
// One workgroup per row, the row held in LDS (n <= 16384 floats).  Element n = i b + j; the odd
// factor mixes the b contiguous entries of each segment i, the Hadamard factor mixes entries with
// equal j across segments (kashin_rot_impl.h).  The two factors commute, so R applies signs,
// C_b, H and R^T applies H, C_b^T, signs.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kashin.h"
#include "kashin_internal.h"
#include "kashin_rot_impl.h"

namespace kashin {
namespace {

constexpr int kRotThreads = 256;
constexpr int kRotMaxN = 16384;
constexpr int kBatch = 16;  // row elements per thread loaded together
constexpr int kPadMaxN = 8192;

__device__ __forceinline__ float load_f32(const float* p) { return *p; }
__device__ __forceinline__ float load_f32(const __half* p) { return __half2float(*p); }
__device__ __forceinline__ float load_f32(const bf16_t* p) { return bf16_to_f32(*p); }

template <int B, bool INV, bool PAD, class IT>
__global__ __launch_bounds__(kRotThreads) void rotate_kernel(int n, uint64_t seed, float scale, const IT* x,
                                                             int64_t ldx, float* y, int64_t ldy, int64_t row0) {
  extern __shared__ float buf[];  // n floats, or n + n/16 with PAD (padded slots, rot_slot)
  const int64_t row = row0 + blockIdx.x;
  const IT* xr = x + row * ldx;
  // loads in batches of kBatch per thread, all issued before the first is used, so a row's
  // load is one memory latency per batch rather than one per element
  for (int i0 = threadIdx.x; i0 < n; i0 += kRotThreads * kBatch) {
    float v[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int i = i0 + k * kRotThreads;
      v[k] = load_f32(xr + (i < n ? i : n - 1));  // unconditional (an in-row index), so all loads issue together
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int i = i0 + k * kRotThreads;
      if (i < n) buf[rot_slot<PAD>(i)] = INV ? v[k] : v[k] * rot_sign(seed, i);
    }
  }
  __syncthreads();
  const int tid = threadIdx.x;
  if constexpr (!INV) {
    rot_odd_factor<B, false, kRotThreads>(buf, n, tid);
    rot_hadamard<B, kRotThreads, PAD>(buf, n, tid);
  } else {
    rot_hadamard<B, kRotThreads, PAD>(buf, n, tid);
    rot_odd_factor<B, true, kRotThreads>(buf, n, tid);
  }
  float* yr = y + row * ldy;
  for (int i = threadIdx.x; i < n; i += kRotThreads) {
    const float v = buf[rot_slot<PAD>(i)] * scale;
    yr[i] = INV ? v * rot_sign(seed, i) : v;
  }
}

template <int B, bool INV, class IT>
hipError_t launch_rot(int n, uint64_t seed, const IT* x, int64_t ldx, float* y, int64_t ldy, int64_t m,
                      hipStream_t s) {
  constexpr int64_t kMaxGrid = int64_t(1) << 30;
  const float scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(n / B)));  // 1 / sqrt(2^a)
  for (int64_t r0 = 0; r0 < m; r0 += kMaxGrid) {
    const int64_t g = (m - r0 < kMaxGrid) ? m - r0 : kMaxGrid;
    // power-of-two rows up to kPadMaxN take the padded layout (at most 34 KB of LDS per row)
    if (B == 1 && n <= kPadMaxN)
      hipLaunchKernelGGL((rotate_kernel<B, INV, B == 1, IT>), dim3(static_cast<unsigned>(g)), dim3(kRotThreads),
                         static_cast<unsigned>((n + (n >> 4)) * sizeof(float)), s, n, seed, scale, x, ldx, y, ldy, r0);
    else
      hipLaunchKernelGGL((rotate_kernel<B, INV, false, IT>), dim3(static_cast<unsigned>(g)), dim3(kRotThreads),
                         static_cast<unsigned>(n * sizeof(float)), s, n, seed, scale, x, ldx, y, ldy, r0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int B, class IT>
hipError_t launch_rot_dir(int n, uint64_t seed, bool inverse, const IT* x, int64_t ldx, float* y, int64_t ldy,
                          int64_t m, hipStream_t s) {
  return inverse ? launch_rot<B, true>(n, seed, x, ldx, y, ldy, m, s) : launch_rot<B, false>(n, seed, x, ldx, y, ldy, m, s);
}

template <class IT>
hipError_t launch_rot_odd(int n, uint64_t seed, bool inverse, const IT* x, int64_t ldx, float* y, int64_t ldy,
                          int64_t m, hipStream_t s) {
  const int b = n / (n & -n);
  if (b == 1) return launch_rot_dir<1>(n, seed, inverse, x, ldx, y, ldy, m, s);
  if (b == 3) return launch_rot_dir<3>(n, seed, inverse, x, ldx, y, ldy, m, s);
  return launch_rot_dir<43>(n, seed, inverse, x, ldx, y, ldy, m, s);
}

}  // namespace

bool rotate_supported_n(int n) {
  if (n < 1 || n > kRotMaxN) return false;
  const int b = n / (n & -n);
  return b == 1 || b == 3 || b == 43;
}

hipError_t launch_rotate(int n, uint64_t seed, bool inverse, const void* x, int dtype, int64_t ldx, float* y,
                         int64_t ldy, int64_t m, hipStream_t stream) {
  if (dtype == KASHIN_F16)
    return launch_rot_odd(n, seed, inverse, static_cast<const __half*>(x), ldx, y, ldy, m, stream);
  if (dtype == KASHIN_BF16)
    return launch_rot_odd(n, seed, inverse, static_cast<const bf16_t*>(x), ldx, y, ldy, m, stream);
  return launch_rot_odd(n, seed, inverse, static_cast<const float*>(x), ldx, y, ldy, m, stream);
}

}  // namespace kashin
