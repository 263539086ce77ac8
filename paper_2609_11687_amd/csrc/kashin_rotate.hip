// Incoherence pre-rotation of rows (the "+H" preprocessing of Sec. 5): y = R x or y = R^T x,
// R = (H_{2^a} / sqrt(2^a) kron C_b) diag(s) for n = 2^a b, b odd, H the Sylvester Hadamard
// matrix, C_b the orthonormal DCT-II of length b, s_i = -1 when the top bit of the i-th
// splitmix64 output of the seed is set (the generator of the plan's sign mask).
//
// One workgroup per row, the row held in LDS (n <= 16384 floats).  Element n = i b + j; the odd
// factor mixes the b contiguous entries of each segment i (one thread per segment, in place, the
// constants compile-time), the Hadamard factor mixes entries with equal j across segments
// (radix-2 stages in place, one barrier per stage).  The two factors commute, so R applies
// signs, C_b, H and R^T applies H, C_b^T, signs.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kashin_internal.h"
#include "kashin_tables.h"

namespace kashin {
namespace {

constexpr int kRotThreads = 256;
constexpr int kRotMaxN = 16384;

__device__ __forceinline__ float rot_sign(uint64_t seed, int i) {
  uint64_t z = seed + static_cast<uint64_t>(i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  return (z >> 63) ? -1.f : 1.f;
}

__device__ __forceinline__ float load_f32(const float* p) { return *p; }
__device__ __forceinline__ float load_f32(const __half* p) { return __half2float(*p); }

// segment i of length B: v <- C_B v (or C_B^T v), in place
template <int B, bool TRANS>
__device__ __forceinline__ void odd_segment(float* seg) {
  float in[B];
#pragma unroll
  for (int j = 0; j < B; ++j) in[j] = seg[j];
#pragma unroll
  for (int k = 0; k < B; ++k) {
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < B; ++j) acc = fmaf(TRANS ? DctTab<B>::m[j * B + k] : DctTab<B>::m[k * B + j], in[j], acc);
    seg[k] = acc;
  }
}

template <int B, bool TRANS>
__device__ __forceinline__ void odd_factor(float* buf, int n) {
  if constexpr (B > 1) {
    for (int i = threadIdx.x; i < n / B; i += kRotThreads) odd_segment<B, TRANS>(buf + i * B);
    __syncthreads();
  }
}

// unnormalised Walsh-Hadamard transform over the 2^a segments (stride B), in place
template <int B>
__device__ __forceinline__ void hadamard_factor(float* buf, int n) {
  const int p2 = n / B;
  for (int lh = 0; (1 << lh) < p2; ++lh) {
    const int h = 1 << lh;
    for (int t = threadIdx.x; t < n / 2; t += kRotThreads) {
      const int q = t / B, j = t - q * B;  // butterfly q of the stage, column j
      const int i0 = ((q >> lh) << (lh + 1)) | (q & (h - 1));
      float* p0 = buf + i0 * B + j;
      float* p1 = p0 + h * B;
      const float a = *p0, b = *p1;
      *p0 = a + b;
      *p1 = a - b;
    }
    __syncthreads();
  }
}

template <int B, bool INV, class IT>
__global__ __launch_bounds__(kRotThreads) void rotate_kernel(int n, uint64_t seed, float scale, const IT* x,
                                                             int64_t ldx, float* y, int64_t ldy, int64_t row0) {
  extern __shared__ float buf[];  // n floats
  const int64_t row = row0 + blockIdx.x;
  const IT* xr = x + row * ldx;
  for (int i = threadIdx.x; i < n; i += kRotThreads) {
    const float v = load_f32(xr + i);
    buf[i] = INV ? v : v * rot_sign(seed, i);
  }
  __syncthreads();
  if constexpr (!INV) {
    odd_factor<B, false>(buf, n);
    hadamard_factor<B>(buf, n);
  } else {
    hadamard_factor<B>(buf, n);
    odd_factor<B, true>(buf, n);
  }
  float* yr = y + row * ldy;
  for (int i = threadIdx.x; i < n; i += kRotThreads) {
    const float v = buf[i] * scale;
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
    hipLaunchKernelGGL((rotate_kernel<B, INV, IT>), dim3(static_cast<unsigned>(g)), dim3(kRotThreads),
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
  if (dtype == 1)
    return launch_rot_odd(n, seed, inverse, static_cast<const __half*>(x), ldx, y, ldy, m, stream);
  return launch_rot_odd(n, seed, inverse, static_cast<const float*>(x), ldx, y, ldy, m, stream);
}

}  // namespace kashin
