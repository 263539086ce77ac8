// Device pieces of the incoherence rotation R = (H_{2^a} / sqrt(2^a) kron C_b) diag(s) (Sec. 5's
// "+H" preprocessing), shared by the standalone rotation kernel and the fused loads of the pair
// kernels.  Element index i b + j (segment i, position j); values are float (one row) or float2
// (two rows at once, the rotation acting on each component).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kashin_tables.h"

namespace kashin {

// s_i: -1 when the top bit of the i-th splitmix64 output of `seed` is set
__device__ __forceinline__ float rot_sign(uint64_t seed, int i) {
  uint64_t z = seed + static_cast<uint64_t>(i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  return (z >> 63) ? -1.f : 1.f;
}

__device__ __forceinline__ float rv_fma(float c, float a, float acc) { return fmaf(c, a, acc); }
__device__ __forceinline__ float2 rv_fma(float c, float2 a, float2 acc) {
  return make_float2(fmaf(c, a.x, acc.x), fmaf(c, a.y, acc.y));
}
__device__ __forceinline__ float rv_zero(float) { return 0.f; }
__device__ __forceinline__ float2 rv_zero(float2) { return make_float2(0.f, 0.f); }
__device__ __forceinline__ float rv_add(float a, float b) { return a + b; }
__device__ __forceinline__ float2 rv_add(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float rv_sub(float a, float b) { return a - b; }
__device__ __forceinline__ float2 rv_sub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float rv_scale(float a, float s) { return a * s; }
__device__ __forceinline__ float2 rv_scale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }

// one segment of length B: v <- C_B v (or C_B^T v), in place, constants compile-time
template <int B, bool TRANS, class V>
__device__ __forceinline__ void rot_odd_segment(V* seg) {
  V in[B];
#pragma unroll
  for (int j = 0; j < B; ++j) in[j] = seg[j];
#pragma unroll
  for (int k = 0; k < B; ++k) {
    V acc = rv_zero(in[0]);
#pragma unroll
    for (int j = 0; j < B; ++j) acc = rv_fma(TRANS ? DctTab<B>::m[j * B + k] : DctTab<B>::m[k * B + j], in[j], acc);
    seg[k] = acc;
  }
}

// the odd factor over all n / B segments (one thread per segment), then a barrier
template <int B, bool TRANS, int T, class V>
__device__ __forceinline__ void rot_odd_factor(V* buf, int n, int tid) {
  if constexpr (B > 1) {
    for (int i = tid; i < n / B; i += T) rot_odd_segment<B, TRANS>(buf + i * B);
    __syncthreads();
  }
}

// unnormalised Walsh-Hadamard transform over the 2^a segments (stride B), in place, radix-2
// stages with a barrier after each
template <int B, int T, class V>
__device__ __forceinline__ void rot_hadamard(V* buf, int n, int tid) {
  const int p2 = n / B;
  for (int lh = 0; (1 << lh) < p2; ++lh) {
    const int h = 1 << lh;
    for (int t = tid; t < n / 2; t += T) {
      const int q = t / B, j = t - q * B;  // butterfly q of the stage, column j
      const int i0 = ((q >> lh) << (lh + 1)) | (q & (h - 1));
      V* p0 = buf + i0 * B + j;
      V* p1 = p0 + h * B;
      const V a = *p0, b = *p1;
      *p0 = rv_add(a, b);
      *p1 = rv_sub(a, b);
    }
    __syncthreads();
  }
}

// b, the odd part of n = 2^a b
__host__ __device__ constexpr int rot_odd_part(int n) { return n / (n & -n); }

}  // namespace kashin
