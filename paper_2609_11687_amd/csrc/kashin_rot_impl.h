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

// outputs K0 .. K0 + KC - 1 (those below B) of C_B seg (or C_B^T seg), each accumulated over the
// inputs in ascending order from zero, as rot_odd_segment does
template <int B, bool TRANS, int K0, int KC, class V>
__device__ __forceinline__ void rot_odd_chunk(const V* seg, V (&acc)[KC]) {
#pragma unroll
  for (int kk = 0; kk < KC; ++kk) acc[kk] = rv_zero(acc[0]);
#pragma unroll
  for (int j = 0; j < B; ++j) {
    const V x = seg[j];
#pragma unroll
    for (int kk = 0; kk < KC; ++kk) {
      if (K0 + kk < B)
        acc[kk] = rv_fma(TRANS ? DctTab<B>::m[j * B + K0 + kk] : DctTab<B>::m[(K0 + kk) * B + j], x, acc[kk]);
    }
  }
}

// The odd factor for a length N known at compile time.  When the workgroup has at least twice
// as many threads as segments and B is large, each segment's outputs are split into NC chunks
// computed by NC threads (all inputs read before the barrier, outputs written after it), so that
// more waves share the work and each holds fewer values; otherwise one thread per segment.
template <int B, bool TRANS, int T, int N, class V>
__device__ __forceinline__ void rot_odd_factor_fixed(V* buf, int tid) {
  constexpr int NSEG = N / B;
  constexpr int NC = (B >= 16 && T >= 2 * NSEG) ? (T / NSEG < 3 ? T / NSEG : 3) : 1;
  if constexpr (NC == 1) {
    rot_odd_factor<B, TRANS, T>(buf, N, tid);
  } else {
    constexpr int KC = (B + NC - 1) / NC;
    V acc[KC];
    const int c = tid / NSEG, sg = tid - c * NSEG;  // chunk and segment of this thread
    const V* seg = buf + sg * B;
    if (c == 0) {
      rot_odd_chunk<B, TRANS, 0, KC>(seg, acc);
    } else if (c == 1) {
      rot_odd_chunk<B, TRANS, KC, KC>(seg, acc);
    } else if (NC == 3 && c == 2) {
      rot_odd_chunk<B, TRANS, 2 * KC, KC>(seg, acc);
    }
    __syncthreads();  // every input read before any output is written
    if (c < NC) {
      V* out = buf + sg * B + c * KC;
#pragma unroll
      for (int kk = 0; kk < KC; ++kk)
        if (c * KC + kk < B) out[kk] = acc[kk];
    }
    __syncthreads();
  }
}

// Slot of entry e of a row held in LDS: e, or with PAD (B = 1 only) e + e/16, one spare word per
// 16 entries, so that the 16 consecutive entries a thread of the first Hadamard pass takes, the
// stride-16 groups of the second and the row-order loads and stores all spread over the banks.
template <bool PAD>
__device__ __forceinline__ int rot_slot(int e) {
  return PAD ? e + (e >> 4) : e;
}

// One pass of the unnormalised Walsh-Hadamard transform over the segment-index bits
// [lh, lh + log2 R): each thread takes groups of R entries at stride 2^lh B, transforms them in
// registers with radix-2 stages in ascending bit order, and writes them back; then a barrier.
// Consecutive threads take consecutive offsets within a stride, so each access is contiguous.
// With PAD the entries sit at rot_slot<true> (the stride 2^lh is then 1 or a multiple of 16, so
// entries hb apart are hb + hb/16 slots apart).
template <int B, int R, int T, bool PAD = false, class V>
__device__ __forceinline__ void rot_hadamard_pass(V* buf, int n, int lh, int tid) {
  static_assert(!PAD || B == 1, "padded rows are power-of-two rows");
  const int hb = (1 << lh) * B;
  const int st = PAD ? hb + (hb >> 4) : hb;
  for (int q = tid; q < n / R; q += T) {
    const int hi = (q >> lh) / B;  // = q / hb
    V* p = buf + rot_slot<PAD>(hi * (R * hb) + (q - hi * hb));
    V x[R];
#pragma unroll
    for (int m = 0; m < R; ++m) x[m] = p[m * st];
#pragma unroll
    for (int st = 1; st < R; st <<= 1) {
#pragma unroll
      for (int m = 0; m < R; ++m) {
        if (!(m & st)) {
          const V u = x[m], v = x[m + st];
          x[m] = rv_add(u, v);
          x[m + st] = rv_sub(u, v);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < R; ++m) p[m * st] = x[m];
  }
  __syncthreads();
}

// unnormalised Walsh-Hadamard transform over the 2^a segments (stride B), in place: passes of
// radix 16 (a last one of radix 2, 4 or 8), the radix-2 stages in ascending bit order overall
template <int B, int T, bool PAD = false, class V>
__device__ __forceinline__ void rot_hadamard(V* buf, int n, int tid) {
  const int a = __builtin_ctz(static_cast<unsigned>(n));  // n = 2^a B, B odd
  int lh = 0;
  for (; lh + 4 <= a; lh += 4) rot_hadamard_pass<B, 16, T, PAD>(buf, n, lh, tid);
  const int r = a - lh;
  if (r == 3) rot_hadamard_pass<B, 8, T, PAD>(buf, n, lh, tid);
  else if (r == 2) rot_hadamard_pass<B, 4, T, PAD>(buf, n, lh, tid);
  else if (r == 1) rot_hadamard_pass<B, 2, T, PAD>(buf, n, lh, tid);
}

// b, the odd part of n = 2^a b
__host__ __device__ constexpr int rot_odd_part(int n) { return n / (n & -n); }

}  // namespace kashin
