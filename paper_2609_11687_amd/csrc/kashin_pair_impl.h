// Kernel templates (included by the per-size translation units kashin_n*.hip).
// HIP kernels for gfx950: Kashin-DCT decomposition (Alg. 2), the operator
// P = IDCT o diag(eps) o DCT (Sec. 4.1), four-peak 2-bit clustering (Sec. 3.1)
// and reconstitution (App. C).
//
// Data flow of one workgroup ("pair kernel"): two rows a, b of the weight matrix
// are held as one complex vector y = v_a + i v_b, where v is the row in the
// even/odd ("Makhoul") order v_m = x_{2m}, v_{N-1-m} = x_{2m+1}.  Then
//   DCT-II / DCT-III of both rows = one length-N complex FFT / inverse FFT of y,
// and the sign flips between them reduce to a per-frequency gather and scale:
//   Y'_k = f_k * Y_{s(k)},  s(k) = k if eps_k == eps_{N-k} else N - k,
//   f_k = eps_k / N  or  eps_k * exp(i pi k / N) / N.
// Because every greedy step is elementwise or a permutation-invariant l1 sum,
// the factors stay in the permuted order for the whole run; only loads and
// stores translate indices.  P never forms a matrix: each application is a
// forward FFT, the gather above fused into the first inverse pass, and an
// inverse FFT (Stockham, mixed radix, LDS-resident between passes).  Between two
// applications of P the residual sits in registers, where the greedy steps run.
// Rows are pre-scaled by a power of two (exact) so both halves of a pair have
// comparable magnitude; a row with NaN/Inf is zeroed inside the pair and
// reported as NaN, so it cannot contaminate its partner.

#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include <cfloat>
#include <cstdint>
#include <type_traits>

#include "kashin.h"
#include "kashin_internal.h"
#include "kashin_rot_impl.h"
#include "kashin_tables.h"

namespace kashin {
namespace {

// ------------------------------------------------------------------ compile-time helpers
template <int B, int E, class F>
__device__ __forceinline__ void sfor(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    sfor<B + 1, E>(f);
  }
}

constexpr int ilog2(int x) {
  int l = 0;
  while ((1 << l) < x) ++l;
  return l;
}
constexpr int bitrev(int x, int bits) {
  int r = 0;
  for (int i = 0; i < bits; ++i) r = (r << 1) | ((x >> i) & 1);
  return r;
}

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }

// cos / sin (2 pi m / 16) in double, for compile-time constants
struct W16 {
  static constexpr double C1 = 0.92387953251128674;  // cos(pi / 8)
  static constexpr double S1 = 0.38268343236508978;  // sin(pi / 8)
  static constexpr double H = 0.70710678118654752;   // sqrt(1 / 2)
  static constexpr double c[16] = {1, C1, H, S1, 0, -S1, -H, -C1, -1, -C1, -H, -S1, 0, S1, H, C1};
  static constexpr double s[16] = {0, S1, H, C1, 1, C1, H, S1, 0, -S1, -H, -C1, -1, -C1, -H, -S1};
};
constexpr double cabs_d(double v) { return v < 0 ? -v : v; }

// Radix-2 butterfly with a compile-time twiddle w = w16^K (forward, w16 = exp(-2 pi i / 16);
// the inverse uses w16^-K): (x, y) <- (x + w y, x - w y).  A general twiddle is applied as
// w y = m p with p = (w / m) y, m whichever of Re w, Im w is larger in magnitude: p takes
// two FMAs with the ratio t = Im w / Re w or Re w / Im w (|t| <= 1), and x +- m p four more,
// six instructions instead of a complex product followed by four additions.
template <int K, bool INV>
__device__ __forceinline__ void bfly(float2& x, float2& y) {
  constexpr int k = K & 15;
  const float2 a = x;
  if constexpr (k == 0) {
    x = cadd(a, y);
    y = csub(a, y);
  } else if constexpr (k == 8) {
    x = csub(a, y);
    y = cadd(a, y);
  } else if constexpr (k == 4 || k == 12) {
    // w = (0, wi), wi = +-1: w y = (-wi y.y, wi y.x)
    constexpr float wi = static_cast<float>(INV ? W16::s[k] : -W16::s[k]);
    const float2 wy = make_float2(-wi * y.y, wi * y.x);
    x = cadd(a, wy);
    y = csub(a, wy);
  } else {
    constexpr double wr = W16::c[k];
    constexpr double wi = INV ? W16::s[k] : -W16::s[k];
    float2 p;
    float m;
    if constexpr (cabs_d(wr) >= cabs_d(wi)) {
      constexpr float t = static_cast<float>(wi / wr);
      m = static_cast<float>(wr);
      p = make_float2(fmaf(-t, y.y, y.x), fmaf(t, y.x, y.y));  // (w / wr) y
    } else {
      constexpr float t = static_cast<float>(wr / wi);
      m = static_cast<float>(wi);
      p = make_float2(fmaf(t, y.x, -y.y), fmaf(t, y.y, y.x));  // (w / wi) y
    }
    x = make_float2(fmaf(m, p.x, a.x), fmaf(m, p.y, a.y));
    y = make_float2(fmaf(-m, p.x, a.x), fmaf(-m, p.y, a.y));
  }
}

// In-register DFT of a power-of-two length R <= 16: radix-2 decimation in time on the
// bit-reversed input (a compile-time renaming), so every twiddle multiplies the second
// operand of a butterfly and fuses with it; output in natural order.
template <int R, bool INV>
__device__ __forceinline__ void dft_pow2(float2 (&a)[R]) {
  constexpr int L = ilog2(R);
  float2 b[R];
  sfor<0, R>([&](auto iv) { b[decltype(iv)::value] = a[bitrev(decltype(iv)::value, L)]; });
  sfor<1, L + 1>([&](auto sv) {
    constexpr int len = 1 << decltype(sv)::value;
    constexpr int half = len >> 1;
    sfor<0, R / len>([&](auto bv) {
      sfor<0, half>([&](auto jv) {
        constexpr int i0 = decltype(bv)::value * len + decltype(jv)::value;
        bfly<decltype(jv)::value * (16 / len), INV>(b[i0], b[i0 + half]);
      });
    });
  });
  sfor<0, R>([&](auto iv) { a[decltype(iv)::value] = b[decltype(iv)::value]; });
}

// DFT of the twiddled inputs a_r tw(r) (tw(0) = 1; conjugated twiddles on the inverse).
// The first DIT stage pairs a_r with a_{r+R/2} (r = bitrev of the pair index): with
// x = a_r tw(r) and w = tw(r + R/2) it forms X = x + w a_{r+R/2} in four FMAs and the other
// output as 2x - X, so the second twiddle costs no separate complex product.
template <int R, bool INV, class TW>
__device__ __forceinline__ void dft_pow2_tw(float2 (&a)[R], TW&& tw) {
  constexpr int L = ilog2(R);
  constexpr int H = R / 2;
  float2 b[R];
  sfor<0, H>([&](auto mv) {
    constexpr int m = decltype(mv)::value;
    constexpr int r = bitrev(m, L - 1);
    float2 x = a[r];
    if constexpr (r > 0) {
      const float2 t = tw(std::integral_constant<int, r>{});
      x = INV ? make_float2(x.x * t.x + x.y * t.y, x.y * t.x - x.x * t.y)
              : make_float2(x.x * t.x - x.y * t.y, x.x * t.y + x.y * t.x);
    }
    const float2 w = tw(std::integral_constant<int, r + H>{});
    const float2 y = a[r + H];
    const float wy = INV ? -w.y : w.y;
    const float2 X = make_float2(fmaf(w.x, y.x, fmaf(-wy, y.y, x.x)), fmaf(w.x, y.y, fmaf(wy, y.x, x.y)));
    b[2 * m] = X;
    b[2 * m + 1] = make_float2(fmaf(2.f, x.x, -X.x), fmaf(2.f, x.y, -X.y));
  });
  sfor<2, L + 1>([&](auto sv) {
    constexpr int len = 1 << decltype(sv)::value;
    constexpr int half = len >> 1;
    sfor<0, R / len>([&](auto bv) {
      sfor<0, half>([&](auto jv) {
        constexpr int i0 = decltype(bv)::value * len + decltype(jv)::value;
        bfly<decltype(jv)::value * (16 / len), INV>(b[i0], b[i0 + half]);
      });
    });
  });
  sfor<0, R>([&](auto iv) { a[decltype(iv)::value] = b[decltype(iv)::value]; });
}

// In-register DFT of an odd length R, directly from its definition, pairing j with R-j
// so each constant multiplies a sum or a difference.  The sums and differences overwrite
// the inputs in place (a[j] <- a[j] + a[R-j], a[R-j] <- a[j] - a[R-j]) and outputs are
// handed to sink(q, A_q) as soon as they are formed, so no second array is live.
// `pre(r, v)` is applied to input r just before it is paired (the pass twiddles), so a
// twiddled input never waits in a register of its own.
template <int R, bool INV, class Pre, class Sink>
__device__ __forceinline__ void dft_odd(float2 (&a)[R], Pre&& pre, Sink&& sink) {
  constexpr int H = (R - 1) / 2;
  sfor<1, H + 1>([&](auto jv) {
    constexpr int j = decltype(jv)::value;
    const float2 p = pre(j, a[j]), m = pre(R - j, a[R - j]);
    a[j] = cadd(p, m);
    a[R - j] = csub(p, m);
    if constexpr (R > 16 && j % 4 == 0) __builtin_amdgcn_sched_barrier(0);
  });
  const float2 x0 = a[0];
  float2 sum = x0;
  sfor<1, H + 1>([&](auto jv) { sum = cadd(sum, a[decltype(jv)::value]); });
  sfor<1, H + 1>([&](auto qv) {
    constexpr int q = decltype(qv)::value;
    float2 re = x0;
    float2 im = make_float2(0.f, 0.f);
    sfor<1, H + 1>([&](auto jv) {
      constexpr int j = decltype(jv)::value;
      constexpr int m = (j * q) % R;
      constexpr float c = CisTab<R>::c[m];
      constexpr float sn = CisTab<R>::s[m];
      re.x = fmaf(a[j].x, c, re.x);
      re.y = fmaf(a[j].y, c, re.y);
      im.x = fmaf(a[R - j].x, sn, im.x);
      im.y = fmaf(a[R - j].y, sn, im.y);
    });
    // forward: A_q = re - i im, A_{R-q} = re + i im; inverse swaps them
    const float2 minus = make_float2(re.x + im.y, re.y - im.x);
    const float2 plus = make_float2(re.x - im.y, re.y + im.x);
    sink(q, INV ? plus : minus);
    sink(R - q, INV ? minus : plus);
    // keep the scheduler from interleaving all output pairs (each pair needs its own
    // accumulators next to the R inputs)
    if constexpr (R > 16) __builtin_amdgcn_sched_barrier(0);
  });
  sink(0, sum);
}

// In-register DFT of an even length R that is not a power of two, from its definition like
// dft_odd: inputs j and R-j (1 <= j < R/2) are paired into sums and differences, a[0] and
// a[R/2] enter every output with the signs (+, (-1)^q), and only nonzero constants multiply.
template <int R, bool INV, class Pre, class Sink>
__device__ __forceinline__ void dft_even(float2 (&a)[R], Pre&& pre, Sink&& sink) {
  constexpr int M = R / 2;
  sfor<1, M>([&](auto jv) {
    constexpr int j = decltype(jv)::value;
    const float2 p = pre(j, a[j]), m = pre(R - j, a[R - j]);
    a[j] = cadd(p, m);
    a[R - j] = csub(p, m);
  });
  const float2 x0 = a[0], xm = pre(M, a[M]);
  float2 sum = cadd(x0, xm), alt = (M % 2) ? csub(x0, xm) : cadd(x0, xm);  // outputs 0 and M
  sfor<1, M>([&](auto jv) {
    constexpr int j = decltype(jv)::value;
    sum = cadd(sum, a[j]);
    alt = (j % 2) ? csub(alt, a[j]) : cadd(alt, a[j]);
  });
  sfor<1, M>([&](auto qv) {
    constexpr int q = decltype(qv)::value;
    float2 re = (q % 2) ? csub(x0, xm) : cadd(x0, xm);
    float2 im = make_float2(0.f, 0.f);
    sfor<1, M>([&](auto jv) {
      constexpr int j = decltype(jv)::value;
      constexpr int m = (j * q) % R;
      constexpr float c = CisTab<R>::c[m];
      constexpr float sn = CisTab<R>::s[m];
      if constexpr (c != 0.f) {
        re.x = fmaf(a[j].x, c, re.x);
        re.y = fmaf(a[j].y, c, re.y);
      }
      if constexpr (sn != 0.f) {
        im.x = fmaf(a[R - j].x, sn, im.x);
        im.y = fmaf(a[R - j].y, sn, im.y);
      }
    });
    // forward: A_q = re - i im, A_{R-q} = re + i im; inverse swaps them
    const float2 minus = make_float2(re.x + im.y, re.y - im.x);
    const float2 plus = make_float2(re.x - im.y, re.y + im.x);
    sink(q, INV ? plus : minus);
    sink(R - q, INV ? minus : plus);
  });
  sink(0, sum);
  sink(M, alt);
}

// DFT of a length R that is not a power of two, outputs handed to sink(q, A_q)
template <int R, bool INV, class Pre, class Sink>
__device__ __forceinline__ void dft_small(float2 (&a)[R], Pre&& pre, Sink&& sink) {
  if constexpr (R % 2 == 1) dft_odd<R, INV>(a, pre, sink);
  else dft_even<R, INV>(a, pre, sink);
}

// DFT of a[] handed to sink(q, A_q) for every q (power-of-two R: computed in place first).
template <int R, bool INV, class Sink>
__device__ __forceinline__ void dft(float2 (&a)[R], Sink&& sink) {
  if constexpr ((R & (R - 1)) == 0) {
    if constexpr (R > 1) dft_pow2<R, INV>(a);
    sfor<0, R>([&](auto qv) { sink(decltype(qv)::value, a[decltype(qv)::value]); });
  } else {
    static_assert(R % 2 == 1, "composite non-power-of-two radices are not implemented");
    dft_odd<R, INV>(a, [](int, float2 v) { return v; }, sink);
  }
}

// ------------------------------------------------------------------ launch configuration
// N: vector length = complex FFT length of a packed pair.  T: threads per workgroup.
// W: occupancy target (waves per SIMD) given to the register allocator.
// Rs: radices of the forward FFT passes; the first radix also fixes the register layout
// in which the greedy steps run: thread t holds elements j + r * (N / R0) for its
// butterflies j = t + T * i, r < R0.
template <int N_, int T_, int W_, int... Rs>
struct Cfg {
  static constexpr int N = N_;
  static constexpr int T = T_;
  static constexpr int W = W_;  // waves per SIMD the register allocation must allow
  static constexpr int NP = sizeof...(Rs);
  static constexpr int rad[NP] = {Rs...};
  static constexpr int R0 = rad[0];
  static constexpr int NB0 = N / R0;
  static constexpr int B0 = (NB0 + T - 1) / T;
  static constexpr int E = B0 * R0;
  static constexpr int NW = (T + 63) / 64;
  static constexpr bool WIDE = uniform_resident(N_, T_, NP, rad);
  static constexpr int PS = pad_shift(N_, WIDE);  // LDS padding: PW spare slots per PG elements
  static constexpr int PW = pad_width(WIDE);
  static constexpr int PG = 1 << PS;
  static constexpr int LDS = N + PW * (N >> PS) + 4;
};

template <class C>
constexpr int ns_fwd(int p) {
  int s = 1;
  for (int i = 0; i < p; ++i) s *= C::rad[i];
  return s;
}
template <class C>
constexpr int ns_inv(int p) {
  int s = 1;
  for (int i = 0; i < p; ++i) s *= C::rad[C::NP - 1 - i];
  return s;
}

// LDS layout: element k of the length-N complex vector lives at float2 slot pad<C>(k) (C::PW
// spare slots per C::PG elements, so that both contiguous and stride-16 accesses of a Stockham
// pass spread over the banks).  pad<C>(x + y) = pad<C>(x) + pad<C>(y) whenever x mod PG +
// y mod PG < PG: a base slot plus compile-time offsets addresses a butterfly's elements.
template <class C>
__host__ __device__ constexpr int pad(int i) { return i + C::PW * (i >> C::PS); }
// Whether a Stockham write (element q of butterfly j to b + q S, b = (j / S) S R + j mod S,
// q < R) can address slots as pad(b) + pad(q S): S a multiple of PG, or S dividing PG with
// S R a multiple or a divisor of PG (then b mod PG + q S mod PG < PG for every q).
template <class C>
constexpr bool pad_offsets_ok(int S, int R) {
  return S % C::PG == 0 || (C::PG % S == 0 && ((S * R) % C::PG == 0 || C::PG % (S * R) == 0));
}

// Opaque copy of the thread index: without it every twiddle load and LDS address of every
// pass is proven invariant across the block loop, hoisted out of it, and kept live in
// registers at once.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Butterfly index of thread l.  With two spare slots per 32 elements the resident transform
// gives the butterflies of each 16-lane group to its lanes in the order 0, 2, .., 14, 1, 3, ..,
// 15: the first pass then writes its outputs 16t + q, q < 16, as 16-byte pairs, and the eight
// lanes of such a write (butterflies of one parity) cover 32 distinct banks.  Every other
// access of the transform touches the same 16- and 32-lane index sets as in lane order.
template <class C>
constexpr bool lane_perm() {
  return C::WIDE;
}
template <class C>
__device__ __forceinline__ int bfly(int l) {
  if constexpr (lane_perm<C>()) {
    const int m = opaque(l);  // recomputed at each use rather than kept live (or spilled) across the kernel
    return (m & ~15) | (2 * (m & 7)) | ((m >> 3) & 1);
  } else {
    return l;
  }
}


// Position m of the even/odd order -> index in the row.
template <int N>
__device__ __forceinline__ int orig_index(int m) {
  return m < N / 2 ? 2 * m : 2 * (N - 1 - m) + 1;
}

// ------------------------------------------------------------------ reductions
// Cross-lane moves with DPP (no LDS round trip).  update_dpp(old = 0, ...): lanes of rows
// outside ROW_MASK keep 0.
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xf, false));
}
__device__ __forceinline__ float lane63(float v) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Sum over the wave in a fixed order: quad xor 1, 2, half-row mirror, row mirror, then the
// row sums folded into lane 63 by row broadcasts; returned as a wave-uniform value.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp<0xb1>(v);       // quad_perm [1,0,3,2]
  v += dpp<0x4e>(v);       // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);      // row_half_mirror
  v += dpp<0x140>(v);      // row_mirror
  v += dpp<0x142, 0xa>(v); // row_bcast:15 into rows 1 and 3
  v += dpp<0x143, 0xc>(v); // row_bcast:31 into rows 2 and 3
  return lane63(v);
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp<0xb1>(v));
  v = fmaxf(v, dpp<0x4e>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  v = fmaxf(v, dpp<0x142, 0xa>(v));
  v = fmaxf(v, dpp<0x143, 0xc>(v));
  return lane63(v);
}

// Sum of K values over the workgroup in a fixed order (every thread gets the same bits).
// `red` holds 2 * NW * 32 floats; consecutive calls alternate halves, so one barrier per
// call suffices.
template <int T, int K>
__device__ __forceinline__ void block_sum(float (&v)[K], float* red, int& slot) {
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = wave_sum(v[k]);
  if constexpr (T > 64) {
    constexpr int NW = (T + 63) / 64;
    float* r = red + (slot & 1) * (NW * 32);
    ++slot;
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
      for (int k = 0; k < K; ++k) r[(threadIdx.x >> 6) * K + k] = v[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < K; ++k) {
      float s = r[k];
#pragma unroll
      for (int w = 1; w < NW; ++w) s += r[w * K + k];
      v[k] = s;
    }
  }
}

// block_sum for many values over many waves: the workgroup's per-wave partials are summed by the
// lanes of one DPP row (lane w holds wave w's partial; a quad, half-row and row fold, the same in
// every wave), so K values cost K registers after the barrier rather than K x (waves), which
// block_sum's unrolled reads need all at once.  A fixed order again, but another one.
template <int T, int K>
__device__ __forceinline__ void block_sum_lanes(float (&v)[K], float* red, int& slot) {
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = wave_sum(v[k]);
  if constexpr (T > 64) {
    constexpr int NW = (T + 63) / 64;
    static_assert(NW <= 16 && K <= 32, "one DPP row of partials, K values per wave in red");
    float* r = red + (slot & 1) * (NW * 32);
    ++slot;
    const int lane = threadIdx.x & 63;
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < K; ++k) r[(threadIdx.x >> 6) * K + k] = v[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < K; ++k) {
      float t = lane < NW ? r[lane * K + k] : 0.f;
      t += dpp<0xb1>(t);   // quad_perm [1,0,3,2]
      t += dpp<0x4e>(t);   // quad_perm [2,3,0,1]
      t += dpp<0x141>(t);  // row_half_mirror
      t += dpp<0x140>(t);  // row_mirror: every lane of row 0 holds the sum of lanes 0..15
      v[k] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(t), 0));
    }
  }
}

template <int T, int K>
__device__ __forceinline__ void block_max(float (&v)[K], float* red, int& slot) {
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = wave_max(v[k]);
  if constexpr (T > 64) {
    constexpr int NW = (T + 63) / 64;
    float* r = red + (slot & 1) * (NW * 32);
    ++slot;
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
      for (int k = 0; k < K; ++k) r[(threadIdx.x >> 6) * K + k] = v[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < K; ++k) {
      float s = r[k];
#pragma unroll
      for (int w = 1; w < NW; ++w) s = fmaxf(s, r[w * K + k]);
      v[k] = s;
    }
  }
}

// ------------------------------------------------------------------ plan tables
// Twiddle tables, one per pass with stride NS > 1, forward passes first then inverse
// passes: entry [jm][r] = w_N^(r * jm * N / (NS R)), jm < NS, r < R (each table padded to
// an even length so every table starts 16-byte aligned).  Every thread reads its R
// twiddles contiguously.
template <class C, bool INV>
constexpr int pass_radix(int p) {
  return INV ? C::rad[C::NP - 1 - p] : C::rad[p];
}
template <class C, bool INV>
constexpr int pass_ns(int p) {
  return INV ? ns_inv<C>(p) : ns_fwd<C>(p);
}
template <class C, bool INV>
constexpr int tw_offset(int p) {
  int off = 0;
  for (int q = 1; q < C::NP; ++q) {
    if (!INV && q == p) return off;
    off += (ns_fwd<C>(q) * C::rad[q] + 1) & ~1;
  }
  for (int q = 1; q < C::NP; ++q) {
    if (INV && q == p) return off;
    off += (ns_inv<C>(q) * C::rad[C::NP - 1 - q] + 1) & ~1;
  }
  return off;
}

// ------------------------------------------------------------------ FFT passes
enum { SRC_REGS = 0, SRC_LDS = 1, SRC_MID = 2 };
enum { DST_LDS = 0, DST_REGS = 1 };

// One Stockham pass of radix R with stride NS: butterfly j reads elements j + r * N/R,
// multiplies by the twiddles w_N^(r * (j mod NS) * N/(NS R)), takes a length-R DFT, and
// writes element q to (j / NS) * NS * R + (j mod NS) + q * NS.  In place in LDS: every
// read completes (barrier) before any write.  SRC_MID (first inverse pass) reads through
// the eps table: element k = j + r N/R comes from LDS byte address mid[j R + r].z, scaled by
// the complex factor mid[j R + r].xy.
template <class C, int P, bool INV, int SRC, int DST>
__device__ __forceinline__ void fft_pass(float2 (&z)[C::E], float2* __restrict__ lds,
                                         const float2* __restrict__ tw, const float4* __restrict__ mid) {
  constexpr int N = C::N;
  constexpr int T = C::T;
  constexpr int R = pass_radix<C, INV>(P);
  constexpr int NS = pass_ns<C, INV>(P);
  constexpr int NB = N / R;
  constexpr int BP = (NB + T - 1) / T;
  constexpr bool FULL = (NB % T) == 0;
  static_assert(SRC != SRC_REGS || (R == C::R0 && NS == 1), "register source must be the first pass");
  static_assert(DST != DST_REGS || (R == C::R0 && NS == N / C::R0), "register target must be the last pass");
  const int tid = opaque(bfly<C>(threadIdx.x));
  float2 a[BP][R];
  sfor<0, BP>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const int j = tid + T * i;
    if constexpr (SRC == SRC_REGS) {
      sfor<0, R>([&](auto rv) { a[i][decltype(rv)::value] = z[i * R + decltype(rv)::value]; });
    } else if (FULL || j < NB) {
      if constexpr (SRC == SRC_MID) {
        const float4* m = mid + j * R;
        const char* lb = reinterpret_cast<const char*>(lds);
        sfor<0, R>([&](auto rv) {
          constexpr int r = decltype(rv)::value;
          const float4 f = m[r];
          const float2 v = *reinterpret_cast<const float2*>(lb + __float_as_int(f.z));
          a[i][r] = make_float2(f.x * v.x - f.y * v.y, f.x * v.y + f.y * v.x);
          if constexpr (R > 16 && r % 8 == 7) __builtin_amdgcn_sched_barrier(0);
        });
      } else if constexpr (NB % C::PG == 0) {
        const float2* base = lds + pad<C>(j);
        sfor<0, R>([&](auto rv) { a[i][decltype(rv)::value] = base[decltype(rv)::value * pad<C>(NB)]; });
      } else {
        sfor<0, R>([&](auto rv) { a[i][decltype(rv)::value] = lds[pad<C>(j + decltype(rv)::value * NB)]; });
      }
    }
  });
  if constexpr (SRC != SRC_REGS) __syncthreads();
  sfor<0, BP>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const int j = tid + T * i;
    if (FULL || j < NB) {
      const int jm = (NS > 1) ? (j % NS) : 0;
      if constexpr (NS > 1 && R % 2 == 0) {
        // a_r *= w_N^(r jm N/(NS R)) (conjugate on the inverse), read pairwise from the
        // thread's contiguous table row and applied as soon as it arrives
        const float2* tp = tw + tw_offset<C, INV>(P) + jm * R;
        auto twmul = [&](float2& v, float2 t) {
          if constexpr (!INV) v = make_float2(v.x * t.x - v.y * t.y, v.x * t.y + v.y * t.x);
          else v = make_float2(v.x * t.x + v.y * t.y, v.y * t.x - v.x * t.y);
        };
        if constexpr (R % 2 == 0) {
          const float4* t4 = reinterpret_cast<const float4*>(tp);
          sfor<0, R / 2>([&](auto hv) {
            constexpr int h = decltype(hv)::value;
            const float4 q = t4[h];
            if constexpr (h > 0) twmul(a[i][2 * h], make_float2(q.x, q.y));
            twmul(a[i][2 * h + 1], make_float2(q.z, q.w));
          });
        }
      }
      if constexpr (DST == DST_LDS) {
        const int idx0 = (j / NS) * NS * R + jm;
        if constexpr (R % 2 == 1 && NS > 1) {
          // odd radix: the twiddle of each input is applied inside the DFT's pairing step
          const float2* tp = tw + tw_offset<C, INV>(P) + jm * R;
          auto pre = [&](int r, float2 v) {
            if (r == 0) return v;
            const float2 t = tp[r];
            if constexpr (!INV) return make_float2(v.x * t.x - v.y * t.y, v.x * t.y + v.y * t.x);
            else return make_float2(v.x * t.x + v.y * t.y, v.y * t.x - v.x * t.y);
          };
          if constexpr (pad_offsets_ok<C>(NS, R)) {
            float2* base = lds + pad<C>(idx0);
            dft_odd<R, INV>(a[i], pre, [&](int q, float2 v) { base[pad<C>(q * NS)] = v; });
          } else {
            dft_odd<R, INV>(a[i], pre, [&](int q, float2 v) { lds[pad<C>(idx0 + q * NS)] = v; });
          }
        } else if constexpr (pad_offsets_ok<C>(NS, R)) {
          float2* base = lds + pad<C>(idx0);
          dft<R, INV>(a[i], [&](int q, float2 v) { base[pad<C>(q * NS)] = v; });
        } else {
          dft<R, INV>(a[i], [&](int q, float2 v) { lds[pad<C>(idx0 + q * NS)] = v; });
        }
      } else {
        dft<R, INV>(a[i], [&](int q, float2 v) { z[i * R + q] = v; });
      }
    }
  });
  if constexpr (DST == DST_LDS) __syncthreads();
}

template <class C, int P>
__device__ __forceinline__ void fwd_passes(float2 (&z)[C::E], float2* lds, const float2* tw, const float4* mid) {
  if constexpr (P < C::NP) {
    fft_pass<C, P, false, (P == 0 ? SRC_REGS : SRC_LDS), DST_LDS>(z, lds, tw, mid);
    fwd_passes<C, P + 1>(z, lds, tw, mid);
  }
}
template <class C, int P>
__device__ __forceinline__ void inv_passes(float2 (&z)[C::E], float2* lds, const float2* tw, const float4* mid) {
  if constexpr (P < C::NP) {
    fft_pass<C, P, true, (P == 0 ? SRC_MID : SRC_LDS), (P == C::NP - 1 ? DST_REGS : DST_LDS)>(z, lds, tw, mid);
    inv_passes<C, P + 1>(z, lds, tw, mid);
  }
}

// z <- P z for both rows of the pair (Alg. 2: P z = IDCT(eps * DCT(z))).
template <class C>
__device__ __forceinline__ void apply_P(float2 (&z)[C::E], float2* lds, const float2* tw, const float4* mid) {
  fwd_passes<C, 0>(z, lds, tw, mid);
  inv_passes<C, 0>(z, lds, tw, mid);
}

// ------------------------------------------------------------------ resident-table path
// Launch shapes whose passes all use one power-of-two radix R <= 16 with exactly one
// butterfly per thread (T == N/R, N/R a multiple of 16) keep the operator's constants out
// of memory inside the block loop: the twiddles of the last pass (stride N/R, one row
// of R per thread) and the eps factors of the middle step live in registers, loaded once;
// the smaller twiddle tables of the inner passes are copied to LDS once.  The forward
// last pass, the eps step and the inverse first pass are fused: thread t holds Y_k for
// k = t + q N/R after the forward FFT and needs exactly those elements for the inverse
// one, plus Y_{N-k}, which thread N/R - t holds; one LDS exchange brings the partner's
// values, and the element to use is chosen by the factor itself (f_k.y == 0 exactly when
// eps_k == eps_{N-k}).
// An inner pass of odd radix R > R0 whose N/R butterflies are each shared by S = T / (N/R)
// threads (wave-uniform sub-groups; see split_pass).  Its stride must be R0 so that the
// forward/inverse first passes can apply its twiddles to their outputs.
template <class C>
constexpr bool is_split_pass(int p) {
  const int R = C::rad[p];
  return C::NP == 3 && p == 1 && R % 2 == 1 && R > C::R0 && (C::N / R) % 64 == 0 && C::T % (C::N / R) == 0 &&
         C::T / (C::N / R) <= (R - 1) / 2;
}
template <class C>
constexpr bool has_split_pass() {
  return C::NP == 3 && is_split_pass<C>(1);
}
// An inner pass of a radix R < R0 that is not a power of two (odd, or 12) between two radix-R0
// passes (N = R0 R R0): its N/R butterflies spread evenly over the T >= N/R0 threads, each read
// once and transformed by one thread with its twiddles applied to the inputs.
template <class C>
constexpr bool is_small_inner_pass(int p) {
  const int R = C::rad[p];
  return C::NP == 3 && p == 1 && (R & (R - 1)) != 0 && (R % 2 == 1 || R == 12) && R < C::R0 && C::T % 64 == 0 &&
         (C::N / R) % C::T == 0;
}
// Resident shapes: first and last radix R0 (a power of two <= 16), one butterfly of those passes
// per thread, and either a split inner pass or inner radices that are powers of two dividing R0
// in a palindromic sequence (so that the inverse transform meets the same radices and strides,
// and reuses the forward twiddle tables conjugated); an inner pass of radix R gives each thread
// R0 / R butterflies.
template <class C>
constexpr bool resident_ok() {
  constexpr int R0 = C::R0;
  if (!(C::NP >= 2 && R0 <= 16 && (R0 & (R0 - 1)) == 0 && C::rad[C::NP - 1] == R0 && (C::N / R0) % C::PG == 0))
    return false;
  if (has_split_pass<C>()) return C::T >= C::N / R0;
  if (is_small_inner_pass<C>(1)) return C::T >= C::N / R0 && (C::N / C::rad[1]) % C::PG == 0;
  for (int p = 0; p < C::NP; ++p) {
    const int r = C::rad[p];
    if (r < 2 || (r & (r - 1)) != 0 || R0 % r != 0 || r != C::rad[C::NP - 1 - p]) return false;
    if ((C::N / r) % C::PG != 0) return false;
  }
  return C::T == C::N / R0;
}
// LDS slots (float2) of the inner-pass twiddle tables (passes 1 .. NP-2), after the FFT buffer
template <class C>
constexpr int small_tw_offset(int p) {
  int off = 0;
  for (int q = 1; q < p; ++q) off += ns_fwd<C>(q) * C::rad[q];
  return off;
}
// LDS after the FFT buffer on the resident path: the inner-pass twiddle tables, then (with a
// split pass) the 256-byte lane order of its butterflies
template <class C>
constexpr int small_tw_total() {
  return resident_ok<C>() ? small_tw_offset<C>(C::NP - 1) + (has_split_pass<C>() ? 32 : 0) : 0;
}

// eps factors f_k of the fused step for the thread's elements k = t + q N/R: kept as R complex
// values, or -- COMPACT, for kernels whose block loop is register-bound on the split shape (which
// also keep only powers 1 and 4 of the last-pass twiddle, see stored_tw) -- as
// e^{i pi t/N}/N and a mask (bit 2q: eps_k < 0, bit 2q + 1: eps_k != eps_{N-k}), from which
// f_k = eps_k / N or eps_k e^{i pi k/N} / N = eps_k (e^{i pi t/N} / N) e^{i pi q/R} is rebuilt at
// each use.
template <class C>
constexpr bool compact_eps() {
  return has_split_pass<C>() || (C::W >= 4 && C::R0 == 16);  // split shape, or a 128-register budget
}
// vhat of the quantizer's block loop kept in private memory between its steps (16-byte loads and
// stores of the whole array around the two vhat-steps of a block) rather than in registers, where
// the 128-register budget would otherwise spill it value by value inside the transforms
template <class C>
constexpr bool vh_in_memory() {
  return !has_split_pass<C>() && C::W >= 4 && C::R0 == 16 && C::E % 2 == 0;
}
template <class C, bool COMPACT>
struct EpsRegs {
  float2 f[C::R0];
};
template <class C>
struct EpsRegs<C, true> {
  float2 base;
  uint32_t bits;
};
// e^{i pi q / 16}
struct Half32 {
  static constexpr double c[16] = {1.0, 0.9807852804032304, 0.9238795325112867, 0.8314696123025452,
                                   0.7071067811865476, 0.5555702330196023, 0.38268343236508984, 0.19509032201612833,
                                   0.0, -0.1950903220161282, -0.3826834323650897, -0.555570233019602,
                                   -0.7071067811865475, -0.8314696123025453, -0.9238795325112867, -0.9807852804032304};
  static constexpr double s[16] = {0.0, 0.19509032201612825, 0.3826834323650898, 0.5555702330196022,
                                   0.7071067811865475, 0.8314696123025452, 0.9238795325112867, 0.9807852804032304,
                                   1.0, 0.9807852804032304, 0.9238795325112867, 0.8314696123025455,
                                   0.7071067811865476, 0.5555702330196022, 0.3826834323650899, 0.1950903220161286};
};
// f_k for element q, and whether it takes the partner value (eps_k != eps_{N-k})
template <class C, int q, bool COMPACT>
__device__ __forceinline__ float2 eps_factor(const EpsRegs<C, COMPACT>& e, bool& partner) {
  if constexpr (COMPACT) {
    static_assert(C::R0 == 16, "compact eps factors assume radix 16");
    partner = (e.bits >> (2 * q + 1)) & 1u;
    const bool neg = (e.bits >> (2 * q)) & 1u;
    constexpr float cx = static_cast<float>(Half32::c[q]), cy = static_cast<float>(Half32::s[q]);
    constexpr float inv_n = static_cast<float>(1.0 / C::N);
    const float2 g = partner ? make_float2(e.base.x * cx - e.base.y * cy, e.base.x * cy + e.base.y * cx)
                             : make_float2(inv_n, 0.f);
    return neg ? make_float2(-g.x, -g.y) : g;
  } else {
    const float2 f = e.f[q];
    partner = f.y != 0.f;
    return f;
  }
}

template <class C, bool COMPACT = false>
struct ResRegs {
  static constexpr bool compact = COMPACT;
  float2 tw[C::R0];         // w_N^(r t) for r in {1, 2, 3, 4, 8, 12}: the rest are products of two of these
  EpsRegs<C, COMPACT> eps;  // eps factors of the fused step for elements k = t + r N/R
};

// twiddle r of the last pass from the stored powers (R = 16: r = 4a + b, w_r = w_4a * w_b)
__device__ __forceinline__ float2 cmulf(float2 x, float2 y) {
  return make_float2(x.x * y.x - x.y * y.y, x.x * y.y + x.y * y.x);
}
// stored power r of w_N^t: all six kept, or (compact) only r = 1 and 4 with 2, 3, 8, 12 derived
template <class C, int r, class RR>
__device__ __forceinline__ float2 stored_tw(const RR& rr) {
  if constexpr (!RR::compact || r == 1 || r == 4) return rr.tw[r];
  else if constexpr (r == 2) return cmulf(rr.tw[1], rr.tw[1]);
  else if constexpr (r == 3) return cmulf(stored_tw<C, 2>(rr), rr.tw[1]);
  else if constexpr (r == 8) return cmulf(rr.tw[4], rr.tw[4]);
  else return cmulf(stored_tw<C, 8>(rr), rr.tw[4]);  // r == 12
}
template <class C, int r, class RR>
__device__ __forceinline__ float2 last_tw(const RR& rr) {
  if constexpr (C::R0 < 16 || r <= 4 || r == 8 || r == 12) {
    return stored_tw<C, r>(rr);
  } else {
    constexpr int hi = r & ~3, lo = r & 3;
    return cmulf(stored_tw<C, hi>(rr), stored_tw<C, lo>(rr));
  }
}

// Before each last pass: declare the stored powers modified (in place, no instruction), so
// the products formed from them are neither hoisted out of the block loop nor shared between
// the two last passes of one application of P, either of which would keep nine more complex
// values live.
template <class C, class RR>
__device__ __forceinline__ void launder_powers(RR& rr) {
  if constexpr (C::R0 == 16) {
    if constexpr (RR::compact)
      asm volatile("" : "+v"(rr.tw[1].x), "+v"(rr.tw[1].y), "+v"(rr.tw[4].x), "+v"(rr.tw[4].y));
    else
      asm volatile(""
                   : "+v"(rr.tw[1].x), "+v"(rr.tw[1].y), "+v"(rr.tw[2].x), "+v"(rr.tw[2].y), "+v"(rr.tw[3].x),
                     "+v"(rr.tw[3].y), "+v"(rr.tw[4].x), "+v"(rr.tw[4].y), "+v"(rr.tw[8].x), "+v"(rr.tw[8].y),
                     "+v"(rr.tw[12].x), "+v"(rr.tw[12].y));
  }
  // the compact eps factors are rebuilt inside the block loop, not hoisted out of it as R live values
  if constexpr (RR::compact) asm volatile("" : "+v"(rr.eps.base.x), "+v"(rr.eps.base.y), "+v"(rr.eps.bits));
}

template <class C, class RR>
__device__ __forceinline__ void resident_load(RR& rr, float2* lds, const float2* __restrict__ tw,
                                              const float4* __restrict__ mid) {
  constexpr int R = C::R0;
  constexpr int NB = C::N / R;
  const int t = bfly<C>(threadIdx.x);
  const int tl = (C::T == NB || t < NB) ? t : 0;  // threads past the last butterfly load row 0 (unused)
  const float4* t4 = reinterpret_cast<const float4*>(tw + tw_offset<C, false>(C::NP - 1) + tl * R);
  sfor<0, R / 2>([&](auto hv) {
    constexpr int h = decltype(hv)::value;
    constexpr bool keep0 = (R < 16) || (2 * h <= 4 || 2 * h == 8 || 2 * h == 12);
    constexpr bool keep1 = (R < 16) || (2 * h + 1 <= 4);
    if constexpr (keep0 || keep1) {
      const float4 q = t4[h];
      if constexpr (keep0) rr.tw[2 * h] = make_float2(q.x, q.y);
      if constexpr (keep1) rr.tw[2 * h + 1] = make_float2(q.z, q.w);
    }
  });
  if constexpr (RR::compact) {
    uint32_t bits = 0;
    sfor<0, R>([&](auto rv) {
      constexpr int q = decltype(rv)::value;
      const float4 m = mid[tl * R + q];  // {Re f_k, Im f_k, -, eps_k}
      bits |= (m.w < 0.f ? 1u : 0u) << (2 * q);
      bits |= (m.y != 0.f ? 1u : 0u) << (2 * q + 1);
    });
    float sn, cs;
    sincospif(static_cast<float>(tl) / static_cast<float>(C::N), &sn, &cs);
    rr.eps.bits = bits;
    rr.eps.base = make_float2(cs * static_cast<float>(1.0 / C::N), sn * static_cast<float>(1.0 / C::N));
  } else {
    sfor<0, R>([&](auto rv) {
      const float4 m = mid[tl * R + decltype(rv)::value];
      rr.eps.f[decltype(rv)::value] = make_float2(m.x, m.y);
    });
  }
  // inner-pass tables, transposed so that the lanes of a wave (consecutive jm) read
  // consecutive LDS words (the [jm][r] rows of the global layout are 8R bytes apart, which
  // would put every lane of a 16-lane group on the same banks): [r][jm] for a split pass,
  // else [r / 2][jm] pairs (entries r and r + 1 side by side, one 16-byte read per pair)
  float2* small = lds + C::LDS;
  sfor<1, C::NP - 1>([&](auto pv) {
    constexpr int P = decltype(pv)::value;
    constexpr int NS = ns_fwd<C>(P);
    constexpr int RP = C::rad[P];
    constexpr int OFF = small_tw_offset<C>(P);
    for (int i = t; i < NS * RP; i += C::T) {
      const int jm = i / RP, r = i % RP;
      if constexpr (is_split_pass<C>(P) || is_small_inner_pass<C>(P))
        small[OFF + r * NS + jm] = tw[tw_offset<C, false>(P) + i];
      else small[OFF + 2 * ((r / 2) * NS + jm) + (r & 1)] = tw[tw_offset<C, false>(P) + i];
    }
  });
  if constexpr (has_split_pass<C>()) {
    const unsigned char* order = SplitOrder<C::rad[1]>::j;
    unsigned char* dst = reinterpret_cast<unsigned char*>(small + small_tw_offset<C>(C::NP - 1));
    for (int i = threadIdx.x; i < 256; i += C::T) dst[i] = order[i];
  }
  __syncthreads();
}

template <bool INV>
__device__ __forceinline__ float2 twmul(float2 v, float2 t) {
  if constexpr (!INV) return make_float2(v.x * t.x - v.y * t.y, v.x * t.y + v.y * t.x);
  else return make_float2(v.x * t.x + v.y * t.y, v.y * t.x - v.x * t.y);
}

// Inner pass p (1 <= p <= NP-2) of the resident path: radix R = rad[p], stride NS = the
// product of the radices before it, LDS -> LDS, twiddles from the LDS copy of the pass-p table;
// thread t takes butterflies t + T i, i < R0 / R.
template <class C, int P, bool INV>
__device__ __forceinline__ void res_small_pass(float2* __restrict__ lds, int t) {
  constexpr int R = C::rad[P];
  constexpr int NB = C::N / R;
  constexpr int NS = ns_fwd<C>(P);
  constexpr int BPT = NB / C::T;
  static_assert(BPT * C::T == NB && NB % C::PG == 0 && pad_offsets_ok<C>(NS, R), "small inner pass shape");
  float2 a[BPT][R];
  sfor<0, BPT>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const float2* rb = lds + pad<C>(t + C::T * i);
    sfor<0, R>([&](auto rv) { a[i][decltype(rv)::value] = rb[decltype(rv)::value * pad<C>(NB)]; });
  });
  __syncthreads();
  sfor<0, BPT>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const int j = t + C::T * i;
    const int jm = j % NS;
    const float2* tb = lds + C::LDS + small_tw_offset<C>(P) + jm;  // table [r][jm]
    auto pre = [&](int r, float2 v) {
      if (r == 0) return v;
      const float2 w = tb[r * NS];
      return INV ? make_float2(v.x * w.x + v.y * w.y, v.y * w.x - v.x * w.y)
                 : make_float2(v.x * w.x - v.y * w.y, v.x * w.y + v.y * w.x);
    };
    float2* wb = lds + pad<C>((j / NS) * NS * R + jm);
    dft_small<R, INV>(a[i], pre, [&](int q, float2 v) { wb[pad<C>(q * NS)] = v; });
  });
  __syncthreads();
}

template <class C, int P, bool INV>
__device__ __forceinline__ void res_inner_pass(float2* __restrict__ lds, int t) {
  constexpr int R = C::rad[P];
  constexpr int NB = C::N / R;
  constexpr int NS = ns_fwd<C>(P);
  constexpr int BPT = NB / C::T;
  static_assert(BPT * C::T == NB && BPT * R == C::R0, "inner pass butterflies per thread");
  float2 a[BPT][R];
  sfor<0, BPT>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const float2* rb = lds + pad<C>(t + C::T * i);
    sfor<0, R>([&](auto rv) { a[i][decltype(rv)::value] = rb[decltype(rv)::value * pad<C>(NB)]; });
  });
  __syncthreads();
  static_assert(R % 2 == 0 && small_tw_offset<C>(P) % 2 == 0 && C::LDS % 2 == 0, "16-byte twiddle pairs");
  static_assert(pad_offsets_ok<C>(NS, R), "inner pass stride");
  sfor<0, BPT>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const int j = t + C::T * i;
    const int jm = j % NS;
    const float4* tb = reinterpret_cast<const float4*>(lds + C::LDS + small_tw_offset<C>(P)) + jm;  // [r / 2][jm]
    dft_pow2_tw<R, INV>(a[i], [&](auto rv) {
      constexpr int r = decltype(rv)::value;
      const float4 q = tb[(r / 2) * NS];
      return (r & 1) ? make_float2(q.z, q.w) : make_float2(q.x, q.y);
    });
    float2* wb = lds + pad<C>((j / NS) * NS * R + jm);
    sfor<0, R>([&](auto qv) { wb[pad<C>(decltype(qv)::value * NS)] = a[i][decltype(qv)::value]; });
  });
  __syncthreads();
}

// Split inner pass: odd radix R, stride NS = R0, NB = N/R butterflies, each shared by the
// S = T/NB threads t = j + s NB (s is uniform across a wave).  Every sub-group streams the
// R inputs of butterfly j from LDS once, forming the pair sums and differences
// a_r +- a_{R-r}, and accumulates only its own share of the (R-1)/2 output pairs (q, R-q);
// the twiddles were applied by the pass before.  All sub-groups run one code path: their
// DFT constants come from a table in constant memory at a wave-uniform address (scalar
// loads into SGPR operands of the FMAs).
template <class C, int P>
struct SplitShape {
  static constexpr int R = C::rad[P];
  static constexpr int NB = C::N / R;
  static constexpr int S = C::T / NB;         // threads per butterfly
  static constexpr int H = (R - 1) / 2;       // output pairs (q, R - q)
  static constexpr int QP = (H + S - 1) / S;  // output pairs per sub-group
};

// {cos, sin}(2 pi r q / R) for sub-group s, input pair r = 1..H and output pair
// q = s QP + 1 + i, at [((s H + r - 1) QP + i) 2] (zero past the last pair).
template <int R, int S>
struct SplitCoef {
  static constexpr int H = (R - 1) / 2;
  static constexpr int QP = (H + S - 1) / S;
  float v[S * H * QP * 2];
};
template <int R, int S>
constexpr SplitCoef<R, S> make_split_coef() {
  SplitCoef<R, S> t{};
  constexpr int H = SplitCoef<R, S>::H, QP = SplitCoef<R, S>::QP;
  for (int s = 0; s < S; ++s)
    for (int r = 1; r <= H; ++r)
      for (int i = 0; i < QP; ++i) {
        const int q = s * QP + 1 + i;
        const int idx = ((s * H + r - 1) * QP + i) * 2;
        if (q <= H) {
          t.v[idx] = CisTab<R>::c[(r * q) % R];
          t.v[idx + 1] = CisTab<R>::s[(r * q) % R];
        }
      }
  return t;
}
template <int R, int S>
__constant__ SplitCoef<R, S> split_coef = make_split_coef<R, S>();

template <class C, int P, bool INV>
__device__ __forceinline__ void split_pass(float2* __restrict__ lds, int t) {
  using SS = SplitShape<C, P>;
  constexpr int R = SS::R;
  constexpr int NB = SS::NB;
  constexpr int S = SS::S;
  constexpr int QP = SS::QP;
  constexpr int H = SS::H;
  constexpr int NS = ns_fwd<C>(P);
  static_assert(NB % 64 == 0 && NS % C::PG == 0, "split pass strides");
  const int s = __builtin_amdgcn_readfirstlane(t / NB);  // uniform across a wave
  // butterfly of this lane: the order of SplitOrder (bank-conflict-free reads in seven of the
  // eight 32-lane halves, conflict-free writes), kept in LDS after the twiddle tables
  static_assert(NB == 256, "split-pass lane order covers 256 butterflies");
  const int j = reinterpret_cast<const unsigned char*>(lds + C::LDS + small_tw_offset<C>(C::NP - 1))[t - s * NB];
  const float* __restrict__ cf = split_coef<R, S>.v + s * (H * QP * 2);
  const float2* rb = lds + pad<C>(j);
  const float2 x0 = rb[0];
  float2 re[QP], im[QP];
  sfor<0, QP>([&](auto iv) {
    re[decltype(iv)::value] = x0;
    im[decltype(iv)::value] = make_float2(0.f, 0.f);
  });
  float2 sum = x0;
  // Input pairs in chunks of CH, software-pipelined: the LDS reads and constant loads of chunk
  // c + 1 are issued after an explicit wait for those of chunk c, so that the wait (LDS and
  // scalar loads share one counter, and scalar loads return out of order) never covers loads
  // that were just issued; chunk c's FMAs then run while chunk c + 1's loads are in flight.
  constexpr int CH = 1;
  constexpr int NCH = (H + CH - 1) / CH;
  float2 pin[2][CH], mnn[2][CH];
  float cin[2][CH][2 * QP];
  auto fetch = [&](auto cv) {
    constexpr int c = decltype(cv)::value;
    sfor<0, CH>([&](auto uv) {
      constexpr int u = decltype(uv)::value;
      constexpr int r = c * CH + u + 1;
      if constexpr (r <= H) {
        pin[c % 2][u] = rb[r * pad<C>(NB)];
        mnn[c % 2][u] = rb[(R - r) * pad<C>(NB)];
        sfor<0, 2 * QP>([&](auto ev) { cin[c % 2][u][decltype(ev)::value] = cf[(r - 1) * QP * 2 + decltype(ev)::value]; });
      }
    });
  };
  fetch(std::integral_constant<int, 0>{});
  sfor<0, NCH>([&](auto cv) {
    constexpr int c = decltype(cv)::value;
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): chunk c's values are in registers
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (c + 1 < NCH) fetch(std::integral_constant<int, c + 1>{});
    __builtin_amdgcn_sched_barrier(0);
    sfor<0, CH>([&](auto uv) {
      constexpr int u = decltype(uv)::value;
      if constexpr (c * CH + u + 1 <= H) {
        const float2 p = pin[c % 2][u], m = mnn[c % 2][u];
        const float2 sp = cadd(p, m), dm = csub(p, m);
        sum = cadd(sum, sp);
        sfor<0, QP>([&](auto iv) {
          constexpr int i = decltype(iv)::value;
          const float cc = cin[c % 2][u][2 * i], sn = cin[c % 2][u][2 * i + 1];
          re[i].x = fmaf(sp.x, cc, re[i].x);
          re[i].y = fmaf(sp.y, cc, re[i].y);
          im[i].x = fmaf(dm.x, sn, im[i].x);
          im[i].y = fmaf(dm.y, sn, im[i].y);
        });
      }
    });
  });
  __syncthreads();
  // forward: A_q = re - i im, A_{R-q} = re + i im; the inverse swaps them
  const int q0 = s * QP + 1;
  float2* wb = lds + pad<C>((j / NS) * NS * R + (j % NS));
  sfor<0, QP>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const float2 minus = make_float2(re[i].x + im[i].y, re[i].y - im[i].x);
    const float2 plus = make_float2(re[i].x - im[i].y, re[i].y + im[i].x);
    if (H % QP == 0 || q0 + i <= H) {
      wb[(q0 + i) * pad<C>(NS)] = INV ? plus : minus;
      wb[(R - q0 - i) * pad<C>(NS)] = INV ? minus : plus;
    }
  });
  if (s == 0) wb[0] = sum;
  __syncthreads();
}

template <class C, int P, bool INV>
__device__ __forceinline__ void res_inner_passes(float2* lds, int t) {
  if constexpr (P >= 1 && P <= C::NP - 2) {
    // the radices are palindromic: the inverse FFT meets the same radices and strides as the forward one
    if constexpr (is_split_pass<C>(P)) split_pass<C, P, INV>(lds, t);
    else if constexpr (is_small_inner_pass<C>(P)) res_small_pass<C, P, INV>(lds, t);
    else res_inner_pass<C, P, INV>(lds, t);
    res_inner_passes<C, P + 1, INV>(lds, t);
  }
}

// First pass (stride 1) of either direction: a[] -> LDS, element q to t R + q.  When the
// next pass is a split pass its input twiddles are applied here, to the outputs: element
// t R0 + q is input r = t / (NB1 / R0) of a butterfly with j mod R0 = q, so its twiddle is
// entry [r][q] of the LDS copy of that pass's table.
template <class C, bool INV>
__device__ __forceinline__ void res_first_pass(float2 (&a)[C::R0], float2* lds, int t) {
  constexpr int R = C::R0;
  static_assert(C::PG % R == 0, "first pass: element q of butterfly t at slot pad(t R) + q");
  float2* wb = lds + pad<C>(t * R);
  if constexpr (has_split_pass<C>()) {
    constexpr int NB1 = C::N / C::rad[1];
    static_assert(NB1 % R == 0 && ns_fwd<C>(1) == R, "split pass after the first pass");
    const float4* tb = reinterpret_cast<const float4*>(lds + C::LDS + small_tw_offset<C>(1) + (t / (NB1 / R)) * R);
    dft_pow2<R, INV>(a);
    wb[0] = a[0];
    sfor<0, R / 2>([&](auto hv) {
      constexpr int h = decltype(hv)::value;
      const float4 q = tb[h];
      if constexpr (h > 0) wb[2 * h] = twmul<INV>(a[2 * h], make_float2(q.x, q.y));
      wb[2 * h + 1] = twmul<INV>(a[2 * h + 1], make_float2(q.z, q.w));
    });
  } else if constexpr (lane_perm<C>()) {
    static_assert(C::PW % 2 == 0 && (C::PG / R) % 2 == 0, "16-byte aligned output pairs");
    float2 o[R];
    dft<R, INV>(a, [&](int q, float2 v) { o[q] = v; });
    float4* w4 = reinterpret_cast<float4*>(wb);
    sfor<0, R / 2>([&](auto hv) {
      constexpr int h = decltype(hv)::value;
      w4[h] = make_float4(o[2 * h].x, o[2 * h].y, o[2 * h + 1].x, o[2 * h + 1].y);
    });
  } else {
    dft<R, INV>(a, [&](int q, float2 v) { wb[q] = v; });
  }
}

// z <- P z on the resident path.  Threads past the last radix-R0 butterfly (T > N/R0, only
// with a split pass) take part in the split pass and the barriers only.
template <class C, class RR>
__device__ __forceinline__ void apply_P_res(float2 (&z)[C::E], float2* lds, RR& rr) {
  constexpr int N = C::N;
  constexpr int R = C::R0;
  constexpr int NB = N / R;
  const int t = opaque(bfly<C>(threadIdx.x));
  const bool act = (C::T == NB) || t < NB;
  // forward pass 0 (stride 1): registers -> LDS
  if (act) {
    float2 a[R];
    sfor<0, R>([&](auto rv) { a[decltype(rv)::value] = z[decltype(rv)::value]; });
    res_first_pass<C, false>(a, lds, t);
  }
  __syncthreads();
  res_inner_passes<C, 1, false>(lds, t);
  // forward last pass (stride N/R), fused with the eps step and the inverse first pass
  float2 y[R];
  const float2* rb = lds + pad<C>(t);
  // the last pass reads and writes the same elements t + q N/R, which no other thread touches:
  // no barrier between its read and its write
  if (act) sfor<0, R>([&](auto rv) { y[decltype(rv)::value] = rb[decltype(rv)::value * pad<C>(NB)]; });
  launder_powers<C>(rr);
  if (act) {
    dft_pow2_tw<R, false>(y, [&](auto rv) { return last_tw<C, decltype(rv)::value>(rr); });  // y[q] = Y_{t + q NB}
    float2* wb = lds + pad<C>(t);
    sfor<0, R>([&](auto qv) { wb[decltype(qv)::value * pad<C>(NB)] = y[decltype(qv)::value]; });
  }
  __syncthreads();
  if (act) {
    // partner values Y_{N - t - q NB} (slot pad<C>(N - t) - q pad<C>(NB); for t = 0, q = 0 the
    // slot just past the buffer is read but never used: k = 0 pairs with itself)
    const float2* pb = lds + pad<C>(N - t);
    sfor<0, R>([&](auto qv) {
      constexpr int q = decltype(qv)::value;
      bool partner;
      const float2 fq = eps_factor<C, q>(rr.eps, partner);
      const float2 own = y[q];
      const float2 oth = pb[-q * pad<C>(NB)];
      const float2 v = partner ? oth : own;
      y[q] = make_float2(fq.x * v.x - fq.y * v.y, fq.x * v.y + fq.y * v.x);
      if constexpr (q % 2 == 1) __builtin_amdgcn_sched_barrier(0);  // bound partner values in flight
    });
  }
  __syncthreads();
  // inverse pass 0 (stride 1)
  if (act) res_first_pass<C, true>(y, lds, t);
  __syncthreads();
  res_inner_passes<C, 1, true>(lds, t);
  // inverse last pass (stride N/R): LDS -> registers
  launder_powers<C>(rr);
  if (act) {
    sfor<0, R>([&](auto rv) { z[decltype(rv)::value] = rb[decltype(rv)::value * pad<C>(NB)]; });
    dft_pow2_tw<R, true>(z, [&](auto rv) { return last_tw<C, decltype(rv)::value>(rr); });
  }
}

// ------------------------------------------------------------------ greedy step
__device__ __forceinline__ int8_t sgn8(float x) { return x > 0.f ? 1 : (x < 0.f ? -1 : 0); }
// sign(x) * c with sign(0) = 0, as the median of (-c, x 2^160, c): every nonzero float times 2^160
// is at least 2^11 in magnitude (or infinite), above any step size c -- on the normalised rows
// (max |w| < 1) c <= ||x||_2 <= ||w||_2 < sqrt(N) < 2^8, since no step raises the residual norm --
// so the median is exactly +-c; x = +-0 gives +-0, and x -/+ 0 leaves x unchanged up to the sign
// of a zero.  Two VALU operations instead of a compare, a copysign and a select.
__device__ __forceinline__ float sgn_times(float x, float c) {
  return __builtin_amdgcn_fmed3f(-c, __builtin_amdgcn_ldexpf(x, 160), c);
}

// s / N: exact for a power of two; otherwise s times the float nearest 1 / N (within one ulp of the
// quotient, and the step size c only enters the greedy as c itself)
template <int N>
__device__ __forceinline__ float div_n(float s) {
  return s * static_cast<float>(1.0 / N);
}

// One atomic greedy step of Alg. 2 on both rows: c = ||x||_1 / N, delta = sign(x) c
// (sign(0) = 0), x -= delta, and acc += delta when ACC.  Returns (c_a, c_b).  With
// `trace`, the signs of one side are written in row order.
template <class C, bool ACC>
__device__ __forceinline__ float2 greedy_step(float2 (&z)[C::E], float2 (&acc)[C::E], float* red, int& slot,
                                              int8_t* trace, int side) {
  float s[2] = {0.f, 0.f};
#pragma unroll
  for (int e = 0; e < C::E; ++e) {
    s[0] += fabsf(z[e].x);
    s[1] += fabsf(z[e].y);
  }
  block_sum<C::T, 2>(s, red, slot);
  const float ca = div_n<C::N>(s[0]);
  const float cb = div_n<C::N>(s[1]);
  if (trace != nullptr) {
    const int tid = opaque(bfly<C>(threadIdx.x));
#pragma unroll
    for (int i = 0; i < C::B0; ++i) {
      const int j = tid + C::T * i;
      if (j < C::NB0) {
#pragma unroll
        for (int r = 0; r < C::R0; ++r) {
          const float2 v = z[i * C::R0 + r];
          trace[orig_index<C::N>(j + r * C::NB0)] = sgn8(side ? v.y : v.x);
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < C::E; ++e) {
    const float da = sgn_times(z[e].x, ca);
    const float db = sgn_times(z[e].y, cb);
    if constexpr (ACC) {
      acc[e].x += da;
      acc[e].y += db;
    }
    z[e].x -= da;
    z[e].y -= db;
  }
  return make_float2(ca, cb);
}

// ------------------------------------------------------------------ loads / stores
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(__half v) { return __half2float(v); }
__device__ __forceinline__ float to_f32(bf16_t v) { return bf16_to_f32(v); }

// Load rows a (and b if >= 0) into the greedy register layout, in even/odd order.
// `tid` is the thread index (a laundered copy in loops whose other values are invariant, so
// that the element offsets are recomputed rather than kept live across the loop).
template <class C, class IT>
__device__ __forceinline__ void load_pair_t(float2 (&z)[C::E], const IT* __restrict__ w, int64_t ldw, int64_t ra,
                                            int64_t rb, int tid = bfly<C>(threadIdx.x)) {
  const IT* __restrict__ pa = w + ra * ldw;
  const IT* __restrict__ pb = w + (rb >= 0 ? rb : ra) * ldw;
#pragma unroll
  for (int i = 0; i < C::B0; ++i) {
    const int j = tid + C::T * i;
#pragma unroll
    for (int r = 0; r < C::R0; ++r) {
      float2 v = make_float2(0.f, 0.f);
      if (C::NB0 % C::T == 0 || j < C::NB0) {
        const int src = orig_index<C::N>(j + r * C::NB0);
        v.x = to_f32(pa[src]);
        v.y = to_f32(pb[src]);
      }
      z[i * C::R0 + r] = v;
    }
  }
  if (rb < 0) {
#pragma unroll
    for (int e = 0; e < C::E; ++e) z[e].y = 0.f;
  }
}

template <class C, class F>
__device__ __forceinline__ void for_each_elem(F&& f, int tid = bfly<C>(threadIdx.x)) {
#pragma unroll
  for (int i = 0; i < C::B0; ++i) {
    const int j = tid + C::T * i;
    if (j < C::NB0) {
#pragma unroll
      for (int r = 0; r < C::R0; ++r) f(i * C::R0 + r, orig_index<C::N>(j + r * C::NB0));
    }
  }
}

// Rows a and b of w (b if >= 0, else zeros) into the LDS buffer in row order as float2 (row a
// in .x, row b in .y), times the rotation's sign s_i when ROT.  Each thread issues its loads in
// batches of eight per row before the first store, so that several are in flight at once.
template <class C, bool ROT, class IT>
__device__ __forceinline__ void stage_pair_t(float2* lds, const IT* __restrict__ w, int64_t ldw, int64_t ra,
                                             int64_t rb, uint64_t seed, int tid) {
  constexpr int K = (C::N + C::T - 1) / C::T;  // entries per thread and row
  constexpr int BATCH = 8;
  const IT* __restrict__ pa = w + ra * ldw;
  const IT* __restrict__ pb = w + (rb >= 0 ? rb : ra) * ldw;
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += BATCH) {
    IT va[BATCH], vb[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int i = tid + (k0 + k) * C::T;
      if (k0 + k < K && (C::N % C::T == 0 || i < C::N)) {
        va[k] = pa[i];
        vb[k] = pb[i];
      }
    }
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int i = tid + (k0 + k) * C::T;
      if (k0 + k < K && (C::N % C::T == 0 || i < C::N)) {
        float2 v = make_float2(to_f32(va[k]), rb >= 0 ? to_f32(vb[k]) : 0.f);
        if constexpr (ROT) v = rv_scale(v, rot_sign(seed, i));
        lds[i] = v;
      }
    }
  }
}

// w (or R w when ROT: the rotation fused into the load) for both rows of the pair, handed to
// f(e, t) entry by entry in the greedy register layout (t = both rows' values at that entry,
// times 1 / sqrt(2^a) when ROT).  The rows are staged in the LDS buffer in row order; for ROT
// they are signed there and mixed by C_b and the Hadamard factor -- the operations of the
// standalone rotation kernel in the same order.  Uses the whole buffer, with a barrier on entry
// (a transform may still read it) and on exit (the next transform overwrites it).
template <class C, bool ROT, class F>
__device__ __forceinline__ void load_pair_staged(const void* w, int dtype, int64_t ldw, int64_t ra, int64_t rb,
                                                 uint64_t seed, float scale, float2* lds, F&& f) {
  const int tid = bfly<C>(threadIdx.x);
  __syncthreads();
  if (dtype == KASHIN_F16) stage_pair_t<C, ROT>(lds, static_cast<const __half*>(w), ldw, ra, rb, seed, tid);
  else if (dtype == KASHIN_BF16) stage_pair_t<C, ROT>(lds, static_cast<const bf16_t*>(w), ldw, ra, rb, seed, tid);
  else stage_pair_t<C, ROT>(lds, static_cast<const float*>(w), ldw, ra, rb, seed, tid);
  __syncthreads();
  if constexpr (ROT) {
    constexpr int B = rot_odd_part(C::N);
    rot_odd_factor_fixed<B, false, C::T, C::N>(lds, tid);
    rot_hadamard<B, C::T>(lds, C::N, tid);
  }
  for_each_elem<C>([&](int e, int i) { f(e, ROT ? rv_scale(lds[i], scale) : lds[i]); }, tid);
  __syncthreads();
}

template <class C>
__device__ __forceinline__ void load_pair(float2 (&z)[C::E], const void* w, int dtype, int64_t ldw, int64_t ra,
                                          int64_t rb, int tid = bfly<C>(threadIdx.x)) {
  if (dtype == KASHIN_F16) load_pair_t<C>(z, static_cast<const __half*>(w), ldw, ra, rb, tid);
  else if (dtype == KASHIN_BF16) load_pair_t<C>(z, static_cast<const bf16_t*>(w), ldw, ra, rb, tid);
  else load_pair_t<C>(z, static_cast<const float*>(w), ldw, ra, rb, tid);
}

// z <- w * scale - z for the pair (rows reloaded in the register layout); zero for a bad row.
template <class C>
__device__ __forceinline__ void sub_from_rows(float2 (&z)[C::E], const void* w, int dtype, int64_t ldw, int64_t ra,
                                              int64_t rb, float2 scale, bool bad_a, bool bad_b) {
  float2 t[C::E];
  load_pair<C>(t, w, dtype, ldw, ra, rb);
#pragma unroll
  for (int e = 0; e < C::E; ++e) {
    z[e].x = bad_a ? 0.f : fmaf(t[e].x, scale.x, -z[e].x);
    z[e].y = bad_b ? 0.f : fmaf(t[e].y, scale.y, -z[e].y);
  }
}



// Per-row power-of-two scale s (|w| * s in [0.5, 1)) and a NaN/Inf flag, for both rows.
// Returns the scales and zeroes a row that is not finite.
template <class C>
__device__ __forceinline__ void normalise_pair(float2 (&z)[C::E], float* red, int& slot, float2& scale,
                                               float2& unscale, bool& bad_a, bool& bad_b) {
  float mx[2] = {0.f, 0.f};
  float nf[2] = {0.f, 0.f};
#pragma unroll
  for (int e = 0; e < C::E; ++e) {
    const float ax = fabsf(z[e].x), ay = fabsf(z[e].y);
    if (ax <= FLT_MAX) mx[0] = fmaxf(mx[0], ax); else nf[0] = 1.f;
    if (ay <= FLT_MAX) mx[1] = fmaxf(mx[1], ay); else nf[1] = 1.f;
  }
  float v[4] = {mx[0], mx[1], nf[0], nf[1]};
  block_max<C::T, 4>(v, red, slot);
  bad_a = v[2] != 0.f;
  bad_b = v[3] != 0.f;
  int ea = 0, eb = 0;
  if (!bad_a && v[0] > 0.f) (void)frexpf(v[0], &ea);
  if (!bad_b && v[1] > 0.f) (void)frexpf(v[1], &eb);
  // a row of subnormals only (max below 2^-126) would need a scale above 2^126: clamp, so that the
  // scale stays finite and the scaled row stays finite and nonzero (it is then below 0.5)
  ea = ea < -126 ? -126 : ea;
  eb = eb < -126 ? -126 : eb;
  scale = make_float2(ldexpf(1.f, -ea), ldexpf(1.f, -eb));
  unscale = make_float2(ldexpf(1.f, ea), ldexpf(1.f, eb));
#pragma unroll
  for (int e = 0; e < C::E; ++e) {
    z[e].x = bad_a ? 0.f : z[e].x * scale.x;
    z[e].y = bad_b ? 0.f : z[e].y * scale.y;
  }
}

__device__ __forceinline__ void sort4(float (&q)[4]) {
  auto cx = [](float& a, float& b) {
    const float lo = fminf(a, b), hi = fmaxf(a, b);
    a = lo;
    b = hi;
  };
  cx(q[0], q[1]);
  cx(q[2], q[3]);
  cx(q[0], q[2]);
  cx(q[1], q[3]);
  cx(q[1], q[2]);
}

// q[c] for a 2-bit code c held in a register (selects, no indexed access)
__device__ __forceinline__ float pick4(const float (&q)[4], uint32_t c) {
  const float lo = (c & 1) ? q[1] : q[0];
  const float hi = (c & 1) ? q[3] : q[2];
  return (c & 2) ? hi : lo;
}

__device__ __forceinline__ int code_of(float x, const float (&mids)[3]) {
  return (x > mids[0] ? 1 : 0) + (x > mids[1] ? 1 : 0) + (x > mids[2] ? 1 : 0);
}

__device__ __forceinline__ void closed_form(float a, float b, float (&q)[4]) {
  const float s = a + b, d = fabsf(a - b);
  q[0] = -s;
  q[1] = -d;
  q[2] = d;
  q[3] = s;
}

__device__ __forceinline__ void midpoints(const float (&q)[4], float (&m)[3]) {
  m[0] = (q[0] + q[1]) * 0.5f;
  m[1] = (q[1] + q[2]) * 0.5f;
  m[2] = (q[2] + q[3]) * 0.5f;
}

// Closed-form centres of both rows from the two step sizes of block 0 (Sec. 3.1), then
// `lloyd` plain 1-D k-means passes when LLOYD (an emptied cluster keeps its centre;
// centres re-sorted after each pass).  q[side][4], ascending.
template <class C, bool LLOYD>
__device__ __forceinline__ void cluster_factor(const float2 (&x)[C::E], float2 c1, float2 c2, int lloyd, float* red,
                                               int& slot, float (&q)[2][4]) {
  closed_form(c1.x, c2.x, q[0]);
  closed_form(c1.y, c2.y, q[1]);
  if constexpr (LLOYD) {
    // one row at a time, the four counts packed as bytes of one word (a thread holds fewer than
    // 256 entries of a row): 5 accumulators live instead of 16, so the pass fits the registers
    // the block loop leaves (sums and counts accumulate in the same order either way)
    static_assert(C::E < 256, "per-thread counts packed in bytes");
    for (int it = 0; it < lloyd; ++it) {
#pragma unroll
      for (int sd = 0; sd < 2; ++sd) {
        float mids[3];
        midpoints(q[sd], mids);
        float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
        uint32_t cnt = 0;
        for_each_elem<C>([&](int e, int) {
          const float xv = sd ? x[e].y : x[e].x;
          const int cd = code_of(xv, mids);
          s0 += (cd == 0) ? xv : 0.f;
          s1 += (cd == 1) ? xv : 0.f;
          s2 += (cd == 2) ? xv : 0.f;
          s3 += (cd == 3) ? xv : 0.f;
          cnt += 1u << (8 * cd);
        });
        float acc[8] = {s0, s1, s2, s3, static_cast<float>(cnt & 255u), static_cast<float>((cnt >> 8) & 255u),
                        static_cast<float>((cnt >> 16) & 255u), static_cast<float>(cnt >> 24)};
        block_sum<C::T, 8>(acc, red, slot);
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (acc[4 + c] > 0.f) q[sd][c] = acc[c] / acc[4 + c];
        sort4(q[sd]);
      }
    }
  }
}

// 2-bit codes of both rows (code = number of midpoints strictly below the value), staged
// in LDS in row order and packed four per byte: byte b holds elements 4b..4b+3, element
// 4b+k in bits 2k.  Leaves the LDS free (barrier on exit).
template <class C>
__device__ __forceinline__ void write_codes(const float2 (&x)[C::E], const float (&q)[2][4], float2* lds,
                                            uint8_t* dst, int64_t ra, int64_t rb, bool bad_a, bool bad_b) {
  float mids[2][3];
  midpoints(q[0], mids[0]);
  midpoints(q[1], mids[1]);
  uint8_t* cb = reinterpret_cast<uint8_t*>(lds);
  __syncthreads();  // the last FFT pass read this buffer without a closing barrier
  for_each_elem<C>([&](int e, int i) {
    cb[i] = static_cast<uint8_t>(code_of(x[e].x, mids[0]));
    cb[C::N + i] = static_cast<uint8_t>(code_of(x[e].y, mids[1]));
  });
  __syncthreads();
  constexpr int NBY = (C::N + 3) / 4;
  for (int b = threadIdx.x; b < NBY; b += C::T) {
#pragma unroll
    for (int sd = 0; sd < 2; ++sd) {
      const int64_t row = sd ? rb : ra;
      if (row < 0) continue;
      uint32_t byte = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int i = 4 * b + k;
        if (C::N % 4 == 0 || i < C::N) byte |= static_cast<uint32_t>(cb[sd * C::N + i] & 3) << (2 * k);
      }
      dst[row * NBY + b] = (sd ? bad_b : bad_a) ? 0 : static_cast<uint8_t>(byte);
    }
  }
  __syncthreads();
}

__device__ __forceinline__ void store_centers(float* centers, int f, const float (&q)[2][4], int64_t ra, int64_t rb,
                                              float2 unscale, bool bad_a, bool bad_b) {
  const float qnan = __int_as_float(0x7fc00000);
#pragma unroll
  for (int c = 0; c < 4; ++c) centers[ra * 8 + f * 4 + c] = bad_a ? qnan : q[0][c] * unscale.x;
  if (rb >= 0) {
#pragma unroll
    for (int c = 0; c < 4; ++c) centers[rb * 8 + f * 4 + c] = bad_b ? qnan : q[1][c] * unscale.y;
  }
}

// ------------------------------------------------------------------ greedy kernel
// Alg. 2 for a pair of rows.  Only the residual z and the accumulated vhat live in
// registers across the blocks; after the last block (whose final P is skipped) the
// first factor is recovered exactly as u = w - P(z + vhat), since w = u + P vhat + P z.
// QUANT selects the fused quantizer instance (MODE_QUANTIZE), the other one serves
// MODE_DECOMPOSE and MODE_TRACE; LLOYD (QUANT only) the instance with k-means refinement
// after the closed form; ROT (QUANT only) the instance with the rotation fused into the loads.
// Each instance carries only the code and registers of its own variant.
template <class C, bool LLOYD, bool QUANT, bool ROT>
__global__ __launch_bounds__(C::T) __attribute__((amdgpu_waves_per_eu(C::W))) void pair_greedy_kernel(
    KArgs ka, int64_t item0) {
  __shared__ __align__(16) float2 lds[C::LDS + small_tw_total<C>()];
  __shared__ float red[2 * C::NW * 32];
  int64_t item = item0 + blockIdx.x;
  KArgs a = ka;
  if constexpr (QUANT) {
    if (ka.ngroup > 0) {  // grouped launch: the matrix of this row pair (uniform over the workgroup)
      int gi = 0;
#pragma unroll
      for (int g = 1; g < kMaxGroup; ++g)
        if (g < ka.ngroup && item >= ka.group[g].pair0) gi = g;
      const GroupItem& it = ka.group[gi];
      a.tw = it.tw;
      a.mid4 = it.mid4;
      a.w = it.w;
      a.ldw = it.ldw;
      a.m = it.m;
      a.codes_u = it.codes_u;
      a.codes_v = it.codes_v;
      a.centers = it.centers;
      item -= it.pair0;
    }
  }
  int64_t ra;
  int side = 0;
  if (!QUANT && a.mode == MODE_TRACE) {
    const int64_t row = a.rows[item];
    if (row < 0 || row >= a.m) return;  // uniform: the whole workgroup reads the same entry
    ra = row & ~int64_t(1);
    side = static_cast<int>(row & 1);
  } else {
    ra = 2 * item;
  }
  const int64_t rb = (ra + 1 < a.m) ? ra + 1 : -1;
  int slot = 0;

  constexpr bool RES = resident_ok<C>();
  ResRegs<C, compact_eps<C>()> rr;
  if constexpr (RES) resident_load<C>(rr, lds, a.tw, a.mid4);
  auto applyP = [&](float2(&v)[C::E]) {
    if constexpr (RES) apply_P_res<C>(v, lds, rr);
    else apply_P<C>(v, lds, a.tw, a.mid4);
  };

  float2 z[C::E], vh[C::E];
  constexpr bool VHM = vh_in_memory<C>();
  float4 vhm[VHM ? C::E / 2 : 1];  // vhat between steps (VHM); a run-time index keeps it in memory
  auto vh_store = [&]() {
    if constexpr (VHM) {
      const int b = opaque(0);
#pragma unroll
      for (int h = 0; h < C::E / 2; ++h)
        vhm[b + h] = make_float4(vh[2 * h].x, vh[2 * h].y, vh[2 * h + 1].x, vh[2 * h + 1].y);
    }
  };
  auto vh_load = [&]() {
    if constexpr (VHM) {
      const int b = opaque(0);
#pragma unroll
      for (int h = 0; h < C::E / 2; ++h) {
        const float4 q = vhm[b + h];
        vh[2 * h] = make_float2(q.x, q.y);
        vh[2 * h + 1] = make_float2(q.z, q.w);
      }
    }
  };
  if constexpr (ROT) {
#pragma unroll
    for (int e = 0; e < C::E; ++e) z[e] = make_float2(0.f, 0.f);
    load_pair_staged<C, true>(a.w, a.dtype, a.ldw, ra, rb, a.rot_seed, a.rot_scale, lds,
                              [&](int e, float2 t) { z[e] = t; });
  } else {
    load_pair<C>(z, a.w, a.dtype, a.ldw, ra, rb);
  }
  float2 scale, unscale;
  bool bad_a, bad_b;
  normalise_pair<C>(z, red, slot, scale, unscale, bad_a, bad_b);
#pragma unroll
  for (int e = 0; e < C::E; ++e) vh[e] = make_float2(0.f, 0.f);
  vh_store();

  const int steps = 4 * a.iters;
  int8_t* trace = nullptr;
  float* trc = nullptr;
  if (!QUANT && a.mode == MODE_TRACE) {
    trace = a.tr_signs + (item * steps) * int64_t(C::N);
    trc = a.tr_c + item * steps;
  }
  // block-0 step sizes (equal in every lane): on the shapes whose block loop sits at its register
  // limit they wait for the epilogue in LDS rather than in registers across the loop
  constexpr bool CS_LDS = has_split_pass<C>() || is_small_inner_pass<C>(1) || vh_in_memory<C>();
  __shared__ float2 cs_lds[4];
  float2 cs_reg[4];
  float2* cs = CS_LDS ? cs_lds : cs_reg;
  float2 csum_u = make_float2(0.f, 0.f), csum_v = make_float2(0.f, 0.f);
  auto step = [&](int t, int st, float2 c) {
    if (t == 0 && (!CS_LDS || threadIdx.x == 0)) cs[st] = c;
    if constexpr (!QUANT) {
      if (trc != nullptr && threadIdx.x == 0) trc[4 * t + st] = (side ? c.y : c.x) * (side ? unscale.y : unscale.x);
    }
  };
  for (int t = 0; t < a.iters; ++t) {
    if (t > 0) applyP(z);  // back to the residual rho
    int8_t* tr = trace ? trace + int64_t(4 * t) * C::N : nullptr;
    // two steps on the cube Q_N, accumulating into u (u itself is recovered at the end)
    float2 c = greedy_step<C, false>(z, vh, red, slot, tr, side);
    step(t, 0, c);
    csum_u = cadd(csum_u, c);
    c = greedy_step<C, false>(z, vh, red, slot, tr ? tr + C::N : nullptr, side);
    step(t, 1, c);
    csum_u = cadd(csum_u, c);
    // two steps on P Q_N, in the z = P rho domain, accumulating into vhat
    applyP(z);
    vh_load();
    c = greedy_step<C, true>(z, vh, red, slot, tr ? tr + 2 * C::N : nullptr, side);
    step(t, 2, c);
    csum_v = cadd(csum_v, c);
    c = greedy_step<C, true>(z, vh, red, slot, tr ? tr + 3 * C::N : nullptr, side);
    step(t, 3, c);
    csum_v = cadd(csum_v, c);
    vh_store();
  }

  vh_load();
  if constexpr (CS_LDS) __syncthreads();  // cs (written by thread 0 in the first block) visible to all
  // Epilogue.  vhat is consumed first (written out, or clustered into codes) so that it is
  // not live while u = w - P(z + vhat) is formed: the register peak stays that of the loop.
  const float qnan = __int_as_float(0x7fc00000);
  const bool want_r = !QUANT && (a.mode == MODE_DECOMPOSE) && a.r != nullptr;
  float vmax[2] = {0.f, 0.f};
  if constexpr (QUANT) {
    float qv[2][4];
    cluster_factor<C, LLOYD>(vh, cs[2], cs[3], a.lloyd, red, slot, qv);
    write_codes<C>(vh, qv, lds, a.codes_v, ra, rb, bad_a, bad_b);
    if (threadIdx.x == 0) store_centers(a.centers, 1, qv, ra, rb, unscale, bad_a, bad_b);
  } else {
    int64_t oa = ra, ob = rb;
    bool wa = true, wb = rb >= 0;
    if (a.mode == MODE_TRACE) {
      wa = side == 0;
      wb = side == 1;
      oa = ob = item;
    }
    if (want_r) {  // keep the final z (scaled) in the r buffer until P z is formed below
      for_each_elem<C>([&](int e, int i) {
        a.r[ra * C::N + i] = z[e].x;
        if (rb >= 0) a.r[rb * C::N + i] = z[e].y;
      });
    }
    for_each_elem<C>([&](int e, int i) {
      if (wa) a.vhat[oa * C::N + i] = bad_a ? qnan : vh[e].x * unscale.x;
      if (wb) a.vhat[ob * C::N + i] = bad_b ? qnan : vh[e].y * unscale.y;
    });
#pragma unroll
    for (int e = 0; e < C::E; ++e) {
      vmax[0] = fmaxf(vmax[0], fabsf(vh[e].x));
      vmax[1] = fmaxf(vmax[1], fabsf(vh[e].y));
    }
  }

  // u = w - P(z + vhat) (row reloaded from HBM)
#pragma unroll
  for (int e = 0; e < C::E; ++e) z[e] = cadd(z[e], vh[e]);
  applyP(z);
  if constexpr (ROT) {
    load_pair_staged<C, true>(a.w, a.dtype, a.ldw, ra, rb, a.rot_seed, a.rot_scale, lds, [&](int e, float2 t) {
      z[e].x = bad_a ? 0.f : fmaf(t.x, scale.x, -z[e].x);
      z[e].y = bad_b ? 0.f : fmaf(t.y, scale.y, -z[e].y);
    });
  } else {
    sub_from_rows<C>(z, a.w, a.dtype, a.ldw, ra, rb, scale, bad_a, bad_b);
  }
  float2(&u)[C::E] = z;

  if constexpr (QUANT) {
    float qu[2][4];
    cluster_factor<C, LLOYD>(u, cs[0], cs[1], a.lloyd, red, slot, qu);
    write_codes<C>(u, qu, lds, a.codes_u, ra, rb, bad_a, bad_b);
    if (threadIdx.x == 0) store_centers(a.centers, 0, qu, ra, rb, unscale, bad_a, bad_b);
    return;
  }

  {
    int64_t oa = ra, ob = rb;
    bool wa = true, wb = rb >= 0;
    if (a.mode == MODE_TRACE) {
      wa = side == 0;
      wb = side == 1;
      oa = ob = item;
    }
    for_each_elem<C>([&](int e, int i) {
      if (wa) a.u[oa * C::N + i] = bad_a ? qnan : u[e].x * unscale.x;
      if (wb) a.u[ob * C::N + i] = bad_b ? qnan : u[e].y * unscale.y;
    });
  }
  if (a.mode != MODE_DECOMPOSE) return;
  if (a.bounds != nullptr) {
    float mx[4] = {0.f, vmax[0], 0.f, vmax[1]};
#pragma unroll
    for (int e = 0; e < C::E; ++e) {
      mx[0] = fmaxf(mx[0], fabsf(u[e].x));
      mx[2] = fmaxf(mx[2], fabsf(u[e].y));
    }
    block_max<C::T, 4>(mx, red, slot);
    if (threadIdx.x == 0) {
      float* bo = a.bounds + ra * 4;
      bo[0] = bad_a ? qnan : mx[0] * unscale.x;
      bo[1] = bad_a ? qnan : mx[1] * unscale.x;
      bo[2] = bad_a ? qnan : csum_u.x * unscale.x;
      bo[3] = bad_a ? qnan : csum_v.x * unscale.x;
      if (rb >= 0) {
        bo[4] = bad_b ? qnan : mx[2] * unscale.y;
        bo[5] = bad_b ? qnan : mx[3] * unscale.y;
        bo[6] = bad_b ? qnan : csum_u.y * unscale.y;
        bo[7] = bad_b ? qnan : csum_v.y * unscale.y;
      }
    }
  }
  if (a.cstep != nullptr && threadIdx.x == 0) {
    float* co = a.cstep + ra * 4;
#pragma unroll
    for (int st = 0; st < 4; ++st) co[st] = bad_a ? qnan : cs[st].x * unscale.x;
    if (rb >= 0) {
#pragma unroll
      for (int st = 0; st < 4; ++st) co[4 + st] = bad_b ? qnan : cs[st].y * unscale.y;
    }
  }
  if (want_r) {
    // r = P z_final (the residual of Alg. 2), from the z saved above
    __syncthreads();  // the saved z is read back by other threads of the workgroup
    load_pair_t<C>(z, a.r, C::N, ra, rb);
    applyP(z);
    for_each_elem<C>([&](int e, int i) {
      a.r[ra * C::N + i] = bad_a ? qnan : z[e].x * unscale.x;
      if (rb >= 0) a.r[rb * C::N + i] = bad_b ? qnan : z[e].y * unscale.y;
    });
  }
}

// ------------------------------------------------------------------ P-only kernel
// MODE_APPLY_P: y = P x.  MODE_RECON: w_hat = u_q + P v_q from codes and centres.
// Persistent over pairs: the grid is capped and each workgroup walks items
// blockIdx.x, blockIdx.x + gridDim.x, ... so the operator constants are loaded once per
// workgroup, not once per pair (one application of P is cheap next to them).  The
// reconstruction moves its rows between HBM and the FFT's register layout through the LDS
// buffer, in row order, so codes are read one byte per four elements and w_hat is written in
// contiguous 16-byte vectors; y = P x loads and stores in the register layout directly
// (measured faster for it than staging).
template <class C, bool ROT, bool GROUPED>
__global__ __launch_bounds__(C::T) __attribute__((amdgpu_waves_per_eu(C::W))) void pair_pmap_kernel(
    KArgs ka, int64_t item0, int64_t nitems) {
  __shared__ __align__(16) float2 lds[C::LDS + small_tw_total<C>()];
  __shared__ float red[2 * C::NW * 32];
  constexpr int N = C::N;
  constexpr int NBY = (N + 3) / 4;
  static_assert(N % 4 == 0, "row staging in 16-byte vectors");
  int slot = 0;
  constexpr bool RES = resident_ok<C>();
  ResRegs<C> rr;
  KArgs a = ka;
  int64_t first = blockIdx.x, stride = gridDim.x;
  if constexpr (GROUPED) {  // grouped reconstruction: this workgroup's matrix (uniform)
    int gi = 0;
#pragma unroll
    for (int g = 1; g < kMaxGroup; ++g)
      if (g < ka.ngroup && static_cast<int64_t>(blockIdx.x) >= ka.group[g].wg0) gi = g;
    const GroupItem& gr = ka.group[gi];
    a.tw = gr.tw;
    a.mid4 = gr.mid4;
    a.m = gr.m;
    a.in_codes_v = gr.codes_v;
    a.in_centers = gr.centers;
    a.w = gr.w;  // codes_u
    a.y = gr.y;
    a.ldy = gr.ldy;
    first = blockIdx.x - gr.wg0;
    stride = (gi + 1 < ka.ngroup ? ka.group[gi + 1].wg0 : static_cast<int64_t>(gridDim.x)) - gr.wg0;
    item0 = 0;
    nitems = (gr.m + 1) / 2;
  }
  if constexpr (RES) resident_load<C>(rr, lds, a.tw, a.mid4);
  const float qnan = __int_as_float(0x7fc00000);
  float* lf = reinterpret_cast<float*>(lds);  // staging: row a at [0, N), row b at [N, 2N)
  float4* lf4 = reinterpret_cast<float4*>(lds);
  const bool recon = a.mode == MODE_RECON;
  const bool vout = (reinterpret_cast<uintptr_t>(a.y) % 16 == 0) && (a.ldy % 4 == 0);
  for (int64_t it = first; it < nitems; it += stride) {
    const int64_t ra = 2 * (item0 + it);
    const int64_t rb = (ra + 1 < a.m) ? ra + 1 : -1;
    const int tid = opaque(bfly<C>(threadIdx.x));
    float2 z[C::E];
#pragma unroll
    for (int e = 0; e < C::E; ++e) z[e] = make_float2(0.f, 0.f);
    // 1. y = P x reads its rows straight into the register layout; the reconstruction decodes
    // the v codes in row order into LDS (row b zero when absent)
    if (!recon) {
      load_pair<C>(z, a.w, /*fp32*/ 0, a.ldw, ra, rb, tid);
    } else {
      const float* cea = a.in_centers + ra * 8 + 4;
      const float* ceb = a.in_centers + (rb >= 0 ? rb : ra) * 8 + 4;
      const float qa[4] = {cea[0], cea[1], cea[2], cea[3]};
      const float qb[4] = {ceb[0], ceb[1], ceb[2], ceb[3]};
      const uint8_t* cva = a.in_codes_v + ra * NBY;
      const uint8_t* cvb = a.in_codes_v + (rb >= 0 ? rb : ra) * NBY;
      for (int q = tid; q < NBY; q += C::T) {
        const uint32_t ba = cva[q], bb = cvb[q];
        float4 va, vb;
        va.x = pick4(qa, ba & 3);
        va.y = pick4(qa, (ba >> 2) & 3);
        va.z = pick4(qa, (ba >> 4) & 3);
        va.w = pick4(qa, (ba >> 6) & 3);
        vb.x = pick4(qb, bb & 3);
        vb.y = pick4(qb, (bb >> 2) & 3);
        vb.z = pick4(qb, (bb >> 4) & 3);
        vb.w = pick4(qb, (bb >> 6) & 3);
        lf4[q] = va;
        lf4[N / 4 + q] = rb >= 0 ? vb : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
    if (recon) {
      __syncthreads();
      for_each_elem<C>([&](int e, int i) { z[e] = make_float2(lf[i], lf[N + i]); }, tid);
      __syncthreads();  // the staged v_q rows are read before the first pass overwrites the buffer
    }
    float2 scale, unscale;
    bool bad_a, bad_b;
    normalise_pair<C>(z, red, slot, scale, unscale, bad_a, bad_b);
    if constexpr (RES) apply_P_res<C>(z, lds, rr);
    else apply_P<C>(z, lds, a.tw, a.mid4);
    if (!recon) {
      for_each_elem<C>([&](int e, int i) {
        a.y[ra * a.ldy + i] = bad_a ? qnan : z[e].x * unscale.x;
        if (rb >= 0) a.y[rb * a.ldy + i] = bad_b ? qnan : z[e].y * unscale.y;
      }, tid);
      __syncthreads();  // the last pass read the buffer the next item's first pass writes
      continue;
    }
    if constexpr (ROT) {
      // w_hat = R^T (P v_q + u_q): both rows in row order as float2, u_q added, then the
      // Hadamard factor, C_b^T, the scale and the signs, as the standalone inverse rotation
      constexpr int B = rot_odd_part(N);
      __syncthreads();  // the last pass read the buffer
      for_each_elem<C>([&](int e, int i) {
        lds[i] = make_float2(bad_a ? qnan : z[e].x * unscale.x, bad_b ? qnan : z[e].y * unscale.y);
      }, tid);
      __syncthreads();
      const uint8_t* cua = static_cast<const uint8_t*>(a.w) + ra * NBY;
      const uint8_t* cub = static_cast<const uint8_t*>(a.w) + (rb >= 0 ? rb : ra) * NBY;
      const float* cea = a.in_centers + ra * 8;
      const float* ceb = a.in_centers + (rb >= 0 ? rb : ra) * 8;
      const float ua[4] = {cea[0], cea[1], cea[2], cea[3]};
      const float ub[4] = {ceb[0], ceb[1], ceb[2], ceb[3]};
      for (int q = tid; q < NBY; q += C::T) {
        const uint32_t ba = cua[q], bb = cub[q];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          float2 v = lds[4 * q + k];
          v.x += pick4(ua, (ba >> (2 * k)) & 3);
          v.y += pick4(ub, (bb >> (2 * k)) & 3);
          lds[4 * q + k] = v;
        }
      }
      __syncthreads();
      rot_hadamard<B, C::T>(lds, N, tid);
      rot_odd_factor_fixed<B, true, C::T, N>(lds, tid);
      float* ya = a.y + ra * a.ldy;
      float* yb = a.y + (rb >= 0 ? rb : ra) * a.ldy;
      for (int i = tid; i < N; i += C::T) {
        const float s = rot_sign(a.rot_seed, i);
        const float2 v = lds[i];
        ya[i] = v.x * a.rot_scale * s;
        if (rb >= 0) yb[i] = v.y * a.rot_scale * s;
      }
      __syncthreads();  // read before the next item's first pass writes the buffer
      continue;
    }
    __syncthreads();  // the last pass read the buffer the outputs are staged in
    for_each_elem<C>([&](int e, int i) {
      lf[i] = bad_a ? qnan : z[e].x * unscale.x;
      lf[N + i] = bad_b ? qnan : z[e].y * unscale.y;
    }, tid);
    __syncthreads();
    // 2. reconstruction: w_hat = P v_q + u_q in row order, 16-byte stores
    const uint8_t* cua = static_cast<const uint8_t*>(a.w) + ra * NBY;
    const uint8_t* cub = static_cast<const uint8_t*>(a.w) + (rb >= 0 ? rb : ra) * NBY;
    const float* cea = a.in_centers + ra * 8;
    const float* ceb = a.in_centers + (rb >= 0 ? rb : ra) * 8;
    const float ua[4] = {cea[0], cea[1], cea[2], cea[3]};
    const float ub[4] = {ceb[0], ceb[1], ceb[2], ceb[3]};
    float* ya = a.y + ra * a.ldy;
    float* yb = a.y + (rb >= 0 ? rb : ra) * a.ldy;
    for (int q = tid; q < N / 4; q += C::T) {
      float4 oa = lf4[q], ob = lf4[N / 4 + q];
      const uint32_t ba = cua[q], bb = cub[q];
      oa.x += pick4(ua, ba & 3);
      oa.y += pick4(ua, (ba >> 2) & 3);
      oa.z += pick4(ua, (ba >> 4) & 3);
      oa.w += pick4(ua, (ba >> 6) & 3);
      ob.x += pick4(ub, bb & 3);
      ob.y += pick4(ub, (bb >> 2) & 3);
      ob.z += pick4(ub, (bb >> 4) & 3);
      ob.w += pick4(ub, (bb >> 6) & 3);
      if (vout) {
        reinterpret_cast<float4*>(ya)[q] = oa;
        if (rb >= 0) reinterpret_cast<float4*>(yb)[q] = ob;
      } else {
        ya[4 * q] = oa.x;
        ya[4 * q + 1] = oa.y;
        ya[4 * q + 2] = oa.z;
        ya[4 * q + 3] = oa.w;
        if (rb >= 0) {
          yb[4 * q] = ob.x;
          yb[4 * q + 1] = ob.y;
          yb[4 * q + 2] = ob.z;
          yb[4 * q + 3] = ob.w;
        }
      }
    }
    __syncthreads();  // staged outputs read before the next item stages its inputs
  }
}

// One output of both rows of a pair (the thread's elements given by f(e) as float2: row a in .x,
// row b in .y) written in row order through the LDS buffer: contiguous 16-byte stores (4-byte
// ones where a row is not 16-byte aligned) instead of the even/odd order's stride-2 stores, which
// leave every line half written per instruction.  out_b may be null (no row b to write).  Starts
// and ends with a barrier, so the buffer is free before and after.
template <class C, class F>
__device__ __forceinline__ void store_pair_staged(float2* lds, float* out_a, float* out_b, F&& f) {
  static_assert(C::N % 4 == 0, "rows staged as float4");
  float* lf = reinterpret_cast<float*>(lds);
  const float4* lf4 = reinterpret_cast<const float4*>(lds);
  __syncthreads();  // earlier readers of the buffer are done
  for_each_elem<C>([&](int e, int i) {
    const float2 v = f(e);
    lf[i] = v.x;
    lf[C::N + i] = v.y;
  });
  __syncthreads();
  const bool vec_a = (reinterpret_cast<uintptr_t>(out_a) & 15) == 0;
  const bool vec_b = (reinterpret_cast<uintptr_t>(out_b) & 15) == 0;
  for (int q = threadIdx.x; q < C::N / 4; q += C::T) {
    if (out_a != nullptr) {
      const float4 o = lf4[q];
      if (vec_a) {
        reinterpret_cast<float4*>(out_a)[q] = o;
      } else {
        out_a[4 * q] = o.x;
        out_a[4 * q + 1] = o.y;
        out_a[4 * q + 2] = o.z;
        out_a[4 * q + 3] = o.w;
      }
    }
    if (out_b != nullptr) {
      const float4 o = lf4[C::N / 4 + q];
      if (vec_b) {
        reinterpret_cast<float4*>(out_b)[q] = o;
      } else {
        out_b[4 * q] = o.x;
        out_b[4 * q + 1] = o.y;
        out_b[4 * q + 2] = o.z;
        out_b[4 * q + 3] = o.w;
      }
    }
  }
  __syncthreads();  // the staged rows are read before the buffer's next writer
}

// ------------------------------------------------------------------ schedule variants
// The greedy over Q_N u P Q_N with another step schedule (MODE_SCHEDULE; a.schedule).  Both
// domains of the residual are kept per row of the pair, rho and z = P rho; a step works in one
// domain per row (the two rows of a pair may choose differently), and one application of P to
// the pair's stepped values refreshes the other domain of both rows (P^2 = I).  That is one P
// per atomic step, twice what the alternating kernel needs; three arrays live across steps (the
// residual in two domains and vhat).  The register budget is relaxed to two waves per SIMD where
// the workgroup allows it.
// With a.rows set, workgroup i decomposes the pair holding row a.rows[i] and records that
// row's signs, step sizes, choices and ||rho||^2 after every step.
//
// Where the workgroup shape caps the registers (more than 512 threads: one workgroup per CU,
// 168 or 128 VGPRs) the four arrays do not fit; vhat then lives in private memory between its
// steps (16-byte loads and stores of the whole array at each vhat-step), so that rho, z and the
// transform's array stay in registers.
template <class C>
constexpr bool sched_vh_in_memory() {
  return (C::T > 512 || C::E >= 32) && C::E % 2 == 0;
}
// With a 128-register budget (1024 threads), and on the five-pass shape with 64 values per array
// (N = 13824), the stepped values wait in private memory too while P runs, so that only the
// transformed array occupies registers across the transform (the compiler otherwise spills
// inside the loop there).
template <class C>
constexpr bool sched_park() {
  return sched_vh_in_memory<C>() && ((C::T > 512 && C::W >= 4) || (C::E >= 32 && C::NP >= 5));
}
// Where LDS has room beside the transform's buffer (N = 10000, 11008: one element per butterfly
// thread, B0 = 1), vhat lives there instead, as many of each thread's 2E values as fit (row a's
// first, then row b's; each thread its own slots, read and written only at vhat-steps), the rest
// in registers: private memory would be written back to HBM at every vhat-step.
template <class C>
constexpr int sched_vh_lds_values() {
  if constexpr (!sched_vh_in_memory<C>() || sched_park<C>() || C::B0 != 1) {
    return 0;
  } else {
    constexpr int used = (C::LDS + small_tw_total<C>()) * 8 + 2 * C::NW * 32 * 4;
    constexpr int fit = (160 * 1024 - used) / (4 * C::NB0);
    return fit < C::E ? 0 : (fit < 2 * C::E ? fit : 2 * C::E);
  }
}
template <class C, bool TRACE>
__global__ __launch_bounds__(C::T) __attribute__((amdgpu_waves_per_eu(C::T <= 512 ? 2 : C::W))) void
pair_schedule_kernel(KArgs a, int64_t item0) {
  __shared__ __align__(16) float2 lds[C::LDS + small_tw_total<C>()];
  __shared__ float red[2 * C::NW * 32];
  const int64_t item = item0 + blockIdx.x;
  constexpr bool tracing = TRACE;  // an instance of its own: the trace code costs registers
  int64_t ra;
  int side = 0;
  if constexpr (tracing) {
    const int64_t row = a.rows[item];
    if (row < 0 || row >= a.m) return;  // uniform
    ra = row & ~int64_t(1);
    side = static_cast<int>(row & 1);
  } else {
    ra = 2 * item;
  }
  const int64_t rb = (ra + 1 < a.m) ? ra + 1 : -1;
  int slot = 0;
  constexpr bool RES = resident_ok<C>();
  ResRegs<C, compact_eps<C>()> rr;
  if constexpr (RES) resident_load<C>(rr, lds, a.tw, a.mid4);
  auto applyP = [&](float2(&v)[C::E]) {
    if constexpr (RES) apply_P_res<C>(v, lds, rr);
    else apply_P<C>(v, lds, a.tw, a.mid4);
  };
  constexpr int VL = sched_vh_lds_values<C>();  // vhat values per thread in LDS
  constexpr bool VHL = VL > 0;
  constexpr bool VHM = sched_vh_in_memory<C>() && !VHL;
  // The residual of each row in both domains: sv holds it in one domain and y = P sv in the other;
  // za / zb say which (true: sv holds z = P rho for that row).  A step takes each row's chosen
  // domain from sv or y, writes the stepped values to sv and transforms them into y, so no select
  // ever lands on the arrays carried from step to step.
  float2 sv[C::E], y[C::E], vh[VHM || VHL ? 1 : C::E];
  float4 vhm[VHM ? C::E / 2 : 1];  // vhat (VHM); a run-time index keeps it in memory
  // VHL: slot s < VL of thread t at vhl[s * NB0 + t], s = e for row a, E + e for row b; row b's
  // elements e >= VL - E in vhr
  __shared__ float vhl[VHL ? VL * C::NB0 : 1];
  float vhr[VHL && VL < 2 * C::E ? 2 * C::E - VL : 1];
  const int vt = threadIdx.x;
  const bool vown = vt < C::NB0;  // threads past the last butterfly hold no elements
  auto vh_slot = [&](int sl) -> float& { return vhl[sl * C::NB0 + vt]; };
  constexpr bool PARK = sched_park<C>();
  float4 park[PARK ? C::E / 2 : 1];  // the stepped values across P (PARK)
  load_pair<C>(sv, a.w, a.dtype, a.ldw, ra, rb);
  float2 scale, unscale;
  bool bad_a, bad_b;
  normalise_pair<C>(sv, red, slot, scale, unscale, bad_a, bad_b);
#pragma unroll
  for (int e = 0; e < C::E; ++e) y[e] = sv[e];
  if constexpr (VHM) {
    const int b = opaque(0);
#pragma unroll
    for (int h = 0; h < C::E / 2; ++h) vhm[b + h] = make_float4(0.f, 0.f, 0.f, 0.f);
  } else if constexpr (VHL) {
    if (vown) {
#pragma unroll
      for (int sl = 0; sl < VL; ++sl) vh_slot(sl) = 0.f;
    }
#pragma unroll
    for (int k = 0; k < 2 * C::E - VL; ++k) vhr[k] = 0.f;
  } else {
#pragma unroll
    for (int e = 0; e < C::E; ++e) vh[e] = make_float2(0.f, 0.f);
  }
  applyP(y);
  bool za = false, zb = false;
  const int steps = 4 * a.iters;
  const int sched = a.schedule;
  const float tola = a.tol * scale.x, tolb = a.tol * scale.y;
  const float unsel = side ? unscale.y : unscale.x;
  for (int st = 0; st < steps; ++st) {
    // l1 norms, nonzero counts and squared norms of sv and y, both rows
    float s12[12];
#pragma unroll
    for (int k = 0; k < 12; ++k) s12[k] = 0.f;
#pragma unroll
    for (int e = 0; e < C::E; ++e) {
      s12[0] += fabsf(sv[e].x);
      s12[1] += fabsf(sv[e].y);
      s12[2] += fabsf(y[e].x);
      s12[3] += fabsf(y[e].y);
      s12[4] += sv[e].x != 0.f ? 1.f : 0.f;
      s12[5] += sv[e].y != 0.f ? 1.f : 0.f;
      s12[6] += y[e].x != 0.f ? 1.f : 0.f;
      s12[7] += y[e].y != 0.f ? 1.f : 0.f;
      s12[8] += sv[e].x * sv[e].x;
      s12[9] += sv[e].y * sv[e].y;
      s12[10] += y[e].x * y[e].x;
      s12[11] += y[e].y * y[e].y;
    }
    if constexpr (C::NW * 12 > 64) block_sum_lanes<C::T, 12>(s12, red, slot);
    else block_sum<C::T, 12>(s12, red, slot);
    // threads past the last butterfly hold zeros: they add nothing to the counts above
    // v: l1 of rho and z, nonzero counts of rho and z, ||rho||^2 (rows a, b in turn)
    const float v[10] = {za ? s12[2] : s12[0],  zb ? s12[3] : s12[1], za ? s12[0] : s12[2], zb ? s12[1] : s12[3],
                         za ? s12[6] : s12[4],  zb ? s12[7] : s12[5], za ? s12[4] : s12[6], zb ? s12[5] : s12[7],
                         za ? s12[10] : s12[8], zb ? s12[11] : s12[9]};
    const int pos = st & 3;
    bool va, vb;  // true: the vhat-half (step on z)
    if (sched == SCHED_ALTERNATING) {
      va = vb = pos >= 2;
    } else if (sched == SCHED_REVERSE) {
      va = vb = pos < 2;
    } else {
      va = !(v[0] > v[2]);
      vb = !(v[1] > v[3]);
    }
    const bool act_a = !(sched == SCHED_ORIGINAL && a.tol > 0.f && sqrtf(v[8]) < tola);
    const bool act_b = !(sched == SCHED_ORIGINAL && a.tol > 0.f && sqrtf(v[9]) < tolb);
    const float l1a = va ? v[2] : v[0], l1b = vb ? v[3] : v[1];
    const float nza = va ? v[6] : v[4], nzb = vb ? v[7] : v[5];
    float ca = sched == SCHED_ORIGINAL ? (nza > 0.f ? l1a / nza : 0.f) : div_n<C::N>(l1a);
    float cb = sched == SCHED_ORIGINAL ? (nzb > 0.f ? l1b / nzb : 0.f) : div_n<C::N>(l1b);
    ca = act_a ? ca : 0.f;
    cb = act_b ? cb : 0.f;
    // each row's chosen domain: in sv when it is the domain sv holds, else in y
    const bool fa = va == za, fb = vb == zb;
    if constexpr (tracing) {
      const bool vs = side ? vb : va;
      const bool fs = side ? fb : fa;
      const int tid = opaque(bfly<C>(threadIdx.x));
      int8_t* trs = a.tr_signs + (item * steps + st) * int64_t(C::N);
#pragma unroll
      for (int i = 0; i < C::B0; ++i) {
        const int j = tid + C::T * i;
        if (j < C::NB0) {
#pragma unroll
          for (int r = 0; r < C::R0; ++r) {
            const float2 xv = fs ? sv[i * C::R0 + r] : y[i * C::R0 + r];
            trs[orig_index<C::N>(j + r * C::NB0)] = sgn8(side ? xv.y : xv.x);
          }
        }
      }
      if (threadIdx.x == 0) {
        a.tr_c[item * steps + st] = (side ? cb : ca) * unsel;
        a.tr_choice[item * steps + st] = (side ? act_b : act_a) ? (vs ? 1 : 0) : -1;
      }
    }
    // vhat += the steps of the rows that step on z (VHM, VHL: the same values, through memory)
    if constexpr (VHL) {
      if (va && vown) {
#pragma unroll
        for (int e = 0; e < C::E; ++e) vh_slot(e) += sgn_times(fa ? sv[e].x : y[e].x, ca);
      }
      if (vb) {
#pragma unroll
        for (int e = 0; e < C::E; ++e) {
          const float d = sgn_times(fb ? sv[e].y : y[e].y, cb);
          if (C::E + e < VL) {
            if (vown) vh_slot(C::E + e) += d;
          } else {
            vhr[e - (VL - C::E)] += d;
          }
        }
      }
    }
    if constexpr (VHM) {
      if (va || vb) {
        const int b = opaque(0);
#pragma unroll
        for (int h = 0; h < C::E / 2; ++h) {
          float4 q = vhm[b + h];
          if (va) {
            q.x += sgn_times(fa ? sv[2 * h].x : y[2 * h].x, ca);
            q.z += sgn_times(fa ? sv[2 * h + 1].x : y[2 * h + 1].x, ca);
          }
          if (vb) {
            q.y += sgn_times(fb ? sv[2 * h].y : y[2 * h].y, cb);
            q.w += sgn_times(fb ? sv[2 * h + 1].y : y[2 * h + 1].y, cb);
          }
          vhm[b + h] = q;
        }
      }
    }
    // the step, in each row's chosen domain; sv collects the stepped values of both rows
#pragma unroll
    for (int e = 0; e < C::E; ++e) {
      float xa = fa ? sv[e].x : y[e].x;
      float xb = fb ? sv[e].y : y[e].y;
      const float da = sgn_times(xa, ca), db = sgn_times(xb, cb);
      xa -= da;
      xb -= db;
      if constexpr (!VHM && !VHL) {
        if (va) vh[e].x += da;
        if (vb) vh[e].y += db;
      }
      sv[e] = make_float2(xa, xb);
      y[e] = sv[e];
    }
    if constexpr (PARK) {
      const int b = opaque(0);
#pragma unroll
      for (int h = 0; h < C::E / 2; ++h)
        park[b + h] = make_float4(sv[2 * h].x, sv[2 * h].y, sv[2 * h + 1].x, sv[2 * h + 1].y);
    }
    applyP(y);  // the other domain of each row
    if constexpr (PARK) {
      const int b = opaque(0);
#pragma unroll
      for (int h = 0; h < C::E / 2; ++h) {
        const float4 q = park[b + h];
        sv[2 * h] = make_float2(q.x, q.y);
        sv[2 * h + 1] = make_float2(q.z, q.w);
      }
    }
    za = va;
    zb = vb;
    if constexpr (tracing) {
      float q[1] = {0.f};
      const bool zs = side ? zb : za;  // rho of the traced row: y if sv holds its z
#pragma unroll
      for (int e = 0; e < C::E; ++e) {
        const float2 rv = zs ? y[e] : sv[e];
        q[0] += side ? rv.y * rv.y : rv.x * rv.x;
      }
      block_sum<C::T, 1>(q, red, slot);
      if (threadIdx.x == 0) a.tr_r2[item * steps + st] = q[0] * unsel * unsel;
    }
  }
  // u = w - r - P vhat (row reloaded from HBM), in steps that keep two arrays live: rho of each
  // row into sv and out to r; then sv = w - rho; then y = P vhat and u = sv - y
  const float qnan = __int_as_float(0x7fc00000);
#pragma unroll
  for (int e = 0; e < C::E; ++e) sv[e] = make_float2(za ? y[e].x : sv[e].x, zb ? y[e].y : sv[e].y);
  int64_t oa = ra, ob = rb;
  bool wa = true, wb = rb >= 0;
  if constexpr (tracing) {
    wa = side == 0;
    wb = side == 1;
    oa = ob = item;
  }
  auto out_rows = [&](float* base, float*& pa, float*& pb) {
    pa = wa ? base + oa * C::N : nullptr;
    pb = wb ? base + ob * C::N : nullptr;
  };
  float *pa, *pb;
  if (a.r != nullptr) {
    out_rows(a.r, pa, pb);
    store_pair_staged<C>(lds, pa, pb, [&](int e) {
      return make_float2(bad_a ? qnan : sv[e].x * unscale.x, bad_b ? qnan : sv[e].y * unscale.y);
    });
  }
  {
    float2 t[C::E];
    load_pair<C>(t, a.w, a.dtype, a.ldw, ra, rb);
#pragma unroll
    for (int e = 0; e < C::E; ++e)
      sv[e] = make_float2(fmaf(t[e].x, scale.x, -sv[e].x), fmaf(t[e].y, scale.y, -sv[e].y));
  }
  auto vhat_at = [&](int e) -> float2 {
    if constexpr (VHM) {
      const float4 q = vhm[opaque(0) + e / 2];
      return (e & 1) ? make_float2(q.z, q.w) : make_float2(q.x, q.y);
    } else if constexpr (VHL) {
      const float b = C::E + e < VL ? (vown ? vh_slot(C::E + e) : 0.f) : vhr[e - (VL - C::E)];
      return make_float2(vown ? vh_slot(e) : 0.f, b);
    } else {
      return vh[e];
    }
  };
#pragma unroll
  for (int e = 0; e < C::E; ++e) y[e] = vhat_at(e);
  applyP(y);
  out_rows(a.u, pa, pb);
  store_pair_staged<C>(lds, pa, pb, [&](int e) {
    return make_float2(bad_a ? qnan : (sv[e].x - y[e].x) * unscale.x, bad_b ? qnan : (sv[e].y - y[e].y) * unscale.y);
  });
  out_rows(a.vhat, pa, pb);
  store_pair_staged<C>(lds, pa, pb, [&](int e) {
    const float2 vhe = vhat_at(e);
    return make_float2(bad_a ? qnan : vhe.x * unscale.x, bad_b ? qnan : vhe.y * unscale.y);
  });
}

// ------------------------------------------------------------------ dispatch
// Whether the incoherence rotation of length N can be fused into the pair kernels: the odd
// factor C_b has compile-time constants for b = 1, 3 and 43 only (the lengths the rotation kernel
// takes); the host layer rejects the rotated entry points for other lengths before any launch.
constexpr bool rot_fusable(int n) {
  const int b = n / (n & -n);
  return n <= 16384 && (b == 1 || b == 3 || b == 43);
}

template <class C>
hipError_t launch_cfg(const KArgs& a, int64_t grid, hipStream_t s) {
  constexpr int64_t kMaxGrid = int64_t(1) << 30;
  if constexpr (!rot_fusable(C::N)) {
    if (a.rot) return hipErrorInvalidValue;
  }
  for (int64_t i0 = 0; i0 < grid; i0 += kMaxGrid) {
    const int64_t g = (grid - i0 < kMaxGrid) ? grid - i0 : kMaxGrid;
    const dim3 gd(static_cast<unsigned>(g)), bd(C::T);
    if (a.mode == MODE_QUANTIZE) {
      if (a.rot) {
        if constexpr (rot_fusable(C::N)) {
          if (a.lloyd > 0) hipLaunchKernelGGL((pair_greedy_kernel<C, true, true, true>), gd, bd, 0, s, a, i0);
          else hipLaunchKernelGGL((pair_greedy_kernel<C, false, true, true>), gd, bd, 0, s, a, i0);
        }
      } else if (a.lloyd > 0) {
        hipLaunchKernelGGL((pair_greedy_kernel<C, true, true, false>), gd, bd, 0, s, a, i0);
      } else {
        hipLaunchKernelGGL((pair_greedy_kernel<C, false, true, false>), gd, bd, 0, s, a, i0);
      }
    } else if (a.mode <= MODE_TRACE) {
      hipLaunchKernelGGL((pair_greedy_kernel<C, false, false, false>), gd, bd, 0, s, a, i0);
    } else if (a.mode == MODE_SCHEDULE) {
      if (a.rows != nullptr)
        hipLaunchKernelGGL((pair_schedule_kernel<C, true>), dim3(static_cast<unsigned>(g)), dim3(C::T), 0, s, a, i0);
      else
        hipLaunchKernelGGL((pair_schedule_kernel<C, false>), dim3(static_cast<unsigned>(g)), dim3(C::T), 0, s, a, i0);
    } else {
      // grouped reconstruction: `grid` is the launch's workgroup count (the matrices' shares)
      const int64_t pg = a.ngroup > 0 ? g : (g < kPmapGrid ? g : kPmapGrid);
      if (a.rot) {
        if constexpr (rot_fusable(C::N))
          hipLaunchKernelGGL((pair_pmap_kernel<C, true, false>), dim3(static_cast<unsigned>(pg)), bd, 0, s, a, i0, g);
      } else if (a.ngroup > 0) hipLaunchKernelGGL((pair_pmap_kernel<C, false, true>), dim3(static_cast<unsigned>(pg)), bd, 0, s, a, i0, g);
      else hipLaunchKernelGGL((pair_pmap_kernel<C, false, false>), dim3(static_cast<unsigned>(pg)), bd, 0, s, a, i0, g);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

// Defines the external launcher launch_n<N> for one launch configuration.
#define KASHIN_DEFINE_SIZE(N, T, W, ...)                                                     \
  hipError_t launch_n##N(const KArgs& a, int64_t grid, hipStream_t stream) {                \
    return launch_cfg<Cfg<N, T, W, __VA_ARGS__>>(a, grid, stream);                          \
  }

}  // namespace kashin
