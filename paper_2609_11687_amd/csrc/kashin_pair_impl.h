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

#include "kashin_internal.h"
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

struct Pow2Tab {  // cos / sin (2 pi m / 16)
  static constexpr float c[16] = {1.0f, 0.923879533f, 0.707106781f, 0.382683432f, 0.0f, -0.382683432f,
                                  -0.707106781f, -0.923879533f, -1.0f, -0.923879533f, -0.707106781f,
                                  -0.382683432f, 0.0f, 0.382683432f, 0.707106781f, 0.923879533f};
  static constexpr float s[16] = {0.0f, 0.382683432f, 0.707106781f, 0.923879533f, 1.0f, 0.923879533f,
                                  0.707106781f, 0.382683432f, 0.0f, -0.382683432f, -0.707106781f,
                                  -0.923879533f, -1.0f, -0.923879533f, -0.707106781f, -0.382683432f};
};

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }

// d * w16^K (forward, w16 = exp(-2 pi i / 16)) or d * w16^-K (inverse), K a compile-time constant.
template <int K, bool INV>
__device__ __forceinline__ float2 tw16(float2 d) {
  constexpr int k = K & 15;
  if constexpr (k == 0) {
    return d;
  } else if constexpr (k == 8) {
    return make_float2(-d.x, -d.y);
  } else if constexpr (k == 4) {
    if constexpr (INV) return make_float2(-d.y, d.x);
    else return make_float2(d.y, -d.x);
  } else if constexpr (k == 12) {
    if constexpr (INV) return make_float2(d.y, -d.x);
    else return make_float2(-d.y, d.x);
  } else {
    constexpr float c = Pow2Tab::c[k];
    constexpr float s = INV ? -Pow2Tab::s[k] : Pow2Tab::s[k];
    return make_float2(fmaf(d.x, c, d.y * s), fmaf(d.y, c, -(d.x * s)));
  }
}

// In-register DFT of a power-of-two length R <= 16 (radix-2 decimation in frequency,
// output reordered to natural order at compile time).
template <int R, bool INV>
__device__ __forceinline__ void dft_pow2(float2 (&a)[R]) {
  constexpr int L = ilog2(R);
  sfor<0, L>([&](auto lv) {
    constexpr int len = R >> decltype(lv)::value;
    constexpr int half = len >> 1;
    sfor<0, R / len>([&](auto sv) {
      sfor<0, half>([&](auto jv) {
        constexpr int i0 = decltype(sv)::value * len + decltype(jv)::value;
        constexpr int i1 = i0 + half;
        const float2 x = a[i0], y = a[i1];
        a[i0] = cadd(x, y);
        a[i1] = tw16<decltype(jv)::value * (16 / len), INV>(csub(x, y));
      });
    });
  });
  float2 t[R];
  sfor<0, R>([&](auto iv) { t[decltype(iv)::value] = a[bitrev(decltype(iv)::value, L)]; });
  sfor<0, R>([&](auto iv) { a[decltype(iv)::value] = t[decltype(iv)::value]; });
}

// In-register DFT of an odd length R, directly from its definition, pairing j with R-j
// so each constant multiplies a sum or a difference.
// Outputs are handed to sink(q, A_q) as soon as they are formed, so they never occupy
// registers next to the inputs.
template <int R, bool INV, class Sink>
__device__ __forceinline__ void dft_odd(const float2 (&a)[R], Sink&& sink) {
  constexpr int H = (R - 1) / 2;
  float2 s[H], d[H];
  sfor<1, H + 1>([&](auto jv) {
    constexpr int j = decltype(jv)::value;
    s[j - 1] = cadd(a[j], a[R - j]);
    d[j - 1] = csub(a[j], a[R - j]);
  });
  const float2 x0 = a[0];
  float2 sum = x0;
  sfor<0, H>([&](auto jv) { sum = cadd(sum, s[decltype(jv)::value]); });
  sink(0, sum);
  sfor<1, H + 1>([&](auto qv) {
    constexpr int q = decltype(qv)::value;
    float2 re = x0;
    float2 im = make_float2(0.f, 0.f);
    sfor<1, H + 1>([&](auto jv) {
      constexpr int j = decltype(jv)::value;
      constexpr int m = (j * q) % R;
      constexpr float c = OddTab<R>::c[m];
      constexpr float sn = OddTab<R>::s[m];
      re.x = fmaf(s[j - 1].x, c, re.x);
      re.y = fmaf(s[j - 1].y, c, re.y);
      im.x = fmaf(d[j - 1].x, sn, im.x);
      im.y = fmaf(d[j - 1].y, sn, im.y);
    });
    // forward: A_q = re - i im, A_{R-q} = re + i im; inverse swaps them
    const float2 minus = make_float2(re.x + im.y, re.y - im.x);
    const float2 plus = make_float2(re.x - im.y, re.y + im.x);
    sink(q, INV ? plus : minus);
    sink(R - q, INV ? minus : plus);
  });
}

// DFT of a[] handed to sink(q, A_q) for every q (power-of-two R: computed in place first).
template <int R, bool INV, class Sink>
__device__ __forceinline__ void dft(float2 (&a)[R], Sink&& sink) {
  if constexpr ((R & (R - 1)) == 0) {
    if constexpr (R > 1) dft_pow2<R, INV>(a);
    sfor<0, R>([&](auto qv) { sink(decltype(qv)::value, a[decltype(qv)::value]); });
  } else {
    static_assert(R % 2 == 1, "composite non-power-of-two radices are not implemented");
    dft_odd<R, INV>(a, sink);
  }
}

// ------------------------------------------------------------------ launch configuration
// N: vector length = complex FFT length of a packed pair.  T: threads per workgroup.
// Rs: radices of the forward FFT passes; the first radix also fixes the register layout
// in which the greedy steps run: thread t holds elements j + r * (N / R0) for its
// butterflies j = t + T * i, r < R0.
template <int N_, int T_, int... Rs>
struct Cfg {
  static constexpr int N = N_;
  static constexpr int T = T_;
  static constexpr int NP = sizeof...(Rs);
  static constexpr int rad[NP] = {Rs...};
  static constexpr int R0 = rad[0];
  static constexpr int NB0 = N / R0;
  static constexpr int B0 = (NB0 + T - 1) / T;
  static constexpr int E = B0 * R0;
  static constexpr int NW = (T + 63) / 64;
  static constexpr int LDS = N + (N >> 4) + 4;
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

__device__ __forceinline__ int pad(int i) { return i + (i >> 4); }  // one spare slot per 16

// Opaque copies: values (thread index, table pointers) that would otherwise be proven
// invariant across the block loop and hoisted out of it, keeping every twiddle and
// address of every pass live in registers at once.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}
template <class P>
__device__ __forceinline__ P* opaque_ptr(P* p) {
  asm volatile("" : "+s"(p));
  return p;
}

// Position m of the even/odd order -> index in the row.
template <int N>
__device__ __forceinline__ int orig_index(int m) {
  return m < N / 2 ? 2 * m : 2 * (N - 1 - m) + 1;
}

// ------------------------------------------------------------------ reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum of K values over the workgroup, in a fixed order (every thread gets the same bits).
// `red` holds 2 * NW * KMAX floats; consecutive calls alternate halves so that one
// barrier per call suffices.
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
      for (int w = 1; w < NW; ++w) s += r[w * K + k];
      v[k] = s;
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
      for (int w = 1; w < NW; ++w) s = fmaxf(s, r[w * K + k]);
      v[k] = s;
    }
  }
}

// ------------------------------------------------------------------ FFT passes
enum { SRC_REGS = 0, SRC_LDS = 1, SRC_MID = 2 };
enum { DST_LDS = 0, DST_REGS = 1 };

// One Stockham pass of radix R with stride NS: butterfly j reads elements j + r * N/R,
// multiplies by the twiddles w_N^(r * (j mod NS) * N/(NS R)), takes a length-R DFT, and
// writes element q to (j / NS) * NS * R + (j mod NS) + q * NS.  In-place in LDS: every
// read completes (barrier) before any write.  SRC_MID applies the eps gather-and-scale
// on the way in (first inverse pass).
template <class C, int R, int NS, bool INV, int SRC, int DST>
__device__ __forceinline__ void fft_pass(float2 (&z)[C::E], float2* __restrict__ lds,
                                         const float2* __restrict__ tw, const float2* __restrict__ mid) {
  constexpr int N = C::N;
  constexpr int T = C::T;
  constexpr int NB = N / R;
  constexpr int BP = (NB + T - 1) / T;
  static_assert(SRC != SRC_REGS || (R == C::R0 && NS == 1), "register source must be the first pass");
  static_assert(DST != DST_REGS || (R == C::R0 && NS == N / C::R0), "register target must be the last pass");
  const int tid = opaque(static_cast<int>(threadIdx.x));
  tw = opaque_ptr(tw);
  mid = opaque_ptr(mid);
  float2 a[BP][R];
  sfor<0, BP>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const int j = tid + T * i;
    if constexpr (SRC == SRC_REGS) {
      sfor<0, R>([&](auto rv) { a[i][decltype(rv)::value] = z[i * R + decltype(rv)::value]; });
    } else {
      if (NB % T == 0 || j < NB) {
        sfor<0, R>([&](auto rv) {
          constexpr int r = decltype(rv)::value;
          const int k = j + r * NB;
          if constexpr (SRC == SRC_MID) {
            const float2 f = mid[k];
            const int src = (f.y != 0.f) ? (N - k) : k;
            const float2 v = lds[pad(src)];
            a[i][r] = make_float2(f.x * v.x - f.y * v.y, f.x * v.y + f.y * v.x);
          } else {
            a[i][r] = lds[pad(k)];
          }
        });
      }
    }
  });
  if constexpr (SRC != SRC_REGS) __syncthreads();
  sfor<0, BP>([&](auto iv) {
    constexpr int i = decltype(iv)::value;
    const int j = tid + T * i;
    if (NB % T == 0 || j < NB) {
      const int jm = (NS > 1) ? (j % NS) : 0;
      if constexpr (NS > 1) {
        sfor<1, R>([&](auto rv) {
          constexpr int r = decltype(rv)::value;
          const float2 w = tw[r * jm * (N / (NS * R))];
          const float2 v = a[i][r];
          if constexpr (!INV) a[i][r] = make_float2(v.x * w.x - v.y * w.y, v.x * w.y + v.y * w.x);
          else a[i][r] = make_float2(v.x * w.x + v.y * w.y, v.y * w.x - v.x * w.y);
        });
      }
      if constexpr (DST == DST_LDS) {
        const int base = (j / NS) * NS * R + jm;
        dft<R, INV>(a[i], [&](int q, float2 v) { lds[pad(base + q * NS)] = v; });
      } else {
        dft<R, INV>(a[i], [&](int q, float2 v) { z[i * R + q] = v; });
      }
    }
  });
  if constexpr (DST == DST_LDS) __syncthreads();
}

template <class C, int P>
__device__ __forceinline__ void fwd_passes(float2 (&z)[C::E], float2* lds, const float2* tw, const float2* mid) {
  if constexpr (P < C::NP) {
    fft_pass<C, C::rad[P], ns_fwd<C>(P), false, (P == 0 ? SRC_REGS : SRC_LDS), DST_LDS>(z, lds, tw, mid);
    fwd_passes<C, P + 1>(z, lds, tw, mid);
  }
}
template <class C, int P>
__device__ __forceinline__ void inv_passes(float2 (&z)[C::E], float2* lds, const float2* tw, const float2* mid) {
  if constexpr (P < C::NP) {
    fft_pass<C, C::rad[C::NP - 1 - P], ns_inv<C>(P), true, (P == 0 ? SRC_MID : SRC_LDS),
             (P == C::NP - 1 ? DST_REGS : DST_LDS)>(z, lds, tw, mid);
    inv_passes<C, P + 1>(z, lds, tw, mid);
  }
}

// z <- P z for both rows of the pair (Alg. 2: P z = IDCT(eps * DCT(z))).
template <class C>
__device__ __forceinline__ void apply_P(float2 (&z)[C::E], float2* lds, const float2* tw, const float2* mid) {
  fwd_passes<C, 0>(z, lds, tw, mid);
  inv_passes<C, 0>(z, lds, tw, mid);
}

// ------------------------------------------------------------------ greedy step
__device__ __forceinline__ float sgn_times(float x, float c) { return x > 0.f ? c : (x < 0.f ? -c : 0.f); }
__device__ __forceinline__ int8_t sgn8(float x) { return x > 0.f ? 1 : (x < 0.f ? -1 : 0); }

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
  const float ca = s[0] / static_cast<float>(C::N);
  const float cb = s[1] / static_cast<float>(C::N);
  if (trace != nullptr) {
    const int tid = opaque(static_cast<int>(threadIdx.x));
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
__device__ __forceinline__ float ld_elem(const void* p, int64_t idx, int dtype) {
  if (dtype == 1) return __half2float(static_cast<const __half*>(p)[idx]);
  return static_cast<const float*>(p)[idx];
}

// Load rows a (and b if >= 0) into the greedy register layout, in even/odd order.
template <class C>
__device__ __forceinline__ void load_pair(float2 (&z)[C::E], const void* w, int dtype, int64_t ldw, int64_t ra,
                                          int64_t rb) {
#pragma unroll
  for (int i = 0; i < C::B0; ++i) {
    const int j = threadIdx.x + C::T * i;
#pragma unroll
    for (int r = 0; r < C::R0; ++r) {
      float2 v = make_float2(0.f, 0.f);
      if (j < C::NB0) {
        const int src = orig_index<C::N>(j + r * C::NB0);
        v.x = ld_elem(w, ra * ldw + src, dtype);
        if (rb >= 0) v.y = ld_elem(w, rb * ldw + src, dtype);
      }
      z[i * C::R0 + r] = v;
    }
  }
}

// z <- w * scale - z for the pair (rows reloaded in the register layout); zero for a bad row.
template <class C>
__device__ __forceinline__ void sub_from_rows(float2 (&z)[C::E], const void* w, int dtype, int64_t ldw, int64_t ra,
                                              int64_t rb, float2 scale, bool bad_a, bool bad_b) {
#pragma unroll
  for (int i = 0; i < C::B0; ++i) {
    const int j = threadIdx.x + C::T * i;
    if (j < C::NB0) {
#pragma unroll
      for (int r = 0; r < C::R0; ++r) {
        const int src = orig_index<C::N>(j + r * C::NB0);
        float2& v = z[i * C::R0 + r];
        v.x = bad_a ? 0.f : fmaf(ld_elem(w, ra * ldw + src, dtype), scale.x, -v.x);
        v.y = (bad_b || rb < 0) ? 0.f : fmaf(ld_elem(w, rb * ldw + src, dtype), scale.y, -v.y);
      }
    }
  }
}

template <class C, class F>
__device__ __forceinline__ void for_each_elem(F&& f) {
#pragma unroll
  for (int i = 0; i < C::B0; ++i) {
    const int j = threadIdx.x + C::T * i;
    if (j < C::NB0) {
#pragma unroll
      for (int r = 0; r < C::R0; ++r) f(i * C::R0 + r, orig_index<C::N>(j + r * C::NB0));
    }
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

// ------------------------------------------------------------------ greedy kernel
// Alg. 2 for a pair of rows.  Only the residual z and the accumulated vhat live in
// registers across the blocks; after the last block (whose final P is skipped) the
// first factor is recovered exactly as u = w - P(z + vhat), since w = u + P vhat + P z.
// LLOYD selects the instance with k-means refinement after the closed form; the
// closed-form-only instance (a.lloyd == 0) carries none of its registers.
template <class C, bool LLOYD>
__global__ __launch_bounds__(C::T) void pair_greedy_kernel(KArgs a, int64_t item0) {
  __shared__ float2 lds[C::LDS];
  __shared__ float red[2 * C::NW * 32];
  const int64_t item = item0 + blockIdx.x;
  int64_t ra;
  int side = 0;
  if (a.mode == MODE_TRACE) {
    const int64_t row = a.rows[item];
    if (row < 0 || row >= a.m) return;  // uniform: the whole workgroup reads the same entry
    ra = row & ~int64_t(1);
    side = static_cast<int>(row & 1);
  } else {
    ra = 2 * item;
  }
  const int64_t rb = (ra + 1 < a.m) ? ra + 1 : -1;
  int slot = 0;

  float2 z[C::E], vh[C::E];
  load_pair<C>(z, a.w, a.dtype, a.ldw, ra, rb);
  float2 scale, unscale;
  bool bad_a, bad_b;
  normalise_pair<C>(z, red, slot, scale, unscale, bad_a, bad_b);
#pragma unroll
  for (int e = 0; e < C::E; ++e) vh[e] = make_float2(0.f, 0.f);

  const int steps = 4 * a.iters;
  int8_t* trace = nullptr;
  float* trc = nullptr;
  if (a.mode == MODE_TRACE) {
    trace = a.tr_signs + (item * steps) * int64_t(C::N);
    trc = a.tr_c + item * steps;
  }
  float2 cs[4];
  float2 csum_u = make_float2(0.f, 0.f), csum_v = make_float2(0.f, 0.f);
  for (int t = 0; t < a.iters; ++t) {
    if (t > 0) apply_P<C>(z, lds, a.tw, a.mid);  // back to the residual rho
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      if (st == 2) apply_P<C>(z, lds, a.tw, a.mid);  // z = P rho
      int8_t* tr = trace ? trace + int64_t(4 * t + st) * C::N : nullptr;
      const float2 c = (st < 2) ? greedy_step<C, false>(z, vh, red, slot, tr, side)
                                : greedy_step<C, true>(z, vh, red, slot, tr, side);
      if (t == 0) cs[st] = c;
      if (st < 2) csum_u = cadd(csum_u, c);
      else csum_v = cadd(csum_v, c);
      if (trc != nullptr && threadIdx.x == 0) trc[4 * t + st] = (side ? c.y : c.x) * (side ? unscale.y : unscale.x);
    }
  }

  // u = w - P(z + vhat): z <- P(z + vhat), then u = w_scaled - z (row reloaded from HBM).
  const bool want_r = (a.mode == MODE_DECOMPOSE) && a.r != nullptr;
#pragma unroll
  for (int e = 0; e < C::E; ++e) z[e] = cadd(z[e], vh[e]);
  apply_P<C>(z, lds, a.tw, a.mid);
  sub_from_rows<C>(z, a.w, a.dtype, a.ldw, ra, rb, scale, bad_a, bad_b);
  // now z holds u (scaled)
  float2 (&u)[C::E] = z;

  const float qnan = __int_as_float(0x7fc00000);
  if (a.mode == MODE_DECOMPOSE || a.mode == MODE_TRACE) {
    bool wa = true, wb = rb >= 0;
    int64_t oa = ra, ob = rb;
    if (a.mode == MODE_TRACE) {
      wa = side == 0;
      wb = side == 1;
      oa = ob = item;
    }
    for_each_elem<C>([&](int e, int i) {
      if (wa) {
        a.u[oa * C::N + i] = bad_a ? qnan : u[e].x * unscale.x;
        a.vhat[oa * C::N + i] = bad_a ? qnan : vh[e].x * unscale.x;
      }
      if (wb) {
        a.u[ob * C::N + i] = bad_b ? qnan : u[e].y * unscale.y;
        a.vhat[ob * C::N + i] = bad_b ? qnan : vh[e].y * unscale.y;
      }
    });
    if (a.mode == MODE_DECOMPOSE && a.bounds != nullptr) {
      float mx[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int e = 0; e < C::E; ++e) {
        mx[0] = fmaxf(mx[0], fabsf(u[e].x));
        mx[1] = fmaxf(mx[1], fabsf(vh[e].x));
        mx[2] = fmaxf(mx[2], fabsf(u[e].y));
        mx[3] = fmaxf(mx[3], fabsf(vh[e].y));
      }
      block_max<C::T, 4>(mx, red, slot);
      if (threadIdx.x == 0) {
        float* b = a.bounds + ra * 4;
        b[0] = bad_a ? qnan : mx[0] * unscale.x;
        b[1] = bad_a ? qnan : mx[1] * unscale.x;
        b[2] = bad_a ? qnan : csum_u.x * unscale.x;
        b[3] = bad_a ? qnan : csum_v.x * unscale.x;
        if (rb >= 0) {
          b[4] = bad_b ? qnan : mx[2] * unscale.y;
          b[5] = bad_b ? qnan : mx[3] * unscale.y;
          b[6] = bad_b ? qnan : csum_u.y * unscale.y;
          b[7] = bad_b ? qnan : csum_v.y * unscale.y;
        }
      }
    }
    if (a.mode == MODE_DECOMPOSE && a.cstep != nullptr && threadIdx.x == 0) {
      float* c = a.cstep + ra * 4;
#pragma unroll
      for (int st = 0; st < 4; ++st) c[st] = bad_a ? qnan : cs[st].x * unscale.x;
      if (rb >= 0) {
#pragma unroll
        for (int st = 0; st < 4; ++st) c[4 + st] = bad_b ? qnan : cs[st].y * unscale.y;
      }
    }
    if (want_r) {
      // r = P z_final = w - u - P vhat: z <- P vhat (vhat moved in first), then r = w - u - z.
#pragma unroll
      for (int e = 0; e < C::E; ++e) {
        const float2 t = vh[e];
        vh[e] = u[e];  // keep u
        u[e] = t;
      }
      apply_P<C>(z, lds, a.tw, a.mid);  // z = P vhat
      sub_from_rows<C>(z, a.w, a.dtype, a.ldw, ra, rb, scale, bad_a, bad_b);  // z = w - P vhat
      for_each_elem<C>([&](int e, int i) {
        a.r[ra * C::N + i] = bad_a ? qnan : (z[e].x - vh[e].x) * unscale.x;
        if (rb >= 0) a.r[rb * C::N + i] = bad_b ? qnan : (z[e].y - vh[e].y) * unscale.y;
      });
    }
    return;
  }

  // MODE_QUANTIZE: four-peak clustering of u and vhat for both rows (Sec. 3.1), in the
  // scaled domain (a power-of-two scale changes no comparison and no mean).
  // q[f][s]: factor f (0 = u, 1 = vhat), side s (0 = row a, 1 = row b).
  float q[2][2][4];
  closed_form(cs[0].x, cs[1].x, q[0][0]);
  closed_form(cs[0].y, cs[1].y, q[0][1]);
  closed_form(cs[2].x, cs[3].x, q[1][0]);
  closed_form(cs[2].y, cs[3].y, q[1][1]);
  for (int it = 0; LLOYD && it < a.lloyd; ++it) {
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      float2(&x)[C::E] = f ? vh : u;
      float mids[2][3];
      midpoints(q[f][0], mids[0]);
      midpoints(q[f][1], mids[1]);
      float acc[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) acc[k] = 0.f;
      for_each_elem<C>([&](int e, int) {
        const float xs[2] = {x[e].x, x[e].y};
#pragma unroll
        for (int sd = 0; sd < 2; ++sd) {
          const int cd = code_of(xs[sd], mids[sd]);
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            acc[sd * 8 + c] += (cd == c) ? xs[sd] : 0.f;
            acc[sd * 8 + 4 + c] += (cd == c) ? 1.f : 0.f;
          }
        }
      });
      block_sum<C::T, 16>(acc, red, slot);
#pragma unroll
      for (int sd = 0; sd < 2; ++sd) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (acc[sd * 8 + 4 + c] > 0.f) q[f][sd][c] = acc[sd * 8 + c] / acc[sd * 8 + 4 + c];
        sort4(q[f][sd]);
      }
    }
  }
  float mids[2][2][3];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int s = 0; s < 2; ++s) midpoints(q[f][s], mids[f][s]);
  // codes in row order into LDS (four byte planes: [f][s][N]), then pack four per byte.
  uint8_t* cb = reinterpret_cast<uint8_t*>(lds);
  for_each_elem<C>([&](int e, int i) {
    cb[0 * C::N + i] = static_cast<uint8_t>(code_of(u[e].x, mids[0][0]));
    cb[1 * C::N + i] = static_cast<uint8_t>(code_of(u[e].y, mids[0][1]));
    cb[2 * C::N + i] = static_cast<uint8_t>(code_of(vh[e].x, mids[1][0]));
    cb[3 * C::N + i] = static_cast<uint8_t>(code_of(vh[e].y, mids[1][1]));
  });
  __syncthreads();
  constexpr int NBY = (C::N + 3) / 4;
  for (int b = threadIdx.x; b < NBY; b += C::T) {
#pragma unroll
    for (int plane = 0; plane < 4; ++plane) {
      const int s = plane & 1;
      const int64_t row = s ? rb : ra;
      if (row < 0) continue;
      const bool bad = s ? bad_b : bad_a;
      uint8_t byte = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int i = 4 * b + k;
        if (i < C::N) byte |= static_cast<uint8_t>((cb[plane * C::N + i] & 3) << (2 * k));
      }
      uint8_t* dst = (plane < 2) ? a.codes_u : a.codes_v;
      dst[row * NBY + b] = bad ? 0 : byte;
    }
  }
  if (threadIdx.x == 0) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int64_t row = s ? rb : ra;
      if (row < 0) continue;
      const bool bad = s ? bad_b : bad_a;
      const float us = s ? unscale.y : unscale.x;
      float* ce = a.centers + row * 8;
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int c = 0; c < 4; ++c) ce[f * 4 + c] = bad ? qnan : q[f][s][c] * us;
    }
  }
}

// ------------------------------------------------------------------ P-only kernel
// MODE_APPLY_P: y = P x.  MODE_RECON: w_hat = u_q + P v_q from codes and centres.
template <class C>
__global__ __launch_bounds__(C::T) void pair_pmap_kernel(KArgs a, int64_t item0) {
  __shared__ float2 lds[C::LDS];
  __shared__ float red[2 * C::NW * 32];
  const int64_t item = item0 + blockIdx.x;
  const int64_t ra = 2 * item;
  const int64_t rb = (ra + 1 < a.m) ? ra + 1 : -1;
  int slot = 0;
  constexpr int NBY = (C::N + 3) / 4;
  float2 z[C::E];
  if (a.mode == MODE_APPLY_P) {
    load_pair<C>(z, a.w, /*fp32*/ 0, a.ldw, ra, rb);
  } else {
    const uint8_t* cv = a.in_codes_v;
    const float* ce = a.in_centers;
#pragma unroll
    for (int e = 0; e < C::E; ++e) z[e] = make_float2(0.f, 0.f);
    for_each_elem<C>([&](int e, int i) {
      const int sh = 2 * (i & 3);
      const int ca = (cv[ra * NBY + (i >> 2)] >> sh) & 3;
      z[e].x = ce[ra * 8 + 4 + ca];
      if (rb >= 0) {
        const int cb2 = (cv[rb * NBY + (i >> 2)] >> sh) & 3;
        z[e].y = ce[rb * 8 + 4 + cb2];
      }
    });
  }
  float2 scale, unscale;
  bool bad_a, bad_b;
  normalise_pair<C>(z, red, slot, scale, unscale, bad_a, bad_b);
  apply_P<C>(z, lds, a.tw, a.mid);
  const float qnan = __int_as_float(0x7fc00000);
  const uint8_t* cu = static_cast<const uint8_t*>(a.w);
  for_each_elem<C>([&](int e, int i) {
    float va = bad_a ? qnan : z[e].x * unscale.x;
    float vb = bad_b ? qnan : z[e].y * unscale.y;
    if (a.mode == MODE_RECON) {
      const int sh = 2 * (i & 3);
      va += a.in_centers[ra * 8 + ((cu[ra * NBY + (i >> 2)] >> sh) & 3)];
      if (rb >= 0) vb += a.in_centers[rb * 8 + ((cu[rb * NBY + (i >> 2)] >> sh) & 3)];
    }
    a.y[ra * a.ldy + i] = va;
    if (rb >= 0) a.y[rb * a.ldy + i] = vb;
  });
}

// ------------------------------------------------------------------ dispatch
template <class C>
hipError_t launch_cfg(const KArgs& a, int64_t grid, hipStream_t s) {
  constexpr int64_t kMaxGrid = int64_t(1) << 30;
  for (int64_t i0 = 0; i0 < grid; i0 += kMaxGrid) {
    const int64_t g = (grid - i0 < kMaxGrid) ? grid - i0 : kMaxGrid;
    if (a.mode == MODE_QUANTIZE && a.lloyd > 0) {
      hipLaunchKernelGGL((pair_greedy_kernel<C, true>), dim3(static_cast<unsigned>(g)), dim3(C::T), 0, s, a, i0);
    } else if (a.mode <= MODE_TRACE) {
      hipLaunchKernelGGL((pair_greedy_kernel<C, false>), dim3(static_cast<unsigned>(g)), dim3(C::T), 0, s, a, i0);
    } else {
      hipLaunchKernelGGL(pair_pmap_kernel<C>, dim3(static_cast<unsigned>(g)), dim3(C::T), 0, s, a, i0);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

// Defines the external launcher launch_n<N> for one launch configuration.
#define KASHIN_DEFINE_SIZE(N, T, ...)                                                        \
  hipError_t launch_n##N(const KArgs& a, int64_t grid, hipStream_t stream) {                \
    return launch_cfg<Cfg<N, T, __VA_ARGS__>>(a, grid, stream);                             \
  }

}  // namespace kashin
