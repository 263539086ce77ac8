// Dispatch by vector length, and the standalone clustering kernel.
#include "kashin_pair_impl.h"

namespace kashin {

// Supported vector lengths: N, threads per workgroup, occupancy target (waves per SIMD),
// forward radices.
#define KASHIN_SIZES(X)          \
  X(64, 64, 2, 8, 8)                \
  X(96, 64, 2, 16, 3, 2)            \
  X(172, 64, 2, 4, 43)              \
  X(256, 64, 2, 16, 16)             \
  X(512, 64, 4, 8, 8, 8)            \
  X(768, 64, 3, 16, 3, 16)          \
  X(1024, 64, 2, 16, 4, 16)         \
  X(2048, 128, 2, 16, 8, 16)        \
  X(3072, 256, 3, 16, 12, 16)      \
  X(4096, 256, 3, 16, 16, 16)       \
  X(5120, 320, 3, 16, 16, 4, 5)     \
  X(6144, 384, 3, 16, 16, 8, 3)     \
  X(8192, 512, 2, 16, 16, 16, 2)    \
  X(10000, 640, 3, 16, 5, 5, 5, 5)  \
  X(11008, 768, 3, 16, 43, 16)      \
  X(13824, 448, 2, 16, 16, 2, 3, 9) \
  X(14336, 448, 2, 16, 16, 8, 7)    \
  X(16384, 1024, 4, 16, 8, 8, 16)

#define X(N, ...) hipError_t launch_n##N(const KArgs& a, int64_t grid, hipStream_t stream);
KASHIN_SIZES(X)
#undef X

namespace {
// ------------------------------------------------------------------ standalone clustering
// One workgroup per row; thread t handles groups of four consecutive elements.
constexpr int CT = 256;

__global__ __launch_bounds__(CT) void cluster_kernel(ClusterArgs a, int64_t row0) {
  __shared__ float red[2 * (CT / 64) * 32];
  const int64_t row = row0 + blockIdx.x;
  const int n = a.n;
  const int nby = (n + 3) / 4;
  int slot = 0;
  const float* uu = a.u + row * n;
  const float* vv = a.vhat + row * n;
  const float* cs = a.cstep + row * 4;
  float q[2][4];
  closed_form(cs[0], cs[1], q[0]);
  closed_form(cs[2], cs[3], q[1]);
  const float qnan = __int_as_float(0x7fc00000);
  const bool bad = !(fabsf(cs[0]) <= FLT_MAX && fabsf(cs[1]) <= FLT_MAX && fabsf(cs[2]) <= FLT_MAX &&
                     fabsf(cs[3]) <= FLT_MAX);
  for (int it = 0; it < a.lloyd; ++it) {
    float mids[2][3];
    midpoints(q[0], mids[0]);
    midpoints(q[1], mids[1]);
    float acc[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k] = 0.f;
    for (int i = threadIdx.x; i < n; i += CT) {
      const float xs[2] = {uu[i], vv[i]};
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        const int cd = code_of(xs[f], mids[f]);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          acc[f * 8 + c] += (cd == c) ? xs[f] : 0.f;
          acc[f * 8 + 4 + c] += (cd == c) ? 1.f : 0.f;
        }
      }
    }
    block_sum<CT, 16>(acc, red, slot);
#pragma unroll
    for (int f = 0; f < 2; ++f) {
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (acc[f * 8 + 4 + c] > 0.f) q[f][c] = acc[f * 8 + c] / acc[f * 8 + 4 + c];
      sort4(q[f]);
    }
  }
  float mids[2][3];
  midpoints(q[0], mids[0]);
  midpoints(q[1], mids[1]);
  for (int b = threadIdx.x; b < nby; b += CT) {
    uint8_t bu = 0, bv = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = 4 * b + k;
      if (i < n) {
        bu |= static_cast<uint8_t>(code_of(uu[i], mids[0]) << (2 * k));
        bv |= static_cast<uint8_t>(code_of(vv[i], mids[1]) << (2 * k));
      }
    }
    a.codes_u[row * nby + b] = bad ? 0 : bu;
    a.codes_v[row * nby + b] = bad ? 0 : bv;
  }
  if (threadIdx.x == 0) {
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int c = 0; c < 4; ++c) a.centers[row * 8 + f * 4 + c] = bad ? qnan : q[f][c];
  }
}

}  // namespace

bool plan_shape(int n, PlanShape* out) {
  switch (n) {
#define X(N, T, W, ...)                               \
  case N: {                                           \
    const int r[] = {__VA_ARGS__};                    \
    out->n = N;                                       \
    out->threads = T;                                 \
    out->np = static_cast<int>(sizeof(r) / sizeof(int)); \
    for (int i = 0; i < out->np; ++i) out->rad[i] = r[i]; \
    return true;                                      \
  }
    KASHIN_SIZES(X)
#undef X
    default:
      return false;
  }
}

bool supported_n(int n) {
  switch (n) {
#define X(N, ...) \
  case N:         \
    return true;
    KASHIN_SIZES(X)
#undef X
    default:
      return false;
  }
}

hipError_t launch_pair(int n, const KArgs& a, int64_t grid, hipStream_t stream) {
  switch (n) {
#define X(N, ...) \
  case N:         \
    return launch_n##N(a, grid, stream);
    KASHIN_SIZES(X)
#undef X
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_cluster(const ClusterArgs& a, hipStream_t stream) {
  constexpr int64_t kMaxGrid = int64_t(1) << 30;
  for (int64_t r0 = 0; r0 < a.m; r0 += kMaxGrid) {
    const int64_t g = (a.m - r0 < kMaxGrid) ? a.m - r0 : kMaxGrid;
    hipLaunchKernelGGL(cluster_kernel, dim3(static_cast<unsigned>(g)), dim3(CT), 0, stream, a, r0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace kashin
