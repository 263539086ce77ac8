// Error-compensated quantisation of a weight matrix (Sec. 5, Fig. 1; eq. optq_update): the
// factor of the damped inverse Hessian and the per-chunk (or per-column) error carry, around the
// quantiser and reconstruction kernels of the pair kernel.
//
// Layout: W^T is held as w_t, d_in rows of n = d_out (the plan's length), so each column of W is
// a row for the quantiser.  U (upper, U^T U = (H + lambda I)^-1) and V = U^-1 are d_in x d_in
// float64, row-major.
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include <cstdint>
#include <mutex>

#include "kashin_internal.h"

namespace kashin {
namespace {

// lambda = damp * mean(diag H), one workgroup
constexpr int kDiagT = 256;
__global__ __launch_bounds__(kDiagT) void diag_mean_kernel(const float* h, int d, int64_t ldh, double damp,
                                                           double* lambda) {
  __shared__ double part[kDiagT];
  double s = 0.0;
  for (int i = threadIdx.x; i < d; i += kDiagT) s += static_cast<double>(h[i * ldh + i]);
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = kDiagT / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *lambda = damp * part[0] / d;
}

// F = J (H + lambda I) J in float64, column-major (J reverses the index order):
// F[i + j d] = H[d-1-i][d-1-j] + lambda [i == j]
__global__ void damp_flip_kernel(const float* h, int d, int64_t ldh, const double* lambda, double* f) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(d) * d) return;
  const int i = static_cast<int>(idx % d), j = static_cast<int>(idx / d);
  double v = static_cast<double>(h[static_cast<int64_t>(d - 1 - i) * ldh + (d - 1 - j)]);
  if (i == j) v += *lambda;
  f[idx] = v;
}

// out (row-major, d x d) = J A J restricted to the upper triangle, A column-major lower:
// out[r][c] = A[(d-1-r) + (d-1-c) d] for c >= r, else 0
__global__ void flip_upper_kernel(const double* a, int d, double* out) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(d) * d) return;
  const int r = static_cast<int>(idx / d), c = static_cast<int>(idx % d);
  out[idx] = c >= r ? a[static_cast<int64_t>(d - 1 - r) + static_cast<int64_t>(d - 1 - c) * d] : 0.0;
}

// e[k][x] = (w[row0 + k][x] - q[row0 + k][x]) * s_k, s_k = 1 / U[row0+k][row0+k] when u != null
__global__ void error_kernel(const float* w, int64_t ldw, const float* q, int n, int64_t row0, int rows,
                             const double* u, int64_t ldu, float* e) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(rows) * n) return;
  const int k = static_cast<int>(idx / n), x = static_cast<int>(idx % n);
  float v = w[(row0 + k) * ldw + x] - q[(row0 + k) * n + x];
  if (u != nullptr) v = static_cast<float>(static_cast<double>(v) / u[(row0 + k) * ldu + (row0 + k)]);
  e[idx] = v;
}

// w[j][x] -= U[i][j] err[x] for j in [j0, j1): the error of column i carried to the later columns
// of its chunk
__global__ void rank1_kernel(float* w, int64_t ldw, int n, int64_t i, int64_t j0, int64_t j1, const double* u,
                             int64_t ldu, const float* err) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= (j1 - j0) * n) return;
  const int64_t j = j0 + idx / n;
  const int x = static_cast<int>(idx % n);
  w[j * ldw + x] -= static_cast<float>(u[i * ldu + j]) * err[x];
}

// m[k][r] = sum_l V[c0 + k][c0 + l] U[c0 + l][c1 + r] (k, l < rows = c1 - c0; r < rest), float64
// accumulation, float32 result: the chunk's U_cc^-1 U_cr.  Workgroup: 64 columns r, 16 rows k;
// the V rows of its k range sit in LDS.
constexpr int kMT = 256, kMR = 64, kMK = 16, kMaxChunk = 128;
__global__ __launch_bounds__(kMT) void chunk_factor_kernel(const double* v, const double* u, int64_t ld, int64_t c0,
                                                           int rows, int64_t c1, int64_t rest, float* m) {
  __shared__ double vs[kMK][kMaxChunk];
  const int k0 = blockIdx.y * kMK;
  for (int t = threadIdx.x; t < kMK * rows; t += kMT) {
    const int kk = t / rows, l = t % rows;
    vs[kk][l] = (k0 + kk < rows) ? v[(c0 + k0 + kk) * ld + (c0 + l)] : 0.0;
  }
  __syncthreads();
  const int64_t r = static_cast<int64_t>(blockIdx.x) * kMR + (threadIdx.x % kMR);
  const int kq = (threadIdx.x / kMR) * (kMK / (kMT / kMR));  // 4 rows per thread
  double acc[kMK / (kMT / kMR)] = {};
  if (r < rest) {
    for (int l = 0; l < rows; ++l) {
      const double ul = u[(c0 + l) * ld + (c1 + r)];
#pragma unroll
      for (int a = 0; a < kMK / (kMT / kMR); ++a) acc[a] += vs[kq + a][l] * ul;
    }
#pragma unroll
    for (int a = 0; a < kMK / (kMT / kMR); ++a)
      if (k0 + kq + a < rows) m[static_cast<int64_t>(k0 + kq + a) * rest + r] = static_cast<float>(acc[a]);
  }
}

// m[k][r] = U[c0 + k][c1 + r] as float32 (the exact form's U_cr)
__global__ void copy_block_kernel(const double* u, int64_t ld, int64_t c0, int rows, int64_t c1, int64_t rest,
                                  float* m) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= rows * rest) return;
  const int64_t k = idx / rest, r = idx % rest;
  m[idx] = static_cast<float>(u[(c0 + k) * ld + (c1 + r)]);
}

// C[r][x] -= sum_k A[k][r] B[k][x]: C rest x n (ld ldc), A rows x rest (ld rest), B rows x n (ld n),
// float32.  64 x 64 tiles of C per workgroup of 256 threads (4 x 4 each), K in steps of 16 through
// LDS; the k-rows of A and B are contiguous, so both tiles load coalesced.
constexpr int kGT = 256, kGB = 64, kGK = 16;
__global__ __launch_bounds__(kGT) void update_gemm_kernel(float* c, int64_t ldc, const float* a, const float* b,
                                                          int rows, int64_t rest, int n) {
  __shared__ float as[kGK][kGB + 4];
  __shared__ float bs[kGK][kGB + 4];
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * kGB;
  const int x0 = blockIdx.x * kGB;
  const int tr = (threadIdx.x / 16) * 4, tx = (threadIdx.x % 16) * 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < rows; k0 += kGK) {
    for (int t = threadIdx.x; t < kGK * kGB; t += kGT) {
      const int kk = t / kGB, j = t % kGB;
      const bool kin = k0 + kk < rows;
      as[kk][j] = (kin && r0 + j < rest) ? a[static_cast<int64_t>(k0 + kk) * rest + r0 + j] : 0.f;
      bs[kk][j] = (kin && x0 + j < n) ? b[static_cast<int64_t>(k0 + kk) * n + x0 + j] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kGK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        av[i] = as[kk][tr + i];
        bv[i] = bs[kk][tx + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t r = r0 + tr + i;
    if (r >= rest) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (x0 + tx + j < n) c[r * ldc + x0 + tx + j] -= acc[i][j];
  }
}

unsigned blocks_for(int64_t count, int threads) { return static_cast<unsigned>((count + threads - 1) / threads); }

}  // namespace

hipError_t optq_factor_device(const float* h, int d, int64_t ldh, double damp, double* u, double* v,
                              hipStream_t stream, int* info_out) {
  *info_out = 0;
  double* f = nullptr;
  double* lambda = nullptr;
  rocblas_int* info = nullptr;
  rocblas_handle handle = nullptr;
  const size_t nn = static_cast<size_t>(d) * d;
  hipError_t e = hipMalloc(&f, nn * sizeof(double));
  if (e == hipSuccess) e = hipMalloc(&lambda, sizeof(double) + sizeof(rocblas_int) * 2);
  if (e == hipSuccess) {
    info = reinterpret_cast<rocblas_int*>(lambda + 1);
    hipLaunchKernelGGL(diag_mean_kernel, dim3(1), dim3(kDiagT), 0, stream, h, d, ldh, damp, lambda);
    hipLaunchKernelGGL(damp_flip_kernel, dim3(blocks_for(nn, 256)), dim3(256), 0, stream, h, d, ldh, lambda, f);
    e = hipGetLastError();
  }
  if (e == hipSuccess && rocblas_create_handle(&handle) != rocblas_status_success) e = hipErrorUnknown;
  if (e == hipSuccess && rocblas_set_stream(handle, stream) != rocblas_status_success) e = hipErrorUnknown;
  // J Hd J = L L^T (L lower); Hd = V V^T with V = J L J upper; U = V^-1 = J L^-1 J
  if (e == hipSuccess && rocsolver_dpotrf(handle, rocblas_fill_lower, d, f, d, info) != rocblas_status_success)
    e = hipErrorUnknown;
  if (e == hipSuccess && v != nullptr) {
    hipLaunchKernelGGL(flip_upper_kernel, dim3(blocks_for(nn, 256)), dim3(256), 0, stream, f, d, v);
    e = hipGetLastError();
  }
  if (e == hipSuccess &&
      rocsolver_dtrtri(handle, rocblas_fill_lower, rocblas_diagonal_non_unit, d, f, d, info + 1) !=
          rocblas_status_success)
    e = hipErrorUnknown;
  if (e == hipSuccess) {
    hipLaunchKernelGGL(flip_upper_kernel, dim3(blocks_for(nn, 256)), dim3(256), 0, stream, f, d, u);
    e = hipGetLastError();
  }
  rocblas_int host_info[2] = {0, 0};
  if (e == hipSuccess) e = hipMemcpyAsync(host_info, info, sizeof(host_info), hipMemcpyDeviceToHost, stream);
  const hipError_t es = hipStreamSynchronize(stream);
  if (e == hipSuccess) e = es;
  if (e == hipSuccess) *info_out = host_info[0] != 0 ? host_info[0] : (host_info[1] != 0 ? -host_info[1] : 0);
  if (handle) rocblas_destroy_handle(handle);
  if (f) (void)hipFree(f);
  if (lambda) (void)hipFree(lambda);
  return e;
}

// Workspace of kashin_optq_quantize_noalloc: one array per device, holding the error matrix and the
// factor block of the chunk being carried (optq_workspace_bytes of the call).  Every call on a
// device uses the same array; both parts are written before they are read within each chunk, so
// nothing needs clearing, and calls that overlap on one device race.
static __device__ __align__(256) char scratch[kOptqStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// The device address of `scratch` on the current device, looked up once per device (the array's
// name is a host-side stand-in: host code passes this address, never the name, to kernels).
hipError_t optq_static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

int64_t optq_workspace_bytes(int64_t d_in, int n, int chunk) {
  const int64_t c = chunk < d_in ? chunk : d_in;
  const int64_t e_bytes = ((c * n * 4) + 255) & ~int64_t(255);
  return e_bytes + c * d_in * 4;
}

hipError_t optq_error(const float* w, int64_t ldw, const float* q, int n, int64_t row0, int rows, const double* u,
                      int64_t ldu, float* e, hipStream_t s) {
  hipLaunchKernelGGL(error_kernel, dim3(blocks_for(static_cast<int64_t>(rows) * n, 256)), dim3(256), 0, s, w, ldw, q,
                     n, row0, rows, u, ldu, e);
  return hipGetLastError();
}

hipError_t optq_rank1(float* w, int64_t ldw, int n, int64_t i, int64_t j0, int64_t j1, const double* u, int64_t ldu,
                      const float* err, hipStream_t s) {
  if (j1 <= j0) return hipSuccess;
  hipLaunchKernelGGL(rank1_kernel, dim3(blocks_for((j1 - j0) * n, 256)), dim3(256), 0, s, w, ldw, n, i, j0, j1, u, ldu,
                     err);
  return hipGetLastError();
}

hipError_t optq_chunk_factor(const double* u, const double* v, int64_t ld, int64_t c0, int rows, int64_t c1,
                             int64_t rest, bool exact, float* m, hipStream_t s) {
  if (rest <= 0) return hipSuccess;
  if (exact) {
    hipLaunchKernelGGL(copy_block_kernel, dim3(blocks_for(rows * rest, 256)), dim3(256), 0, s, u, ld, c0, rows, c1,
                       rest, m);
  } else {
    if (rows > kMaxChunk) return hipErrorInvalidValue;
    const dim3 grid(blocks_for(rest, kMR), static_cast<unsigned>((rows + kMK - 1) / kMK));
    hipLaunchKernelGGL(chunk_factor_kernel, grid, dim3(kMT), 0, s, v, u, ld, c0, rows, c1, rest, m);
  }
  return hipGetLastError();
}

hipError_t optq_update(float* w_rest, int64_t ldw, const float* m, const float* e, int rows, int64_t rest, int n,
                       hipStream_t s) {
  if (rest <= 0) return hipSuccess;
  const dim3 grid(blocks_for(n, kGB), static_cast<unsigned>((rest + kGB - 1) / kGB));
  hipLaunchKernelGGL(update_gemm_kernel, grid, dim3(kGT), 0, s, w_rest, ldw, m, e, rows, rest, n);
  return hipGetLastError();
}

}  // namespace kashin
