// Internal interface between the C-ABI host layer (kashin_api.cpp) and the HIP
// kernels (kashin_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace kashin {

// bfloat16 input (KASHIN_BF16): the upper 16 bits of an IEEE binary32, widened exactly by a shift
struct bf16_t {
  uint16_t bits;
};
__device__ inline float bf16_to_f32(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v.bits) << 16);
}

enum Mode : int32_t {
  MODE_DECOMPOSE = 0,  // write u, vhat (+ r, cstep, bounds)
  MODE_QUANTIZE = 1,   // fused decompose + cluster + pack, write codes and centres only
  MODE_TRACE = 2,      // decompose listed rows and record every sign decision
  MODE_APPLY_P = 3,    // y = P x
  MODE_RECON = 4,      // w_hat = u_q + P v_q
  MODE_SCHEDULE = 5,   // greedy with another step schedule (writes u, vhat, r; traces listed rows)
};

enum Schedule : int32_t {
  SCHED_ALTERNATING = 0,  // blocks u, u, vhat, vhat (Alg. 2)
  SCHED_REVERSE = 1,      // blocks vhat, vhat, u, u
  SCHED_ADAPTIVE = 2,     // the half with the larger l1 correlation, step ||.||_1 / N
  SCHED_ORIGINAL = 3,     // Alg. 1: that choice, projection step ||.||_1 / nnz, stop at ||rho|| < tol
};

// One matrix of a grouped launch: its plan's tables, rows, codes, centres, output rows, and the
// index of its first row pair among the launch's items.  Quantisation reads w and writes the
// codes and centres; reconstruction reads the codes (w = codes_u) and centres and writes y.
struct GroupItem {
  const float2* tw;
  const float4* mid4;
  const void* w;
  int64_t ldw;
  int64_t m;
  uint8_t* codes_u;
  uint8_t* codes_v;
  float* centers;
  float* y;
  int64_t ldy;
  int64_t pair0;
  int64_t wg0;  // reconstruction: the matrix's first workgroup (it takes wg0 .. next matrix's wg0 - 1)
};
constexpr int kMaxGroup = 16;  // matrices per grouped launch (the table travels in the kernel arguments)
constexpr int64_t kPmapGrid = 2048;  // persistent y = P x / reconstruction grid: resident workgroups, a few times over

// Everything a launch needs, passed to the kernel by value.
struct KArgs {
  // operator tables (plan-owned, device)
  const float2* tw;    // per-pass twiddle tables (layout: see build_tables in kashin_api.cpp)
  const float4* mid4;  // first inverse pass, per (j, r): {f.x, f.y, LDS byte address of the source, 0}
  int32_t iters;       // blocks of Alg. 2
  int32_t mode;
  int32_t dtype;       // input dtype (KASHIN_F32 / KASHIN_F16)
  int32_t lloyd;       // Lloyd passes for the fused clustering
  int64_t m;           // rows in the matrix
  int64_t ldw;         // leading dimension of the input matrix
  const void* w;       // input rows (w, x, or codes_u for MODE_RECON)
  // outputs / other inputs
  float* u;
  float* vhat;
  float* r;
  float* cstep;
  float* bounds;
  uint8_t* codes_u;
  uint8_t* codes_v;
  float* centers;
  const uint8_t* in_codes_v;  // MODE_RECON
  const float* in_centers;    // MODE_RECON
  float* y;                   // MODE_APPLY_P / MODE_RECON output
  int64_t ldy;
  // trace
  const int64_t* rows;
  int64_t nrows;
  int8_t* tr_signs;
  float* tr_c;
  // MODE_SCHEDULE
  int32_t schedule;
  float tol;
  int8_t* tr_choice;
  float* tr_r2;
  // incoherence rotation fused into the load (quantize, decompose, trace) or the store (recon)
  int32_t rot;
  float rot_scale;  // 1 / sqrt(2^a), n = 2^a b
  uint64_t rot_seed;
  // MODE_QUANTIZE over several matrices of one vector length (ngroup > 0): item p is row pair
  // p - group[g].pair0 of the last matrix g with group[g].pair0 <= p.  MODE_RECON: workgroup b
  // serves the last matrix g with group[g].wg0 <= b, walking its row pairs with the stride of
  // that matrix's workgroup count
  int32_t ngroup;
  GroupItem group[kMaxGroup];
};

struct ClusterArgs {
  const float* u;
  const float* vhat;
  const float* cstep;
  int64_t m;
  int32_t n;
  int32_t lloyd;
  uint8_t* codes_u;
  uint8_t* codes_v;
  float* centers;
};

// Radix plan of the pair kernel for vector length n: threads per workgroup and the radices
// of the forward FFT passes.
struct PlanShape {
  int n = 0;
  int threads = 0;
  int np = 0;
  int rad[8] = {};
};
bool plan_shape(int n, PlanShape* out);

// Whether the pair kernel's transform of length n (threads per workgroup, forward radices
// rad[0..np)) has a single radix r = rad[0] <= 16, a power of two, with one butterfly of every
// pass per thread (threads = n / r, a multiple of 32): such transforms stay resident in LDS and
// take the wide padding below.
__host__ __device__ constexpr bool uniform_resident(int n, int threads, int np, const int* rad) {
  if (np < 2 || rad[0] > 16 || (rad[0] & (rad[0] - 1)) != 0 || threads != n / rad[0] || (n / rad[0]) % 32 != 0)
    return false;
  for (int p = 1; p < np; ++p)
    if (rad[p] != rad[0]) return false;
  return true;
}

// LDS layout of the pair kernel's transform buffer: element i of a length-n vector lives at
// float2 slot i + pad_width(w) * (i >> pad_shift(n, w)), w = uniform_resident(...).  gfx950
// resolves bank conflicts of an 8-byte LDS read per 32 lanes over 64 four-byte banks, of an
// 8-byte write per 16 lanes over 32 banks and of a 16-byte write per 8 lanes over 32 banks.
// Contiguous reads therefore want no gap inside an aligned run of 32 elements and stride-16
// writes a spare slot per 16 elements.  Uniform resident transforms take two spare slots per
// 32 elements (their first pass writes its stride-16 outputs as 16-byte pairs from a lane
// order that puts one parity of butterflies in each eight lanes); other lengths that are
// multiples of 512 one per 32, the rest (pass strides of 16 times an odd number) one per 16.
__host__ __device__ constexpr int pad_shift(int n, bool wide) { return (wide || n % 512 == 0) ? 5 : 4; }
__host__ __device__ constexpr int pad_width(bool wide) { return wide ? 2 : 1; }
__host__ __device__ constexpr int pad_slot(int n, bool wide, int i) {
  return i + pad_width(wide) * (i >> pad_shift(n, wide));
}

bool supported_n(int n);
// Launch the pair kernel for vector length n; grid = number of work items (pairs or listed rows).
hipError_t launch_pair(int n, const KArgs& a, int64_t grid, hipStream_t stream);
hipError_t launch_cluster(const ClusterArgs& a, hipStream_t stream);

// Error-compensated quantisation (kashin_optq.hip).  optq_factor_device: U (upper, U^T U =
// (H + lambda I)^-1, lambda = damp mean(diag H)) and, if v != null, V = U^-1, both d x d float64
// row-major; allocates and frees its temporaries and synchronises `stream`; *info != 0 when the
// damped Hessian is not positive definite (> 0) or its factor singular (< 0).
hipError_t optq_factor_device(const float* h, int d, int64_t ldh, double damp, double* u, double* v,
                              hipStream_t stream, int* info);
constexpr int kOptqMaxChunk = 128;
int64_t optq_workspace_bytes(int64_t d_in, int n, int chunk);
// kashin_optq_quantize_noalloc's workspace: a static device array of this many bytes per device;
// optq_static_scratch gives its address on the current device
constexpr int64_t kOptqStaticScratchBytes = int64_t(16) << 20;
hipError_t optq_static_scratch(void** out);
hipError_t optq_error(const float* w, int64_t ldw, const float* q, int n, int64_t row0, int rows, const double* u,
                      int64_t ldu, float* e, hipStream_t s);
hipError_t optq_rank1(float* w, int64_t ldw, int n, int64_t i, int64_t j0, int64_t j1, const double* u, int64_t ldu,
                      const float* err, hipStream_t s);
hipError_t optq_chunk_factor(const double* u, const double* v, int64_t ld, int64_t c0, int rows, int64_t c1,
                             int64_t rest, bool exact, float* m, hipStream_t s);
hipError_t optq_update(float* w_rest, int64_t ldw, const float* m, const float* e, int rows, int64_t rest, int n,
                       hipStream_t s);

// Incoherence rotation of rows (kashin_rotate.hip).
bool rotate_supported_n(int n);
hipError_t launch_rotate(int n, uint64_t seed, bool inverse, const void* x, int dtype, int64_t ldx, float* y,
                         int64_t ldy, int64_t m, hipStream_t stream);

}  // namespace kashin
