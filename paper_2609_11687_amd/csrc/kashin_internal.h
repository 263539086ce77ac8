// Internal interface between the C-ABI host layer (kashin_api.cpp) and the HIP
// kernels (kashin_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace kashin {

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

bool supported_n(int n);
// Launch the pair kernel for vector length n; grid = number of work items (pairs or listed rows).
hipError_t launch_pair(int n, const KArgs& a, int64_t grid, hipStream_t stream);
hipError_t launch_cluster(const ClusterArgs& a, hipStream_t stream);

// Incoherence rotation of rows (kashin_rotate.hip).
bool rotate_supported_n(int n);
hipError_t launch_rotate(int n, uint64_t seed, bool inverse, const void* x, int dtype, int64_t ldx, float* y,
                         int64_t ldy, int64_t m, hipStream_t stream);

}  // namespace kashin
