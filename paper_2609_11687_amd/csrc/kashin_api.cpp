// C-ABI host layer: argument validation, plan construction (sign mask, FFT twiddles,
// eps-folded frequency table) and kernel dispatch.  Every check runs on the host before
// any HIP call, so argument errors are reported without touching a device.
#include "kashin.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <set>
#include <string>
#include <vector>

#include "kashin_internal.h"

struct kashin_plan_s {
  int32_t n = 0;
  int32_t iters = 0;
  uint64_t seed = 0;
  int device = 0;
  std::vector<int8_t> eps;
  void* d_tables = nullptr;  // twiddle tables, then the eps table (16-byte aligned)
  float2* d_tw = nullptr;
  float4* d_mid = nullptr;
};

namespace {

thread_local std::string g_last_error;
std::mutex g_plans_mu;
std::set<const kashin_plan_s*> g_plans;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return KASHIN_OK;
}

bool dtype_ok(int32_t dtype) { return dtype == KASHIN_F32 || dtype == KASHIN_F16 || dtype == KASHIN_BF16; }

bool live(const kashin_plan_s* p) {
  std::lock_guard<std::mutex> lk(g_plans_mu);
  return p != nullptr && g_plans.count(p) != 0;
}

// splitmix64 (Steele, Lea, Flood 2014): the eps generator, see kashin_signs.
void make_signs(int32_t n, uint64_t seed, int8_t* out) {
  uint64_t s = seed;
  for (int32_t i = 0; i < n; ++i) {
    s += 0x9E3779B97F4A7C15ull;
    uint64_t z = s;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    out[i] = (z >> 63) ? int8_t(-1) : int8_t(1);
  }
}

// Tables of the pair kernel for length n (layout shared with kashin_pair_impl.h):
//  tw:  one table per Stockham pass with stride NS > 1 -- forward passes 1..np-1, then
//       inverse passes 1..np-1 (radices in reverse order) -- entry [jm][r] =
//       exp(-2 pi i r jm / (NS R)), each table padded to an even length;
//  mid: for the first inverse pass (radix R = last forward radix, stride 1), entry j R + r
//       for element k = j + r n/R: Y'_k = f_k Y_s(k) with s(k) = k and f_k = eps_k / n when
//       eps_k == eps_{n-k} (k = 0 and k = n/2 pair with themselves), else s(k) = n - k and
//       f_k = eps_k exp(i pi k / n) / n; stored as {Re f, Im f, LDS byte address of s(k), eps_k}.
void build_tables(int n, const int8_t* eps, std::vector<float2>* tw, std::vector<float4>* mid) {
  kashin::PlanShape sh;
  kashin::plan_shape(n, &sh);
  const bool wide = kashin::uniform_resident(n, sh.threads, sh.np, sh.rad);
  const double pi = 3.14159265358979323846;
  auto add_table = [&](int R, int NS) {
    for (int jm = 0; jm < NS; ++jm)
      for (int r = 0; r < R; ++r) {
        const double ang = -2.0 * pi * double(r) * double(jm) / (double(NS) * double(R));
        tw->push_back(make_float2(float(std::cos(ang)), float(std::sin(ang))));
      }
    if (tw->size() % 2) tw->push_back(make_float2(0.f, 0.f));
  };
  for (int q = 1; q < sh.np; ++q) {  // forward passes
    int ns = 1;
    for (int i = 0; i < q; ++i) ns *= sh.rad[i];
    add_table(sh.rad[q], ns);
  }
  for (int q = 1; q < sh.np; ++q) {  // inverse passes
    int ns = 1;
    for (int i = 0; i < q; ++i) ns *= sh.rad[sh.np - 1 - i];
    add_table(sh.rad[sh.np - 1 - q], ns);
  }
  const int R = sh.rad[sh.np - 1];
  const int nb = n / R;
  mid->assign(n, make_float4(0.f, 0.f, 0.f, 0.f));
  for (int j = 0; j < nb; ++j)
    for (int r = 0; r < R; ++r) {
      const int k = j + r * nb;
      const int partner = (n - k) % n;
      const double ek = eps[k];
      float fx, fy;
      int src;
      if (eps[k] == eps[partner]) {
        fx = float(ek / n);
        fy = 0.f;
        src = k;
      } else {
        const double ang = pi * double(k) / double(n);
        fx = float(ek * std::cos(ang) / n);
        fy = float(ek * std::sin(ang) / n);
        src = partner;
      }
      const int addr = kashin::pad_slot(n, wide, src) * int(sizeof(float2));
      float faddr;
      std::memcpy(&faddr, &addr, sizeof(faddr));
      (*mid)[j * R + r] = make_float4(fx, fy, faddr, float(ek));
    }
}

int hip_fail(hipError_t e, const char* what) {
  return fail(KASHIN_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

int check_common(kashin_plan_t plan, int64_t m) {
  if (!live(plan)) return fail(KASHIN_E_INVALID, "plan is null or destroyed");
  if (m < 0) return fail(KASHIN_E_INVALID, "m must be >= 0 (got %lld)", (long long)m);
  return KASHIN_OK;
}

kashin::KArgs base_args(const kashin_plan_s* p, int mode) {
  kashin::KArgs a;
  std::memset(&a, 0, sizeof(a));
  a.tw = p->d_tw;
  a.mid4 = p->d_mid;
  a.iters = p->iters;
  a.mode = mode;
  return a;
}

// the rotation fused into a pair kernel: seed and 1 / sqrt(2^a), n = 2^a b (as kashin_rotate)
void set_rotation(kashin::KArgs* a, int n, uint64_t seed) {
  a->rot = 1;
  a->rot_seed = seed;
  a->rot_scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(n & -n)));
}

int launch(const kashin_plan_s* p, const kashin::KArgs& a, int64_t grid, void* stream) {
  const hipError_t e = kashin::launch_pair(p->n, a, grid, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return ok();
}

}  // namespace

extern "C" {

int kashin_supported_n(int32_t n) { return (n >= 2 && (n % 2) == 0 && kashin::supported_n(n)) ? 1 : 0; }

int kashin_signs(int32_t n, uint64_t seed, int8_t* eps_host) {
  if (n < 1) return fail(KASHIN_E_INVALID, "n must be >= 1");
  if (eps_host == nullptr) return fail(KASHIN_E_INVALID, "eps_host is null");
  make_signs(n, seed, eps_host);
  return ok();
}

int kashin_plan(kashin_plan_t* out, int32_t n, uint64_t sign_seed, int32_t iters) {
  if (out == nullptr) return fail(KASHIN_E_INVALID, "out is null");
  *out = nullptr;
  if (iters < 1) return fail(KASHIN_E_INVALID, "iters must be >= 1 (got %d)", iters);
  if (!kashin_supported_n(n)) return fail(KASHIN_E_UNSUPPORTED_N, "vector length %d has no compiled kernel", n);
  kashin_plan_s* p = new (std::nothrow) kashin_plan_s();
  if (p == nullptr) return fail(KASHIN_E_NOMEM, "host allocation failed");
  p->n = n;
  p->iters = iters;
  p->seed = sign_seed;
  p->eps.resize(n);
  make_signs(n, sign_seed, p->eps.data());

  std::vector<float2> tw;
  std::vector<float4> mid;
  build_tables(n, p->eps.data(), &tw, &mid);
  const size_t tw_bytes = ((tw.size() * sizeof(float2)) + 255) & ~size_t(255);
  const size_t bytes = tw_bytes + mid.size() * sizeof(float4);
  hipError_t e = hipGetDevice(&p->device);
  if (e == hipSuccess) e = hipMalloc(&p->d_tables, bytes);
  if (e == hipSuccess) {
    p->d_tw = static_cast<float2*>(p->d_tables);
    p->d_mid = reinterpret_cast<float4*>(static_cast<char*>(p->d_tables) + tw_bytes);
    if (!tw.empty()) e = hipMemcpy(p->d_tw, tw.data(), tw.size() * sizeof(float2), hipMemcpyHostToDevice);
  }
  if (e == hipSuccess) e = hipMemcpy(p->d_mid, mid.data(), mid.size() * sizeof(float4), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    if (p->d_tables) (void)hipFree(p->d_tables);
    delete p;
    return hip_fail(e, "plan device tables");
  }
  {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    g_plans.insert(p);
  }
  *out = p;
  return ok();
}

int kashin_plan_destroy(kashin_plan_t plan) {
  {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    if (plan == nullptr || g_plans.erase(plan) == 0) return fail(KASHIN_E_INVALID, "plan is null or destroyed");
  }
  if (plan->d_tables) (void)hipFree(plan->d_tables);
  delete plan;
  return ok();
}

int kashin_plan_signs(kashin_plan_t plan, int8_t* eps_host) {
  if (!live(plan)) return fail(KASHIN_E_INVALID, "plan is null or destroyed");
  if (eps_host == nullptr) return fail(KASHIN_E_INVALID, "eps_host is null");
  std::memcpy(eps_host, plan->eps.data(), plan->eps.size());
  return ok();
}

int kashin_plan_info(kashin_plan_t plan, int32_t* n, int32_t* iters, uint64_t* seed) {
  if (!live(plan)) return fail(KASHIN_E_INVALID, "plan is null or destroyed");
  if (n) *n = plan->n;
  if (iters) *iters = plan->iters;
  if (seed) *seed = plan->seed;
  return ok();
}

int kashin_decompose(kashin_plan_t plan, const void* w, int32_t dtype, int64_t m, int64_t ldw, float* u,
                     float* vhat, float* r, float* cstep, float* bounds, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  if (!dtype_ok(dtype)) return fail(KASHIN_E_INVALID, "dtype must be F32, F16 or BF16");
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (m == 0) return ok();
  if (!w || !u || !vhat) return fail(KASHIN_E_INVALID, "w, u and vhat must be non-null");
  kashin::KArgs a = base_args(plan, kashin::MODE_DECOMPOSE);
  a.w = w;
  a.dtype = dtype;
  a.m = m;
  a.ldw = ldw;
  a.u = u;
  a.vhat = vhat;
  a.r = r;
  a.cstep = cstep;
  a.bounds = bounds;
  return launch(plan, a, (m + 1) / 2, stream);
}

int kashin_quantize(kashin_plan_t plan, const void* w, int32_t dtype, int64_t m, int64_t ldw, int32_t lloyd_iters,
                    uint8_t* codes_u, uint8_t* codes_v, float* centers, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  if (!dtype_ok(dtype)) return fail(KASHIN_E_INVALID, "dtype must be F32, F16 or BF16");
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (lloyd_iters < 0) return fail(KASHIN_E_INVALID, "lloyd_iters must be >= 0");
  if (m == 0) return ok();
  if (!w || !codes_u || !codes_v || !centers) return fail(KASHIN_E_INVALID, "w, codes and centers must be non-null");
  kashin::KArgs a = base_args(plan, kashin::MODE_QUANTIZE);
  a.w = w;
  a.dtype = dtype;
  a.m = m;
  a.ldw = ldw;
  a.lloyd = lloyd_iters;
  a.codes_u = codes_u;
  a.codes_v = codes_v;
  a.centers = centers;
  return launch(plan, a, (m + 1) / 2, stream);
}

int kashin_quantize_grouped(const kashin_quantize_item* items, int32_t count, int32_t dtype, int32_t lloyd_iters,
                            const uint64_t* rot_seed, void* stream) {
  if (count < 0) return fail(KASHIN_E_INVALID, "count must be >= 0 (got %d)", count);
  if (count == 0) return ok();
  if (items == nullptr) return fail(KASHIN_E_INVALID, "items is null");
  if (!dtype_ok(dtype)) return fail(KASHIN_E_INVALID, "dtype must be F32, F16 or BF16");
  if (lloyd_iters < 0) return fail(KASHIN_E_INVALID, "lloyd_iters must be >= 0");
  const kashin_plan_s* p0 = nullptr;
  for (int32_t i = 0; i < count; ++i) {
    const kashin_quantize_item& it = items[i];
    if (!live(it.plan)) return fail(KASHIN_E_INVALID, "item %d: plan is null or destroyed", i);
    if (p0 == nullptr) {
      p0 = it.plan;
    } else if (it.plan->n != p0->n || it.plan->iters != p0->iters || it.plan->device != p0->device) {
      return fail(KASHIN_E_INVALID, "item %d: plan (n %d, iters %d, device %d) differs from item 0's (n %d, iters %d, "
                  "device %d)", i, it.plan->n, it.plan->iters, it.plan->device, p0->n, p0->iters, p0->device);
    }
    if (it.m < 0) return fail(KASHIN_E_INVALID, "item %d: m must be >= 0 (got %lld)", i, (long long)it.m);
    if (it.ldw < p0->n) return fail(KASHIN_E_INVALID, "item %d: ldw (%lld) < n (%d)", i, (long long)it.ldw, p0->n);
    if (it.m > 0 && (!it.w || !it.codes_u || !it.codes_v || !it.centers))
      return fail(KASHIN_E_INVALID, "item %d: w, codes and centers must be non-null", i);
  }
  kashin::KArgs a = base_args(p0, kashin::MODE_QUANTIZE);
  a.dtype = dtype;
  a.lloyd = lloyd_iters;
  if (rot_seed != nullptr) {
    if (!kashin::rotate_supported_n(p0->n))
      return fail(KASHIN_E_UNSUPPORTED_N, "n = %d: the rotation needs n <= 16384 with odd part 1, 3 or 43", p0->n);
    set_rotation(&a, p0->n, *rot_seed);
  }
  int32_t g = 0;
  int64_t pairs = 0;
  for (int32_t i = 0; i < count; ++i) {
    const kashin_quantize_item& it = items[i];
    if (it.m == 0) continue;
    a.group[g] = kashin::GroupItem{it.plan->d_tw, it.plan->d_mid, it.w, it.ldw, it.m, it.codes_u, it.codes_v,
                                   it.centers, nullptr, 0, pairs, 0};
    pairs += (it.m + 1) / 2;
    if (++g == kashin::kMaxGroup || i == count - 1) {
      a.ngroup = g;
      const int st = launch(p0, a, pairs, stream);
      if (st) return st;
      g = 0;
      pairs = 0;
    }
  }
  if (g > 0) {  // the last items were empty
    a.ngroup = g;
    return launch(p0, a, pairs, stream);
  }
  return ok();
}

int kashin_trace(kashin_plan_t plan, const void* w, int32_t dtype, int64_t m, int64_t ldw, const int64_t* rows,
                 int64_t nrows, int8_t* sign_trace, float* c_trace, float* u, float* vhat, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  if (!dtype_ok(dtype)) return fail(KASHIN_E_INVALID, "dtype must be F32, F16 or BF16");
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (nrows < 0) return fail(KASHIN_E_INVALID, "nrows must be >= 0");
  if (nrows == 0 || m == 0) return ok();
  if (!w || !rows || !sign_trace || !c_trace || !u || !vhat)
    return fail(KASHIN_E_INVALID, "w, rows, sign_trace, c_trace, u and vhat must be non-null");
  kashin::KArgs a = base_args(plan, kashin::MODE_TRACE);
  a.w = w;
  a.dtype = dtype;
  a.m = m;
  a.ldw = ldw;
  a.rows = rows;
  a.nrows = nrows;
  a.tr_signs = sign_trace;
  a.tr_c = c_trace;
  a.u = u;
  a.vhat = vhat;
  return launch(plan, a, nrows, stream);
}

namespace {
int check_schedule(int32_t schedule, float tol) {
  if (schedule < KASHIN_SCHED_ALTERNATING || schedule > KASHIN_SCHED_ORIGINAL)
    return fail(KASHIN_E_INVALID, "schedule must be one of KASHIN_SCHED_*");
  if (!(tol >= 0.f)) return fail(KASHIN_E_INVALID, "tol must be >= 0");
  return KASHIN_OK;
}
}  // namespace

int kashin_decompose_schedule(kashin_plan_t plan, int32_t schedule, float tol, const void* w, int32_t dtype,
                              int64_t m, int64_t ldw, float* u, float* vhat, float* r, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  st = check_schedule(schedule, tol);
  if (st) return st;
  if (!dtype_ok(dtype)) return fail(KASHIN_E_INVALID, "dtype must be F32, F16 or BF16");
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (m == 0) return ok();
  if (!w || !u || !vhat) return fail(KASHIN_E_INVALID, "w, u and vhat must be non-null");
  kashin::KArgs a = base_args(plan, kashin::MODE_SCHEDULE);
  a.w = w;
  a.dtype = dtype;
  a.m = m;
  a.ldw = ldw;
  a.u = u;
  a.vhat = vhat;
  a.r = r;
  a.schedule = schedule;
  a.tol = tol;
  return launch(plan, a, (m + 1) / 2, stream);
}

int kashin_trace_schedule(kashin_plan_t plan, int32_t schedule, float tol, const void* w, int32_t dtype, int64_t m,
                          int64_t ldw, const int64_t* rows, int64_t nrows, int8_t* sign_trace, float* c_trace,
                          int8_t* choice_trace, float* r2_trace, float* u, float* vhat, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  st = check_schedule(schedule, tol);
  if (st) return st;
  if (!dtype_ok(dtype)) return fail(KASHIN_E_INVALID, "dtype must be F32, F16 or BF16");
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (nrows < 0) return fail(KASHIN_E_INVALID, "nrows must be >= 0");
  if (nrows == 0 || m == 0) return ok();
  if (!w || !rows || !sign_trace || !c_trace || !choice_trace || !r2_trace || !u || !vhat)
    return fail(KASHIN_E_INVALID, "w, rows, the four traces, u and vhat must be non-null");
  kashin::KArgs a = base_args(plan, kashin::MODE_SCHEDULE);
  a.w = w;
  a.dtype = dtype;
  a.m = m;
  a.ldw = ldw;
  a.rows = rows;
  a.nrows = nrows;
  a.tr_signs = sign_trace;
  a.tr_c = c_trace;
  a.tr_choice = choice_trace;
  a.tr_r2 = r2_trace;
  a.u = u;
  a.vhat = vhat;
  a.schedule = schedule;
  a.tol = tol;
  return launch(plan, a, nrows, stream);
}

int kashin_apply_p(kashin_plan_t plan, const float* x, float* y, int64_t m, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  if (m == 0) return ok();
  if (!x || !y) return fail(KASHIN_E_INVALID, "x and y must be non-null");
  if (x == y) return fail(KASHIN_E_INVALID, "x and y must not alias");
  kashin::KArgs a = base_args(plan, kashin::MODE_APPLY_P);
  a.w = x;
  a.m = m;
  a.ldw = plan->n;
  a.y = y;
  a.ldy = plan->n;
  return launch(plan, a, (m + 1) / 2, stream);
}

int kashin_quantize_rotated(kashin_plan_t plan, uint64_t rot_seed, const void* w, int32_t dtype, int64_t m,
                            int64_t ldw, int32_t lloyd_iters, uint8_t* codes_u, uint8_t* codes_v, float* centers,
                            void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  if (!kashin::rotate_supported_n(plan->n))
    return fail(KASHIN_E_UNSUPPORTED_N, "n = %d: the rotation needs n <= 16384 with odd part 1, 3 or 43", plan->n);
  if (!dtype_ok(dtype)) return fail(KASHIN_E_INVALID, "dtype must be F32, F16 or BF16");
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (lloyd_iters < 0) return fail(KASHIN_E_INVALID, "lloyd_iters must be >= 0");
  if (m == 0) return ok();
  if (!w || !codes_u || !codes_v || !centers) return fail(KASHIN_E_INVALID, "w, codes and centers must be non-null");
  kashin::KArgs a = base_args(plan, kashin::MODE_QUANTIZE);
  a.w = w;
  a.dtype = dtype;
  a.m = m;
  a.ldw = ldw;
  a.lloyd = lloyd_iters;
  a.codes_u = codes_u;
  a.codes_v = codes_v;
  a.centers = centers;
  set_rotation(&a, plan->n, rot_seed);
  return launch(plan, a, (m + 1) / 2, stream);
}

int kashin_reconstruct_rotated(kashin_plan_t plan, uint64_t rot_seed, const uint8_t* codes_u, const uint8_t* codes_v,
                               const float* centers, int64_t m, float* w_hat, int64_t ldw, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  if (!kashin::rotate_supported_n(plan->n))
    return fail(KASHIN_E_UNSUPPORTED_N, "n = %d: the rotation needs n <= 16384 with odd part 1, 3 or 43", plan->n);
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (m == 0) return ok();
  if (!codes_u || !codes_v || !centers || !w_hat) return fail(KASHIN_E_INVALID, "codes, centers and w_hat must be non-null");
  kashin::KArgs a = base_args(plan, kashin::MODE_RECON);
  a.w = codes_u;
  a.in_codes_v = codes_v;
  a.in_centers = centers;
  a.m = m;
  a.y = w_hat;
  a.ldy = ldw;
  set_rotation(&a, plan->n, rot_seed);
  return launch(plan, a, (m + 1) / 2, stream);
}

int kashin_rotate(int32_t n, uint64_t seed, int32_t inverse, const void* x, int32_t dtype, int64_t m, int64_t ldx,
                  float* y, int64_t ldy, void* stream) {
  if (!kashin::rotate_supported_n(n))
    return fail(KASHIN_E_UNSUPPORTED_N, "n = %d: the rotation needs n <= 16384 with odd part 1, 3 or 43", n);
  if (inverse != 0 && inverse != 1) return fail(KASHIN_E_INVALID, "inverse must be 0 or 1");
  if (!dtype_ok(dtype)) return fail(KASHIN_E_INVALID, "dtype must be F32, F16 or BF16");
  if (m < 0) return fail(KASHIN_E_INVALID, "m must be >= 0 (got %lld)", (long long)m);
  if (ldx < n || ldy < n) return fail(KASHIN_E_INVALID, "ldx (%lld) and ldy (%lld) must be >= n (%d)", (long long)ldx,
                                      (long long)ldy, n);
  if (m == 0) return ok();
  if (!x || !y) return fail(KASHIN_E_INVALID, "x and y must be non-null");
  const size_t esz = dtype == KASHIN_F32 ? 4 : 2;
  const uintptr_t x0 = reinterpret_cast<uintptr_t>(x), y0 = reinterpret_cast<uintptr_t>(y);
  const uintptr_t x1 = x0 + ((m - 1) * ldx + n) * esz, y1 = y0 + ((m - 1) * ldy + n) * 4;
  const bool in_place = x0 == y0 && dtype == KASHIN_F32 && ldx == ldy;
  if (!in_place && x0 < y1 && y0 < x1) return fail(KASHIN_E_INVALID, "x and y overlap without being the same rows");
  const hipError_t e =
      kashin::launch_rotate(n, seed, inverse != 0, x, dtype, ldx, y, ldy, m, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return ok();
}

int kashin_reconstruct(kashin_plan_t plan, const uint8_t* codes_u, const uint8_t* codes_v, const float* centers,
                       int64_t m, float* w_hat, int64_t ldw, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (m == 0) return ok();
  if (!codes_u || !codes_v || !centers || !w_hat) return fail(KASHIN_E_INVALID, "codes, centers and w_hat must be non-null");
  kashin::KArgs a = base_args(plan, kashin::MODE_RECON);
  a.w = codes_u;
  a.in_codes_v = codes_v;
  a.in_centers = centers;
  a.m = m;
  a.y = w_hat;
  a.ldy = ldw;
  return launch(plan, a, (m + 1) / 2, stream);
}

int kashin_reconstruct_grouped(const kashin_reconstruct_item* items, int32_t count, void* stream) {
  if (count < 0) return fail(KASHIN_E_INVALID, "count must be >= 0 (got %d)", count);
  if (count == 0) return ok();
  if (items == nullptr) return fail(KASHIN_E_INVALID, "items is null");
  const kashin_plan_s* p0 = nullptr;
  for (int32_t i = 0; i < count; ++i) {
    const kashin_reconstruct_item& it = items[i];
    if (!live(it.plan)) return fail(KASHIN_E_INVALID, "item %d: plan is null or destroyed", i);
    if (p0 == nullptr) {
      p0 = it.plan;
    } else if (it.plan->n != p0->n || it.plan->device != p0->device) {
      return fail(KASHIN_E_INVALID, "item %d: plan (n %d, device %d) differs from item 0's (n %d, device %d)", i,
                  it.plan->n, it.plan->device, p0->n, p0->device);
    }
    if (it.m < 0) return fail(KASHIN_E_INVALID, "item %d: m must be >= 0 (got %lld)", i, (long long)it.m);
    if (it.ldw < p0->n) return fail(KASHIN_E_INVALID, "item %d: ldw (%lld) < n (%d)", i, (long long)it.ldw, p0->n);
    if (it.m > 0 && (!it.codes_u || !it.codes_v || !it.centers || !it.w_hat))
      return fail(KASHIN_E_INVALID, "item %d: codes, centers and w_hat must be non-null", i);
  }
  // launches of up to kMaxGroup non-empty matrices; each matrix gets a share of the persistent
  // grid in proportion to its row pairs (at least one workgroup, at most one per pair)
  std::vector<int32_t> idx;
  for (int32_t i = 0; i < count; ++i)
    if (items[i].m > 0) idx.push_back(i);
  for (size_t c0 = 0; c0 < idx.size(); c0 += kashin::kMaxGroup) {
    const size_t c1 = std::min(idx.size(), c0 + kashin::kMaxGroup);
    int64_t pairs = 0;
    for (size_t k = c0; k < c1; ++k) pairs += (items[idx[k]].m + 1) / 2;
    const int64_t grid = std::min<int64_t>(pairs, kashin::kPmapGrid);
    kashin::KArgs a = base_args(p0, kashin::MODE_RECON);
    int64_t wg = 0, pair0 = 0;
    for (size_t k = c0; k < c1; ++k) {
      const kashin_reconstruct_item& it = items[idx[k]];
      const int64_t np = (it.m + 1) / 2;
      const int64_t nwg = std::max<int64_t>(1, std::min<int64_t>(np, grid * np / pairs));
      a.group[k - c0] = kashin::GroupItem{it.plan->d_tw, it.plan->d_mid, it.codes_u, 0, it.m, nullptr,
                                          const_cast<uint8_t*>(it.codes_v), const_cast<float*>(it.centers), it.w_hat,
                                          it.ldw, pair0, wg};
      wg += nwg;
      pair0 += np;
    }
    a.ngroup = static_cast<int32_t>(c1 - c0);
    const hipError_t e = kashin::launch_pair(p0->n, a, wg, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
  }
  return ok();
}

int kashin_cluster2bit(kashin_plan_t plan, const float* u, const float* vhat, const float* cstep, int64_t m,
                       int32_t lloyd_iters, uint8_t* codes_u, uint8_t* codes_v, float* centers, void* stream) {
  int st = check_common(plan, m);
  if (st) return st;
  if (lloyd_iters < 0) return fail(KASHIN_E_INVALID, "lloyd_iters must be >= 0");
  if (m == 0) return ok();
  if (!u || !vhat || !cstep || !codes_u || !codes_v || !centers)
    return fail(KASHIN_E_INVALID, "u, vhat, cstep, codes and centers must be non-null");
  kashin::ClusterArgs a;
  a.u = u;
  a.vhat = vhat;
  a.cstep = cstep;
  a.m = m;
  a.n = plan->n;
  a.lloyd = lloyd_iters;
  a.codes_u = codes_u;
  a.codes_v = codes_v;
  a.centers = centers;
  const hipError_t e = kashin::launch_cluster(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "cluster launch");
  return ok();
}

int kashin_optq_factor(const float* h, int32_t d, int64_t ldh, double damp, double* u, double* v, void* stream) {
  if (d < 1) return fail(KASHIN_E_INVALID, "d must be >= 1 (got %d)", d);
  if (ldh < d) return fail(KASHIN_E_INVALID, "ldh (%lld) < d (%d)", (long long)ldh, d);
  if (!(damp >= 0.0) || !(damp <= 1e30)) return fail(KASHIN_E_INVALID, "damp must be finite and >= 0");
  if (!h || !u) return fail(KASHIN_E_INVALID, "h and u must be non-null");
  int info = 0;
  const hipError_t e = kashin::optq_factor_device(h, d, ldh, damp, u, v, static_cast<hipStream_t>(stream), &info);
  if (e != hipSuccess) return hip_fail(e, "compensation factor");
  if (info > 0)
    return fail(KASHIN_E_INVALID, "the damped Hessian is not positive definite (leading minor %d)", info);
  if (info < 0) return fail(KASHIN_E_INVALID, "the Cholesky factor is singular (diagonal entry %d)", -info);
  return ok();
}

int64_t kashin_optq_workspace_bytes(int64_t d_in, int32_t n, int32_t chunk) {
  if (d_in < 0 || n < 1 || chunk < 1 || chunk > kashin::kOptqMaxChunk) return -1;
  return kashin::optq_workspace_bytes(d_in, n, chunk);
}

namespace {
// The compensation loop of kashin_optq_quantize with workspace `work` (at least
// optq_workspace_bytes(d_in, n, chunk) bytes of device memory).
int optq_run(kashin_plan_t plan, float* w_t, int64_t d_in, int64_t ldw, const double* u, const double* v,
             int64_t ldu, int64_t quantize_rows, int32_t chunk, int32_t exact, int32_t lloyd_iters, uint8_t* codes_u,
             uint8_t* codes_v, float* centers, float* q_t, char* work, void* stream) {
  const int n = plan->n;
  const int64_t nb = (n + 3) / 4;
  const int64_t ce = std::min<int64_t>(chunk, d_in);
  float* e_buf = reinterpret_cast<float*>(work);
  float* m_buf = reinterpret_cast<float*>(work + (((ce * n * 4) + 255) & ~int64_t(255)));
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int64_t c0 = 0; c0 < quantize_rows; c0 += chunk) {
    const int64_t c1 = std::min<int64_t>(c0 + chunk, quantize_rows);
    const int rows = static_cast<int>(c1 - c0);
    const int64_t steps = exact ? rows : 1;  // exact: one column at a time
    for (int64_t t = 0; t < steps; ++t) {
      const int64_t r0 = exact ? c0 + t : c0, r1 = exact ? r0 + 1 : c1;
      int st = kashin_quantize(plan, w_t + r0 * ldw, KASHIN_F32, r1 - r0, ldw, lloyd_iters, codes_u + r0 * nb,
                               codes_v + r0 * nb, centers + r0 * 8, stream);
      if (st) return st;
      st = kashin_reconstruct(plan, codes_u + r0 * nb, codes_v + r0 * nb, centers + r0 * 8, r1 - r0, q_t + r0 * n, n,
                              stream);
      if (st) return st;
      if (exact) {
        // err_i = (w_i - q_i) / U_ii into row i - c0 of the chunk's error matrix, then carried to
        // the chunk's later columns
        hipError_t e = kashin::optq_error(w_t, ldw, q_t, n, r0, 1, u, ldu, e_buf + (r0 - c0) * n, s);
        if (e == hipSuccess) e = kashin::optq_rank1(w_t, ldw, n, r0, r0 + 1, c1, u, ldu, e_buf + (r0 - c0) * n, s);
        if (e != hipSuccess) return hip_fail(e, "compensation kernels");
      }
    }
    const int64_t rest = d_in - c1;
    if (rest <= 0) continue;
    hipError_t e = hipSuccess;
    if (!exact) e = kashin::optq_error(w_t, ldw, q_t, n, c0, rows, nullptr, 0, e_buf, s);  // Delta
    if (e == hipSuccess) e = kashin::optq_chunk_factor(u, v, ldu, c0, rows, c1, rest, exact != 0, m_buf, s);
    if (e == hipSuccess) e = kashin::optq_update(w_t + c1 * ldw, ldw, m_buf, e_buf, rows, rest, n, s);
    if (e != hipSuccess) return hip_fail(e, "compensation kernels");
  }
  return ok();
}

int optq_check(kashin_plan_t plan, float* w_t, int64_t d_in, int64_t ldw, const double* u, const double* v,
               int64_t ldu, int64_t quantize_rows, int32_t chunk, int32_t exact, int32_t lloyd_iters,
               uint8_t* codes_u, uint8_t* codes_v, float* centers, float* q_t) {
  int st = check_common(plan, d_in);
  if (st) return st;
  if (ldu < d_in) return fail(KASHIN_E_INVALID, "ldu (%lld) < d_in (%lld)", (long long)ldu, (long long)d_in);
  if (quantize_rows < 0 || quantize_rows > d_in)
    return fail(KASHIN_E_INVALID, "quantize_rows must be in [0, d_in] (got %lld)", (long long)quantize_rows);
  if (ldw < plan->n) return fail(KASHIN_E_INVALID, "ldw (%lld) < n (%d)", (long long)ldw, plan->n);
  if (chunk < 1 || chunk > kashin::kOptqMaxChunk)
    return fail(KASHIN_E_INVALID, "chunk must be in [1, %d] (got %d)", kashin::kOptqMaxChunk, chunk);
  if (exact != 0 && exact != 1) return fail(KASHIN_E_INVALID, "exact must be 0 or 1");
  if (lloyd_iters < 0) return fail(KASHIN_E_INVALID, "lloyd_iters must be >= 0");
  if (d_in > 0 && (!w_t || !u || !codes_u || !codes_v || !centers || !q_t))
    return fail(KASHIN_E_INVALID, "w_t, u, codes, centers and q_t must be non-null");
  if (d_in > 0 && !exact && !v) return fail(KASHIN_E_INVALID, "the chunk form needs v");
  return KASHIN_OK;
}
}  // namespace

int kashin_optq_quantize(kashin_plan_t plan, float* w_t, int64_t d_in, int64_t ldw, const double* u, const double* v,
                         int64_t ldu, int64_t quantize_rows, int32_t chunk, int32_t exact, int32_t lloyd_iters,
                         uint8_t* codes_u, uint8_t* codes_v, float* centers, float* q_t, void* work,
                         int64_t work_bytes, void* stream) {
  int st = optq_check(plan, w_t, d_in, ldw, u, v, ldu, quantize_rows, chunk, exact, lloyd_iters, codes_u, codes_v,
                      centers, q_t);
  if (st) return st;
  if (quantize_rows == 0) return ok();
  const int64_t need = kashin::optq_workspace_bytes(d_in, plan->n, chunk);
  if (!work || work_bytes < need)
    return fail(KASHIN_E_INVALID, "work must hold %lld bytes (got %lld)", (long long)need, (long long)work_bytes);
  return optq_run(plan, w_t, d_in, ldw, u, v, ldu, quantize_rows, chunk, exact, lloyd_iters, codes_u, codes_v,
                  centers, q_t, static_cast<char*>(work), stream);
}

int kashin_optq_quantize_noalloc(kashin_plan_t plan, float* w_t, int64_t d_in, int64_t ldw, const double* u,
                                 const double* v, int64_t ldu, int64_t quantize_rows, int32_t chunk, int32_t exact,
                                 int32_t lloyd_iters, uint8_t* codes_u, uint8_t* codes_v, float* centers, float* q_t,
                                 void* stream) {
  int st = optq_check(plan, w_t, d_in, ldw, u, v, ldu, quantize_rows, chunk, exact, lloyd_iters, codes_u, codes_v,
                      centers, q_t);
  if (st) return st;
  if (quantize_rows == 0) return ok();
  const int64_t need = kashin::optq_workspace_bytes(d_in, plan->n, chunk);
  if (need > kashin::kOptqStaticScratchBytes)
    return fail(KASHIN_E_INVALID, "d_in = %lld, n = %d, chunk = %d need %lld bytes of workspace, above the %lld of the "
                "static array (use kashin_optq_quantize)", (long long)d_in, plan->n, chunk, (long long)need,
                (long long)kashin::kOptqStaticScratchBytes);
  void* work = nullptr;
  const hipError_t e = kashin::optq_static_scratch(&work);
  if (e != hipSuccess) return hip_fail(e, "static workspace address");
  return optq_run(plan, w_t, d_in, ldw, u, v, ldu, quantize_rows, chunk, exact, lloyd_iters, codes_u, codes_v,
                  centers, q_t, static_cast<char*>(work), stream);
}

const char* kashin_status_string(int status) {
  switch (status) {
    case KASHIN_OK: return "ok";
    case KASHIN_E_INVALID: return "invalid argument";
    case KASHIN_E_UNSUPPORTED_N: return "unsupported vector length";
    case KASHIN_E_NOMEM: return "out of memory";
    case KASHIN_E_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* kashin_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
