// Route (K5): SMetric's stick-or-balance rule.
//
// Paper: Sec. 4.2 pseudocode, (a) stateless session-centric routing -- prev = argmax c,
// stick when the request is a follow-up, prev still caches its session and (prev meets
// its TTFT deadline or no instance does), else balance by rr_argmin of the estimated
// load; (b) SLO checks -- meets_ttft compares the estimated prefill time with SLACK times
// the TTFT SLO b + a L (Sec. 4.1), none_meets_ttft is the last resort; (c) load model --
// estimate_load = q[i] + prefill_cost, prefill_cost = Eq. (1) with n = L - hit.
//
// Exact integer form (smetric.h): all quantities are doubled so that Eq. (1)'s n/2 term
// stays integral, and products are formed in 128 bits.
//
// Mapping to gfx950: one wavefront per request; lane l scans instances l, l+64, ...,
// keeping (max c, lowest id) and (min est2, rotation distance); two butterfly
// reductions across the wavefront finish the argmax and the argmin; lane 0 decides.
#include "common.h"

namespace smk {
namespace {

constexpr int RW = 4;  // waves per workgroup
typedef __int128 i128;
constexpr int64_t NO_DECODE = int64_t(1) << 62;  // decode slack meaning "no live decode"

struct RouteParams {
  int64_t c_lin, c_att, slo_b, slo_a;
  int32_t slack_num, slack_den, hit_num, hit_den, B;
};

__device__ __forceinline__ i128 est2(const RouteParams &p, int64_t L, int32_t c, int64_t q) {
  const i128 n = L - int64_t(p.B) * c;
  return i128(2) * q + i128(2) * p.c_lin * n + i128(p.c_att) * n * (i128(2) * L - n);
}

__device__ __forceinline__ i128 shfl_xor128(i128 v, int m) {
  const uint64_t lo = uint64_t(v), hi = uint64_t(v >> 64);
  const uint64_t lo2 = (uint64_t(uint32_t(__shfl_xor(int(lo >> 32), m, 64))) << 32) |
                       uint32_t(__shfl_xor(int(uint32_t(lo)), m, 64));
  const uint64_t hi2 = (uint64_t(uint32_t(__shfl_xor(int(hi >> 32), m, 64))) << 32) |
                       uint32_t(__shfl_xor(int(uint32_t(hi)), m, 64));
  return (i128(hi2) << 64) | i128(lo2);
}

__global__ __launch_bounds__(64 * RW) void route_kernel(const int32_t *__restrict__ matched,
                                                        int32_t n_req, int32_t I,
                                                        const int32_t *__restrict__ prompt_len,
                                                        const int32_t *__restrict__ hist_len,
                                                        const int32_t *__restrict__ turn,
                                                        const int64_t *__restrict__ q,
                                                        RouteParams p, uint64_t rr_base,
                                                        int32_t *__restrict__ target,
                                                        uint8_t *__restrict__ branch) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * RW + wave;
  if (r >= n_req) return;
  const int32_t *c = matched + int64_t(r) * I;
  const int64_t L = prompt_len[r];
  const int32_t hist = hist_len[r], tr = turn[r];
  bool ok = L >= 0 && L <= (int64_t(1) << 24) && hist >= 0 && tr >= 0;
  const int64_t max_c = ok ? L / p.B : -1;
  const int32_t start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));

  int32_t best_c = -1, best_ci = 0x7FFFFFFF;  // argmax c, lowest id
  i128 best_e = 0;
  int32_t best_d = 0x7FFFFFFF;                // argmin (est2, rotation distance)
  for (int32_t i = lane; i < I; i += 64) {
    const int32_t ci = c[i];
    const int64_t qi = q[i];
    if (ci < 0 || ci > max_c || qi < 0 || qi >= (int64_t(1) << 62)) ok = false;
    if (ci > best_c) {
      best_c = ci;
      best_ci = i;
    }
    const i128 e = est2(p, L, ci, qi);
    const int32_t d = i >= start ? i - start : i - start + I;
    if (best_d == 0x7FFFFFFF || e < best_e || (e == best_e && d < best_d)) {
      best_e = e;
      best_d = d;
    }
  }
  ok = __ballot(!ok) == 0;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const int32_t oc = __shfl_xor(best_c, m, 64), oi = __shfl_xor(best_ci, m, 64);
    if (oc > best_c || (oc == best_c && oi < best_ci)) {
      best_c = oc;
      best_ci = oi;
    }
    const i128 oe = shfl_xor128(best_e, m);
    const int32_t od = __shfl_xor(best_d, m, 64);
    if (od != 0x7FFFFFFF && (best_d == 0x7FFFFFFF || oe < best_e || (oe == best_e && od < best_d))) {
      best_e = oe;
      best_d = od;
    }
  }
  if (lane != 0) return;
  if (!ok) {
    target[r] = -1;
    branch[r] = SMETRIC_INVALID;
    return;
  }
  const int32_t prev = best_ci;
  const int32_t bal = (start + best_d) % I;
  const i128 bound2 = i128(2) * (i128(p.slo_b) + i128(p.slo_a) * L);
  const bool slack_inf = p.slack_den == 0;
  const i128 e_prev = est2(p, L, c[prev], q[prev]);
  const bool meets_prev = slack_inf || e_prev * p.slack_den <= i128(p.slack_num) * bound2;
  const bool none_meets = !slack_inf && best_e * p.slack_den > i128(p.slack_num) * bound2;
  const bool cached = i128(p.B) * c[prev] * p.hit_den > i128(p.hit_num) * hist;
  int32_t t;
  uint8_t br;
  if (tr == 0) {
    t = bal;
    br = SMETRIC_FIRST_TURN;
  } else if (!cached) {
    t = bal;
    br = SMETRIC_EVICTED;
  } else if (meets_prev) {
    t = prev;
    br = SMETRIC_STICK;
  } else if (none_meets) {
    t = prev;
    br = SMETRIC_LAST_RESORT;
  } else {
    t = bal;
    br = SMETRIC_MIGRATE;
  }
  target[r] = t;
  branch[r] = br;
}

// (score, rotation distance) minimum; d = INT_MAX marks "none yet"
struct MinSD {
  i128 s;
  int32_t d;
};
__device__ __forceinline__ void min_sd(MinSD &a, i128 s, int32_t d) {
  if (d != 0x7FFFFFFF && (a.d == 0x7FFFFFFF || s < a.s || (s == a.s && d < a.d))) {
    a.s = s;
    a.d = d;
  }
}

// Route under PD colocation (App. B pseudocode).  Same mapping as route_kernel; each lane
// also tests the TPOT filter of its instances and keeps two minima of the LMetric score
// est2 * n_run: over the instances that pass, and over all (used when none passes).
__global__ __launch_bounds__(64 * RW) void route_coloc_kernel(
    const int32_t *__restrict__ matched, int32_t n_req, int32_t I, const int32_t *__restrict__ prompt_len,
    const int32_t *__restrict__ hist_len, const int32_t *__restrict__ turn, const int64_t *__restrict__ q,
    const int64_t *__restrict__ slack, const int32_t *__restrict__ n_run, RouteParams p, uint64_t rr_base,
    int32_t *__restrict__ target, uint8_t *__restrict__ branch) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * RW + wave;
  if (r >= n_req) return;
  const int32_t *c = matched + int64_t(r) * I;
  const int64_t L = prompt_len[r];
  const int32_t hist = hist_len[r], tr = turn[r];
  bool ok = L >= 0 && L <= (int64_t(1) << 24) && hist >= 0 && tr >= 0;
  const int64_t max_c = ok ? L / p.B : -1;
  const int32_t start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));

  int32_t best_c = -1, best_ci = 0x7FFFFFFF;
  MinSD pass{0, 0x7FFFFFFF}, all{0, 0x7FFFFFFF};
  for (int32_t i = lane; i < I; i += 64) {
    const int32_t ci = c[i];
    const int64_t qi = q[i];
    const int32_t ni = n_run[i];
    if (ci < 0 || ci > max_c || qi < 0 || qi >= (int64_t(1) << 62) || ni < 0) ok = false;
    if (ci > best_c) {
      best_c = ci;
      best_ci = i;
    }
    const i128 cost = est2(p, L, ci, 0);
    const i128 sc = (cost + i128(2) * qi) * ni;
    const int32_t d = i >= start ? i - start : i - start + I;
    min_sd(all, sc, d);
    if (slack[i] >= NO_DECODE || cost <= i128(2) * slack[i]) min_sd(pass, sc, d);
  }
  ok = __ballot(!ok) == 0;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const int32_t oc = __shfl_xor(best_c, m, 64), oi = __shfl_xor(best_ci, m, 64);
    if (oc > best_c || (oc == best_c && oi < best_ci)) {
      best_c = oc;
      best_ci = oi;
    }
    min_sd(all, shfl_xor128(all.s, m), __shfl_xor(all.d, m, 64));
    min_sd(pass, shfl_xor128(pass.s, m), __shfl_xor(pass.d, m, 64));
  }
  if (lane != 0) return;
  if (!ok) {
    target[r] = -1;
    branch[r] = SMETRIC_INVALID;
    return;
  }
  const bool any_pass = pass.d != 0x7FFFFFFF;
  const int32_t prev = best_ci;
  const int32_t bal = (start + (any_pass ? pass.d : all.d)) % I;
  const i128 cost_prev = est2(p, L, c[prev], 0);
  const bool prev_in = !any_pass || slack[prev] >= NO_DECODE || cost_prev <= i128(2) * slack[prev];
  const i128 bound2 = i128(2) * (i128(p.slo_b) + i128(p.slo_a) * L);
  const bool meets_prev =
      p.slack_den == 0 || (cost_prev + i128(2) * q[prev]) * p.slack_den <= i128(p.slack_num) * bound2;
  const bool cached = i128(p.B) * c[prev] * p.hit_den > i128(p.hit_num) * hist;
  int32_t t = bal;
  uint8_t br;
  if (tr == 0) {
    br = SMETRIC_FIRST_TURN;
  } else if (!cached) {
    br = SMETRIC_EVICTED;
  } else if (!meets_prev) {
    br = SMETRIC_MIGRATE;
  } else if (!prev_in) {
    br = SMETRIC_MIGRATE_TPOT;
  } else {
    t = prev;
    br = SMETRIC_STICK;
  }
  target[r] = t;
  branch[r] = br;
}

int route_params(const smetric_params *params, int32_t n_req, int32_t n_instances, RouteParams &rp) {
  if (!params || n_req < 0 || n_instances < 1 || n_instances > 65536) return SMETRIC_EINVAL;
  const smetric_params &P = *params;
  const int64_t LIM = int64_t(1) << 32;
  if (P.c_lin < 0 || P.c_lin > LIM || P.c_att < 0 || P.c_att > LIM || P.slo_b < 0 || P.slo_b > LIM ||
      P.slo_a < 0 || P.slo_a > LIM || P.slack_num < 0 || P.slack_den < 0 || P.hit_num < 0 ||
      P.hit_den <= 0 || P.hit_num >= P.hit_den || P.block_size < 2 || P.block_size > 256 ||
      (P.block_size & 1))
    return SMETRIC_EINVAL;
  rp = RouteParams{P.c_lin, P.c_att, P.slo_b, P.slo_a, P.slack_num, P.slack_den, P.hit_num, P.hit_den,
                   P.block_size};
  return SMETRIC_OK;
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_route(const int32_t *matched, int32_t n_req, int32_t n_instances,
                             const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                             const int64_t *q, const smetric_params *params, uint64_t rr_base,
                             int32_t *target, uint8_t *branch, hipStream_t stream) {
  RouteParams rp;
  if (int rc = route_params(params, n_req, n_instances, rp)) return rc;
  if (n_req == 0) return SMETRIC_OK;
  if (!matched || !prompt_len || !hist_len || !turn || !q || !target || !branch) return SMETRIC_EINVAL;
  hipLaunchKernelGGL(route_kernel, dim3((n_req + RW - 1) / RW), dim3(64 * RW), 0, stream, matched, n_req,
                     n_instances, prompt_len, hist_len, turn, q, rp, rr_base, target, branch);
  return hip_rc(hipGetLastError());
}

extern "C" int smetric_route_coloc(const int32_t *matched, int32_t n_req, int32_t n_instances,
                                   const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                                   const int64_t *q, const int64_t *tpot_slack, const int32_t *n_running,
                                   const smetric_params *params, uint64_t rr_base, int32_t *target,
                                   uint8_t *branch, hipStream_t stream) {
  RouteParams rp;
  if (int rc = route_params(params, n_req, n_instances, rp)) return rc;
  if (n_req == 0) return SMETRIC_OK;
  if (!matched || !prompt_len || !hist_len || !turn || !q || !tpot_slack || !n_running || !target || !branch)
    return SMETRIC_EINVAL;
  hipLaunchKernelGGL(route_coloc_kernel, dim3((n_req + RW - 1) / RW), dim3(64 * RW), 0, stream, matched, n_req,
                     n_instances, prompt_len, hist_len, turn, q, tpot_slack, n_running, rp, rr_base, target,
                     branch);
  return hip_rc(hipGetLastError());
}
