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
// keeping (max c, lowest id, its est2) and (min est2, rotation distance); two butterfly
// reductions across the wavefront finish the argmax and the argmin; lane 0 decides.  The
// main rule's scan runs in double precision while that is exact (every score an integer
// below 2^51), which cuts the kernel's vector instructions by more than a third.
#include <mutex>

#include "common.h"

namespace smk {
namespace {

constexpr int RW = 4;  // waves per workgroup
constexpr int RU = 4;  // instances per lane whose loads a route kernel issues together
typedef __int128 i128;
constexpr int64_t NO_DECODE = int64_t(1) << 62;  // decode slack meaning "no live decode"

struct RouteParams {
  int64_t c_lin, c_att, slo_b, slo_a;
  int32_t slack_num, slack_den, hit_num, hit_den, B;
};

// 2 q + 2 x Eq. (1): for requests in domain n = L - B c and L are at most 2^24, so
// 2 C_LIN n < 2^58 and n (2L - n) < 2^49 fit 64 bits, and the only wide product is
// C_ATT x n (2L - n) (64 x 64 -> 128 bits).
__device__ __forceinline__ i128 est2(const RouteParams &p, int64_t L, int32_t c, int64_t q) {
  const uint64_t n = uint64_t(L - int64_t(p.B) * c);
  const uint64_t w = n * (uint64_t(2 * L) - n);
  typedef unsigned __int128 u128_;
  return i128(2) * q + i128(uint64_t(2 * p.c_lin) * n) + i128(u128_(uint64_t(p.c_att)) * w);
}

__device__ __forceinline__ double shfl_xor_f64(double v, int m) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = uint32_t(__shfl_xor(int(uint32_t(b)), m, 64));
  const uint32_t hi = uint32_t(__shfl_xor(int(uint32_t(b >> 32)), m, 64));
  return __builtin_bit_cast(double, (uint64_t(hi) << 32) | lo);
}

__device__ __forceinline__ i128 shfl_xor128(i128 v, int m) {
  const uint64_t lo = uint64_t(v), hi = uint64_t(v >> 64);
  const uint64_t lo2 = (uint64_t(uint32_t(__shfl_xor(int(lo >> 32), m, 64))) << 32) |
                       uint32_t(__shfl_xor(int(uint32_t(lo)), m, 64));
  const uint64_t hi2 = (uint64_t(uint32_t(__shfl_xor(int(hi >> 32), m, 64))) << 32) |
                       uint32_t(__shfl_xor(int(uint32_t(hi)), m, 64));
  return (i128(hi2) << 64) | i128(lo2);
}

// RULE 0: SMetric (Sec. 4.2).  RULE 1: the Sec. 5.4 ablation's load-aware filter -- a
// cached follow-up sticks unless prev's load exceeds the mean by the margin m_num/m_den:
// load[prev] * I * m_den > (sum of loads) * (m_den + m_num); m_den == 0: never leaves.
template <int RULE>
__global__ __launch_bounds__(64 * RW) void route_kernel(const int32_t *__restrict__ matched,
                                                        int32_t n_req, int32_t I,
                                                        const int32_t *__restrict__ prompt_len,
                                                        const int32_t *__restrict__ hist_len,
                                                        const int32_t *__restrict__ turn,
                                                        const int64_t *__restrict__ q,
                                                        RouteParams p, uint64_t rr_base,
                                                        int32_t *__restrict__ target,
                                                        uint8_t *__restrict__ branch,
                                                        const int64_t *__restrict__ load = nullptr,
                                                        int32_t m_num = 0, int32_t m_den = 0) {
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
  i128 prev_e = 0;                            // est2 of that instance
  i128 best_e = 0;
  int32_t best_d = 0x7FFFFFFF;                // argmin (est2, rotation distance)
  i128 load_sum = 0;                          // RULE 1
  // Fast scan, exact in doubles: with n = L - B c, est2 = 2q + C0 - c (a1 + a2 c) where
  // C0 = 2 C_LIN L + C_ATT L^2, a1 = 2 C_LIN B and a2 = C_ATT B^2 (at most 2^41 and 2^48 for
  // parameters in range).  While C0 and every 2q stay below 2^50, each in-domain score is an
  // integer below 2^51 (and c (a1 + a2 c) <= C0), so two fused multiply-adds give it
  // exactly and doubles compare it exactly.  A wavefront that meets a larger queue scans
  // again in 128 bits.
  const i128 c0 = i128(2) * p.c_lin * L + i128(p.c_att) * L * L;
  bool fast = RULE == 0 && ok && c0 < (i128(1) << 50);
  if (fast) {
    const double a1 = double(2 * p.c_lin * p.B), a2 = double(p.c_att * p.B * p.B), c0d = double(int64_t(c0));
    double bs = 0.0, ps = 0.0;
    bool small = true;
    for (int32_t i0 = lane; i0 < I; i0 += 64 * RU) {
      int32_t cv[RU];
      int64_t qv[RU];
#pragma unroll
      for (int u = 0; u < RU; ++u) {
        const int32_t ii = i0 + 64 * u < I ? i0 + 64 * u : I - 1;
        cv[u] = c[ii];
        qv[u] = q[ii];
      }
#pragma unroll
      for (int u = 0; u < RU; ++u) {
        const int32_t i = i0 + 64 * u;
        if (i >= I) break;
        const int32_t ci = cv[u];
        const int64_t qi = qv[u];
        if (ci < 0 || ci > max_c || qi < 0 || qi >= (int64_t(1) << 62)) ok = false;
        small = small && uint64_t(qi) < (uint64_t(1) << 49);
        const double cd = double(ci);
        const double sc = __builtin_fma(-cd, __builtin_fma(a2, cd, a1), c0d + 2.0 * double(qi));
        if (ci > best_c) {
          best_c = ci;
          best_ci = i;
          ps = sc;
        }
        const int32_t d = i >= start ? i - start : i - start + I;
        if (best_d == 0x7FFFFFFF || sc < bs || (sc == bs && d < best_d)) {
          bs = sc;
          best_d = d;
        }
      }
    }
    fast = __ballot(!small) == 0;
    if (fast) {
      ok = __ballot(!ok) == 0;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        const int32_t oc = __shfl_xor(best_c, m, 64), oi = __shfl_xor(best_ci, m, 64);
        const double ops = shfl_xor_f64(ps, m), obs = shfl_xor_f64(bs, m);
        const int32_t od = __shfl_xor(best_d, m, 64);
        if (oc > best_c || (oc == best_c && oi < best_ci)) {
          best_c = oc;
          best_ci = oi;
          ps = ops;
        }
        if (od != 0x7FFFFFFF && (best_d == 0x7FFFFFFF || obs < bs || (obs == bs && od < best_d))) {
          bs = obs;
          best_d = od;
        }
      }
      prev_e = i128(int64_t(ps));
      best_e = i128(int64_t(bs));
    } else {  // back to the 128-bit scan from the start
      ok = L >= 0 && L <= (int64_t(1) << 24) && hist >= 0 && tr >= 0;
      best_c = -1;
      best_ci = 0x7FFFFFFF;
      best_d = 0x7FFFFFFF;
    }
  }
  // RU instances per lane at a time, their loads issued first (clamped, so branch-free)
  for (int32_t i0 = lane; !fast && i0 < I; i0 += 64 * RU) {
    int32_t cv[RU];
    int64_t qv[RU], lv[RU];
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int32_t ii = i0 + 64 * u < I ? i0 + 64 * u : I - 1;
      cv[u] = c[ii];
      qv[u] = q[ii];
      lv[u] = RULE == 1 ? load[ii] : 0;
    }
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int32_t i = i0 + 64 * u;
      if (i >= I) break;
      const int32_t ci = cv[u];
      const int64_t qi = qv[u];
      if (ci < 0 || ci > max_c || qi < 0 || qi >= (int64_t(1) << 62)) ok = false;
      if (RULE == 1) {
        const int64_t li = lv[u];
        if (li < 0 || li >= (int64_t(1) << 62)) ok = false;
        load_sum += li;
      }
      const i128 e = est2(p, L, ci, qi);
      if (ci > best_c) {
        best_c = ci;
        best_ci = i;
        prev_e = e;
      }
      const int32_t d = i >= start ? i - start : i - start + I;
      if (best_d == 0x7FFFFFFF || e < best_e || (e == best_e && d < best_d)) {
        best_e = e;
        best_d = d;
      }
    }
  }
  if (!fast) ok = __ballot(!ok) == 0;
#pragma unroll
  for (int m = 32; m >= 1 && !fast; m >>= 1) {
    const int32_t oc = __shfl_xor(best_c, m, 64), oi = __shfl_xor(best_ci, m, 64);
    const i128 ope = shfl_xor128(prev_e, m);
    if (oc > best_c || (oc == best_c && oi < best_ci)) {
      best_c = oc;
      best_ci = oi;
      prev_e = ope;
    }
    const i128 oe = shfl_xor128(best_e, m);
    const int32_t od = __shfl_xor(best_d, m, 64);
    if (od != 0x7FFFFFFF && (best_d == 0x7FFFFFFF || oe < best_e || (oe == best_e && od < best_d))) {
      best_e = oe;
      best_d = od;
    }
    if (RULE == 1) load_sum += shfl_xor128(load_sum, m);
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
  const bool meets_prev = slack_inf || prev_e * p.slack_den <= i128(p.slack_num) * bound2;
  const bool none_meets = !slack_inf && best_e * p.slack_den > i128(p.slack_num) * bound2;
  const bool cached = i128(p.B) * best_c * p.hit_den > i128(p.hit_num) * hist;
  int32_t t;
  uint8_t br;
  if (RULE == 1) {
    const bool over = m_den != 0 && i128(load[prev]) * I * m_den > load_sum * (i128(m_den) + m_num);
    t = (tr != 0 && cached && !over) ? prev : bal;
    br = tr == 0 ? SMETRIC_FIRST_TURN : !cached ? SMETRIC_EVICTED : !over ? SMETRIC_STICK : SMETRIC_MIGRATE;
    target[r] = t;
    branch[r] = br;
    return;
  }
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
  for (int32_t i0 = lane; i0 < I; i0 += 64 * RU) {  // loads first, as in route_kernel
    int32_t cv[RU], nv[RU];
    int64_t qv[RU], sv[RU];
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int32_t ii = i0 + 64 * u < I ? i0 + 64 * u : I - 1;
      cv[u] = c[ii];
      qv[u] = q[ii];
      nv[u] = n_run[ii];
      sv[u] = slack[ii];
    }
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int32_t i = i0 + 64 * u;
      if (i >= I) break;
      const int32_t ci = cv[u], ni = nv[u];
      const int64_t qi = qv[u];
      if (ci < 0 || ci > max_c || qi < 0 || qi >= (int64_t(1) << 62) || ni < 0) ok = false;
      if (ci > best_c) {
        best_c = ci;
        best_ci = i;
      }
      const i128 cost = est2(p, L, ci, 0);
      const i128 sc = (cost + i128(2) * qi) * ni;
      const int32_t d = i >= start ? i - start : i - start + I;
      min_sd(all, sc, d);
      if (sv[u] >= NO_DECODE || cost <= i128(2) * sv[u]) min_sd(pass, sc, d);
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

// ---------------------------------------------------------------------------------
// Online load update (Sec. 4.2 (a): q is what is queued when each request is routed).
//   prep  one wavefront per request, in parallel: what does not depend on the running
//         loads -- domain check, prev = argmax c, session_cached, the costs on prev and at
//         the best other hit, the deadline, and the smallest other est2 on the starting
//         loads -- into an 80-byte record.
//   seq   ONE wavefront routes the batch in index order; the running loads 2q[i] live in
//         LDS as 128-bit integers (and as doubles, exact while they stay below 2^50),
//         with a lower bound of their minimum.  Per request:
//           * cached follow-up whose prev meets its deadline: stick (no scan);
//           * cached follow-up for which min(2q) + cost(best other hit), or the smallest
//             other est2 on the starting loads, is past the deadline: no instance can meet
//             it, last-resort stick (no scan);
//           * otherwise the row is scanned for the argmin with the current loads (in
//             double precision while every score is an integer below 2^51, else in 128
//             bits).
//         The first two need only prev's load, so 64 requests are settled per step (see
//         route_seq_kernel); the rest go one at a time, their rows (for <= 1024 instances)
//         and records loaded into registers ahead of use.
// ---------------------------------------------------------------------------------
constexpr int SEQ_MAX_I = 4096;  // LDS: the loads (64 KB), as doubles (32 KB), step counters (16 KB)

struct SeqRec {
  int32_t prev;    // argmax c, lowest id
  int32_t flags;   // bit 0: in domain (apart from q), bit 1: session cached, bit 2: follow-up
  int32_t L;       // prompt length
  int32_t start;   // (rr_base + r) mod I: where the rotation of rr_argmin starts
  i128 cost_prev;  // 2 x prefill_cost(req, c[prev]), Eq. (1)
  i128 cost_rest;  // 2 x prefill_cost at the largest hit of any other instance: a lower
                   // bound of every other instance's cost (Eq. (1) falls as the hit grows)
  i128 bound;      // SLACK_num x 2 (b + a L): i meets its deadline iff est2(i) SLACK_den <= bound
  i128 m0;         // min over i != prev of est2(i) on the loads the batch starts with: a lower
                   // bound of every other instance's est2 at any later point (loads only grow)
};
constexpr int64_t SEQ_NO_OTHER = int64_t(1) << 60;  // m0 with no other instance (x 2^30: never meets)

__global__ __launch_bounds__(64 * RW) void route_seq_prep_kernel(const int32_t *__restrict__ matched, int32_t n_req,
                                                                 int32_t I, const int32_t *__restrict__ prompt_len,
                                                                 const int32_t *__restrict__ hist_len,
                                                                 const int32_t *__restrict__ turn,
                                                                 const int64_t *__restrict__ q, RouteParams p,
                                                                 uint64_t rr_base, SeqRec *__restrict__ rec) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * RW + wave;
  if (r >= n_req) return;
  const int32_t *c = matched + int64_t(r) * I;
  const int64_t L = prompt_len[r];
  const int32_t hist = hist_len[r], tr = turn[r];
  bool ok = L >= 0 && L <= (int64_t(1) << 24) && hist >= 0 && tr >= 0;
  const int64_t max_c = ok ? L / p.B : -1;
  int32_t bc = -1, bi = 0x7FFFFFFF;
  for (int32_t i = lane; i < I; i += 64) {
    const int32_t ci = c[i];
    if (ci < 0 || ci > max_c) ok = false;
    if (ci > bc) {
      bc = ci;
      bi = i;
    }
  }
  ok = __ballot(!ok) == 0;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const int32_t oc = __shfl_xor(bc, m, 64), oi = __shfl_xor(bi, m, 64);
    if (oc > bc || (oc == bc && oi < bi)) {
      bc = oc;
      bi = oi;
    }
  }
  // the largest hit of any instance but prev (none: no other instance)
  int32_t c2 = -1;
  for (int32_t i = lane; i < I; i += 64)
    if (i != bi) c2 = c[i] > c2 ? c[i] : c2;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const int32_t o = __shfl_xor(c2, m, 64);
    c2 = o > c2 ? o : c2;
  }
  // the smallest est2 of any other instance on the starting loads (the row is in range
  // whenever ok; a load outside [0, 2^62) makes the whole batch invalid later)
  i128 m0 = i128(SEQ_NO_OTHER) << 30;
  if (ok)
    for (int32_t i = lane; i < I; i += 64)
      if (i != bi) {
        const int64_t qi = q[i];
        const i128 e = est2(p, L, c[i], qi < 0 || qi >= (int64_t(1) << 62) ? 0 : qi);
        m0 = e < m0 ? e : m0;
      }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const i128 o = shfl_xor128(m0, m);
    m0 = o < m0 ? o : m0;
  }
  if (lane != 0) return;
  const bool cached = ok && i128(p.B) * bc * p.hit_den > i128(p.hit_num) * hist;
  SeqRec out;
  out.prev = ok ? bi : 0;
  out.flags = int32_t(ok) | (int32_t(cached) << 1) | (int32_t(tr != 0) << 2);
  out.L = ok ? int32_t(L) : 0;
  out.start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));
  out.cost_prev = ok ? est2(p, L, bc, 0) : i128(0);
  // one instance: nothing else to bound, any value will do
  out.cost_rest = ok ? est2(p, L, c2 < 0 ? bc : c2, 0) : i128(0);
  out.bound = i128(p.slack_num) * (i128(2) * (i128(p.slo_b) + i128(p.slo_a) * (ok ? L : 0)));
  out.m0 = m0;
  rec[r] = out;
}

template <int K>
struct SeqRow {
  int32_t v[K];  // c[r][lane + 64 k] (K = 0: read on demand)
  SeqRec rec;
};

template <int K>
__device__ __forceinline__ void seq_load(const int32_t *__restrict__ matched, int32_t I, int32_t r, int32_t n_req,
                                         const SeqRec *__restrict__ recs, SeqRow<K> &row) {
  // Unconditional, clamped loads keep this straight-line code, so the compiler can wait
  // for exactly the loads a request needs; lanes past the last instance are never read.
  const int lane = threadIdx.x;
  const int32_t rr = r < n_req ? r : n_req - 1;
  const int32_t *c = matched + int64_t(rr) * I;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int i = lane + 64 * k;
    row.v[k] = c[i < I ? i : I - 1];
  }
  // Vector loads on purpose: as scalar loads (the index is uniform) they would complete
  // out of order, and every later wait on LDS or on the current request's scalars would
  // also wait for these prefetches.
  int32_t rv = rr;
  asm volatile("" : "+v"(rv));
  row.rec = recs[rv];
}

// Minimum of the running loads (every lane gets it).
__device__ __forceinline__ i128 seq_qmin(const i128 *q2, int32_t I) {
  i128 m = q2[0];
  for (int32_t i = threadIdx.x; i < I; i += 64) m = q2[i] < m ? q2[i] : m;
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) {
    const i128 o = shfl_xor128(m, s);
    m = o < m ? o : m;
  }
  return m;
}

__device__ __forceinline__ int32_t uni(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// readlane returns int: each word goes through uint32_t, or a set bit 31 of a low word
// would sign-extend into the word above it
__device__ __forceinline__ i128 readlane128(i128 v, int l) {
  const uint64_t lo = uint64_t(v), hi = uint64_t(v >> 64);
  const uint32_t w0 = uint32_t(__builtin_amdgcn_readlane(uint32_t(lo), l));
  const uint32_t w1 = uint32_t(__builtin_amdgcn_readlane(uint32_t(lo >> 32), l));
  const uint32_t w2 = uint32_t(__builtin_amdgcn_readlane(uint32_t(hi), l));
  const uint32_t w3 = uint32_t(__builtin_amdgcn_readlane(uint32_t(hi >> 32), l));
  return (i128((uint64_t(w3) << 32) | w2) << 64) | i128((uint64_t(w1) << 32) | w0);
}

// Minimum of a 32-bit value over the wavefront by DPP moves toward lane 63 (lanes without a
// source, or outside the row mask, take all ones: the identity of the minimum, which lets
// the move fold into the minimum's DPP form); every lane gets it.
template <int CTRL, int RM>
__device__ __forceinline__ uint32_t dpp_min_u32(uint32_t k) {
  const uint32_t o = uint32_t(__builtin_amdgcn_update_dpp(-1, int(k), CTRL, RM, 0xF, false));
  return o < k ? o : k;
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t k) {
  k = dpp_min_u32<0x111, 0xF>(k);
  k = dpp_min_u32<0x112, 0xF>(k);
  k = dpp_min_u32<0x114, 0xF>(k);
  k = dpp_min_u32<0x118, 0xF>(k);
  k = dpp_min_u32<0x142, 0xA>(k);  // row_bcast:15 into rows 1 and 3
  k = dpp_min_u32<0x143, 0xC>(k);  // row_bcast:31 into rows 2 and 3
  return uint32_t(__builtin_amdgcn_readlane(int(k), 63));
}
// Minimum of a 64-bit key over the wavefront: the smallest high word, then the smallest low
// word among the lanes holding it; every lane gets it.
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t k) {
  const uint32_t hi = wave_min_u32(uint32_t(k >> 32));
  const uint32_t lo = wave_min_u32(uint32_t(k >> 32) == hi ? uint32_t(k) : ~0u);
  return (uint64_t(hi) << 32) | lo;
}

// The running state of the online route, held by its one wavefront (all fields uniform but
// the LDS arrays).  Besides the exact loads 2q it keeps them as doubles for the scan's fast
// path: exact while q_small (every 2q below 2^50), which stops holding for good once any
// load reaches it.  With a1 = 2 C_LIN B and a2 = C_ATT B^2, Eq. (1) doubled is
// est2(c) = C0 - c (a1 + a2 c) on the request's domain 0 <= c <= L / B, C0 = est2(0).
constexpr double SEQ_PAD_2Q = 3377699720527872.0;  // 3 x 2^50

struct SeqState {
  i128 *q2;      // LDS: 2q per instance (exact)
  double *q2d;   // LDS: the same values as doubles (exact while q_small)
  i128 qmin;     // a lower bound of min(2q), exact unless qmin_stale
  bool qmin_stale;
  bool q_small;  // every 2q < 2^50
  bool a_ok;     // a1, a2 < 2^53: exact as doubles
  double a1, a2;
};

// The last-resort test of a cached follow-up whose prev misses its deadline: every other
// instance i has est2(i) >= min(2q) + cost_rest and est2(i) >= m0, so if either misses the
// deadline nobody can meet it.  qmin is a lower bound of min(2q) (loads only grow), exact
// unless qmin_stale; a stale bound that does not settle the test is refreshed first, so the
// minimum is recomputed only when a request needs it.
__device__ __forceinline__ bool seq_none_meets(const SeqRec &rec, const RouteParams &p, int32_t I, SeqState &st) {
  const i128 bound = rec.bound;
  if (uni(int32_t(rec.m0 * p.slack_den > bound || (st.qmin + rec.cost_rest) * p.slack_den > bound)) != 0) return true;
  if (!st.qmin_stale) return false;
  st.qmin = seq_qmin(st.q2, I);
  st.qmin_stale = false;
  return uni(int32_t((st.qmin + rec.cost_rest) * p.slack_den > bound)) != 0;
}

// A load update: the exact value, its double, and whether the doubles stay exact.
__device__ __forceinline__ void seq_store(SeqState &st, int32_t i, i128 v) {
  st.q2[i] = v;
  st.q2d[i] = double(int64_t(v < (i128(1) << 62) ? v : i128(0)));
}

// Decide request r.  Every branch below is on wavefront-uniform values (read with
// readfirstlane), and every lane performs the identical stores, so the code has no divergent
// regions: the compiler can then wait for exactly the prefetched loads it uses.
template <int K>
__device__ __forceinline__ void seq_decide(const SeqRow<K> &row, const int32_t *__restrict__ matched, int32_t r,
                                           int32_t I, const RouteParams &p, bool q_ok, SeqState &st,
                                           int32_t *__restrict__ target, uint8_t *__restrict__ branch) {
  const int lane = threadIdx.x;
  const int32_t flags = uni(row.rec.flags);
  if (!q_ok || !(flags & 1)) {
    target[r] = -1;
    branch[r] = SMETRIC_INVALID;
    return;
  }
  const int32_t prev = uni(row.rec.prev);
  const bool cached = flags & 2, follow_up = flags & 4;
  const bool slack_inf = p.slack_den == 0;
  const i128 cost_prev = row.rec.cost_prev, bound = row.rec.bound;  // uniform across lanes
  i128 *q2 = st.q2;
  const bool meets_prev =
      follow_up && cached && (slack_inf || uni(int32_t((q2[prev] + cost_prev) * p.slack_den <= bound)) != 0);
  int32_t t;
  uint8_t br;
  i128 cost_t;
  if (follow_up && cached && meets_prev) {
    t = prev;
    br = SMETRIC_STICK;
    cost_t = cost_prev;
  } else if (follow_up && cached && !slack_inf && seq_none_meets(row.rec, p, I, st)) {
    // prev misses its deadline, and every other instance i has est2(i) >= min(2q) +
    // cost_rest and est2(i) >= m0: nobody can meet it
    t = prev;
    br = SMETRIC_LAST_RESORT;
    cost_t = cost_prev;
  } else {
    const int64_t L = uni(row.rec.L);
    const int32_t tr = follow_up ? 1 : 0;
    const int32_t start = uni(row.rec.start);
    const int32_t *c = matched + int64_t(r) * I;
    MinSD best{0, 0x7FFFFFFF};
    // Fast path, while every 2q < 2^50 and C0 < 2^50: each candidate's score
    // 2q + est2 = 2q + C0 - c (a1 + a2 c) is an integer below 2^51, and two fused
    // multiply-adds in double precision give it exactly, offset by 2^52 so that its bit
    // pattern holds the score in the low 52 bits under a fixed exponent field.  Shifting the
    // exponent out leaves room for the rotation distance (I <= 4096): one 64-bit key per
    // instance, minimised with two 32-bit DPP minima.
    bool fast = false;
    if (st.q_small && st.a_ok) {
      const i128 c0 = est2(p, L, 0, 0);
      if (c0 < (i128(1) << 50)) {
        fast = true;
        const double off = double(int64_t(c0)) + 4503599627370496.0;  // C0 + 2^52, exact
        const double a1 = st.a1, a2 = st.a2;
        const double *q2d = st.q2d;
        uint64_t kmin = ~uint64_t(0);
        int32_t d = lane >= start ? lane - start : lane - start + I;  // rotation distance of i
        auto scan_one = [&](int32_t ci, double q2i) {
          const double cd = double(ci);
          const double s2 = __builtin_fma(-cd, __builtin_fma(a2, cd, a1), q2i + off);
          const uint64_t key = (__builtin_bit_cast(uint64_t, s2) << 12) | uint32_t(d);
          kmin = key < kmin ? key : kmin;
        };
        if (K > 0) {
          // Slots past the last instance hold 2q = 3 x 2^50 (SEQ_PAD_2Q): their scores fall
          // in [2^51, 2^52) under the same exponent, above every real one, so the loop has
          // no per-lane conditions and all its LDS reads go out before the first is used.
          double qv[K > 0 ? K : 1];
#pragma unroll
          for (int k = 0; k < (K > 0 ? K : 1); ++k) qv[k] = q2d[lane + 64 * k];
#pragma unroll
          for (int k = 0; k < (K > 0 ? K : 1); ++k) {
            scan_one(row.v[k], qv[k]);
            d = d + 64 >= I ? d + 64 - I : d + 64;  // I > 64 whenever K > 1
          }
        } else {
          for (int32_t i = lane; i < I; i += 64) {
            scan_one(c[i], q2d[i]);
            d = d + 64 >= I ? d + 64 - I : d + 64;
          }
        }
        const uint64_t m = wave_min_u64(kmin);
        best.s = i128(m >> 12);
        best.d = int32_t(m & 4095u);
      }
    }
    if (!fast) {
      if (K > 0) {
#pragma unroll
        for (int k = 0; k < (K > 0 ? K : 1); ++k) {
          const int32_t i = lane + 64 * k;
          const int32_t ii = i < I ? i : I - 1;
          const i128 e = q2[ii] + est2(p, L, row.v[k], 0);
          min_sd(best, e, i < I ? (i >= start ? i - start : i - start + I) : 0x7FFFFFFF);
        }
      } else {
        for (int32_t i = lane; i < I; i += 64)
          min_sd(best, q2[i] + est2(p, L, c[i], 0), i >= start ? i - start : i - start + I);
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) min_sd(best, shfl_xor128(best.s, m), __shfl_xor(best.d, m, 64));
    }
    const int32_t bal0 = start + uni(best.d);  // start, d < I
    const int32_t bal = bal0 >= I ? bal0 - I : bal0;
    if (tr == 0) {
      t = bal;
      br = SMETRIC_FIRST_TURN;
    } else if (!cached) {
      t = bal;
      br = SMETRIC_EVICTED;
    } else if (!slack_inf && uni(int32_t(best.s * p.slack_den > bound)) != 0) {
      t = prev;
      br = SMETRIC_LAST_RESORT;
    } else {
      t = bal;
      br = SMETRIC_MIGRATE;
    }
    int32_t ct;
    if (K > 0) {
      int32_t v = 0;
#pragma unroll
      for (int k = 0; k < (K > 0 ? K : 1); ++k)
        if (k == t / 64) v = row.v[k];
      ct = uni(__shfl(v, t % 64, 64));
    } else {
      ct = uni(c[t]);
    }
    cost_t = t == prev ? cost_prev : est2(p, L, ct, 0);
  }
  // One wavefront does every LDS access, and its LDS operations complete in program
  // order, so the next request reads this update without a fence (a fence here would also
  // wait for the rows prefetched for later requests).  All lanes store the same values.
  const i128 old = q2[t];
  target[r] = t;
  branch[r] = br;
  seq_store(st, t, old + cost_t);  // the request's prefill joins its target's queue
  // both flags stay wavefront-uniform (every lane holds the same values): read as scalars
  st.q_small = st.q_small && uni(int32_t(old + cost_t < (i128(1) << 50))) != 0;
  if (uni(int32_t(old == st.qmin && cost_t != 0)) != 0) st.qmin_stale = true;
}

// Requests [rs, re) one at a time, rows and records prefetched D requests ahead.
template <int K, int D>
__device__ __forceinline__ void seq_exact_block(const int32_t *__restrict__ matched, int32_t n_req, int32_t I,
                                                const RouteParams &p, bool q_ok,
                                                const SeqRec *__restrict__ recs, SeqState &st,
                                                int32_t *__restrict__ target, uint8_t *__restrict__ branch,
                                                int32_t rs, int32_t re) {
  SeqRow<K> ring[D];
#pragma unroll
  for (int d = 0; d < D; ++d) seq_load<K>(matched, I, rs + d, n_req, recs, ring[d]);
  for (int32_t r0 = rs; r0 < re; r0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int32_t r = r0 + d;
      if (r < re) {
        seq_decide<K>(ring[d], matched, r, I, p, q_ok, st, target, branch);
        seq_load<K>(matched, I, r + D, n_req, recs, ring[d]);
      }
    }
  }
}

// The batch in blocks of 64 requests, one per lane.  A cached follow-up puts its prefill on
// prev whether it sticks or takes the last resort, so -- if every earlier request of the
// block is decided that way -- request l's load on prev is exactly q2[prev] plus the costs
// of the earlier requests with the same prev.  With that load, "prev meets its deadline"
// (stick) is exact, and "min(2q) + cost_rest misses it" (last resort) is exact with any
// lower bound of min(2q), which only grows; out-of-domain requests change nothing.  The
// requests before the first one not settled this way are decided together, that one
// alone with the sequential rule, and the next block starts after it.  After two blocks in
// a row that settle nothing (e.g. first turns, which always need a scan), the next 64
// requests go through the sequential rule with prefetching.
template <int K, int D>
__global__ __launch_bounds__(64) void route_seq_kernel(const int32_t *__restrict__ matched, int32_t n_req,
                                                       int32_t I, const int64_t *__restrict__ q, RouteParams p,
                                                       const SeqRec *__restrict__ recs,
                                                       int32_t *__restrict__ target, uint8_t *__restrict__ branch,
                                                       int64_t *__restrict__ q_out) {
  __shared__ i128 q2[SEQ_MAX_I];
  __shared__ double q2d[SEQ_MAX_I];
  __shared__ uint32_t n_on[SEQ_MAX_I];  // block requests per prev (0 between blocks)
  const int lane = threadIdx.x;
  bool q_ok = true, small = true;
  for (int32_t i = lane; i < I; i += 64) {
    const int64_t qi = q[i];
    if (qi < 0 || qi >= (int64_t(1) << 62)) q_ok = false;
    if (qi >= (int64_t(1) << 49)) small = false;
    q2[i] = i128(2) * qi;
    q2d[i] = 2.0 * double(qi < 0 ? 0 : qi);
    n_on[i] = 0;
  }
  for (int32_t i = I + lane; i < 64 * K; i += 64) q2d[i] = SEQ_PAD_2Q;
  q_ok = __ballot(!q_ok) == 0;
  __syncthreads();
  SeqState st;
  st.q2 = q2;
  st.q2d = q2d;
  st.qmin = seq_qmin(q2, I);  // a lower bound of min(2q) from here on (loads only grow)
  st.qmin_stale = false;
  st.q_small = __ballot(!small) == 0;
  const i128 a1 = i128(2) * p.c_lin * p.B, a2 = i128(p.c_att) * p.B * p.B;
  st.a_ok = a1 < (i128(1) << 53) && a2 < (i128(1) << 53);
  st.a1 = double(int64_t(st.a_ok ? a1 : 0));
  st.a2 = double(int64_t(st.a_ok ? a2 : 0));
  const bool slack_inf = p.slack_den == 0;
  int32_t r0 = 0;
  int streak = 0;
  while (r0 < n_req) {
    if (streak >= 2) {
      const int32_t re = n_req - r0 < 64 ? n_req : r0 + 64;
      seq_exact_block<K, D>(matched, n_req, I, p, q_ok, recs, st, target, branch, r0, re);
      r0 = re;
      streak = 0;
      continue;
    }
    const int32_t nv = n_req - r0 < 64 ? n_req - r0 : 64;
    const int32_t r = r0 + lane;
    int32_t rv = r < n_req ? r : n_req - 1;
    asm volatile("" : "+v"(rv));  // a vector load: see seq_load
    const SeqRec rec = recs[rv];
    const bool in = lane < nv;
    const bool ok = q_ok && (rec.flags & 1);
    const bool sticky = ok && (rec.flags & 2) && (rec.flags & 4);  // cached follow-up: its prefill goes to prev
    const int32_t prev = rec.prev;
    const bool mine = in && sticky;
    if (mine) atomicAdd(&n_on[prev], 1u);
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    // requests sharing a prev within the block form a group (lanes in index order): each
    // adds the costs of the group's earlier requests to its load on prev
    uint64_t todo = __ballot(mine && n_on[prev] > 1);
    __builtin_amdgcn_wave_barrier();
    if (mine) n_on[prev] = 0;
    i128 excl = 0;
    uint64_t group = 0;  // lanes with my prev (0: nobody else has it)
    while (todo) {
      const int32_t p0 = __builtin_amdgcn_readlane(prev, __builtin_ctzll(todo));
      const uint64_t m = __ballot(mine && prev == p0);
      todo &= ~m;
      i128 run = 0;
      for (uint64_t mm = m; mm; mm &= mm - 1) {
        const int l = __builtin_ctzll(mm);
        if (lane == l) {
          excl = run;
          group = m;
        }
        run += readlane128(rec.cost_prev, l);
      }
    }
    const i128 q_pre = mine ? q2[prev] : i128(0);
    const i128 q_prev = q_pre + excl;
    bool settled = !ok;  // out of domain: settled, nothing queued
    uint8_t br = SMETRIC_INVALID;
    const bool stick = sticky && (slack_inf || (q_prev + rec.cost_prev) * p.slack_den <= rec.bound);
    bool none = sticky && !stick &&
                ((st.qmin + rec.cost_rest) * p.slack_den > rec.bound || rec.m0 * p.slack_den > rec.bound);
    if (st.qmin_stale && __ballot(in && sticky && !stick && !none)) {  // a stale bound left one open
      st.qmin = seq_qmin(q2, I);
      st.qmin_stale = false;
      none = sticky && !stick && (st.qmin + rec.cost_rest) * p.slack_den > rec.bound;
      none |= sticky && !stick && rec.m0 * p.slack_den > rec.bound;
    }
    if (stick) {
      settled = true;
      br = SMETRIC_STICK;
    } else if (none) {
      settled = true;
      br = SMETRIC_LAST_RESORT;
    }
    const uint64_t open = __ballot(in && !settled);
    const int32_t f = open ? __builtin_ctzll(open) : nv;  // requests [r0, r0 + f) are decided
    // the first request not settled needs its row: requested now, used below
    SeqRow<K> row;
    if (f < nv) seq_load<K>(matched, I, r0 + f, n_req, recs, row);
    if (lane < f) {
      target[r] = ok ? prev : -1;
      branch[r] = br;
    }
    // prev's new load, written by the last of the decided requests with that prev
    const uint64_t decided = f >= 64 ? ~uint64_t(0) : (uint64_t(1) << f) - 1;
    const uint64_t after_me = lane == 63 ? uint64_t(0) : ~((uint64_t(2) << lane) - 1);
    const bool last = mine && lane < f && (group & after_me & decided) == 0;
    __builtin_amdgcn_wave_barrier();
    if (last) seq_store(st, prev, q_prev + rec.cost_prev);
    st.q_small = st.q_small && __ballot(last && q_prev + rec.cost_prev >= (i128(1) << 50)) == 0;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    // the minimum can only have moved if an instance at the minimum took load
    if (__ballot(mine && lane < f && q_pre == st.qmin)) st.qmin_stale = true;
    r0 += f;
    if (f < nv) {  // the first request not settled: the sequential rule
      seq_decide<K>(row, matched, r0, I, p, q_ok, st, target, branch);
      r0 += 1;
      streak = f == 0 ? streak + 1 : 0;
    }
  }
  __syncthreads();
  if (q_out)
    for (int32_t i = lane; i < I; i += 64) {
      const i128 v = q2[i] >> 1;
      q_out[i] = v > i128(INT64_MAX) ? INT64_MAX : int64_t(v);
    }
}

// ---------------------------------------------------------------------------------
// Online load update under PD colocation (App. B, whose req = receive() takes one request
// at a time).  The running state is the queued prefill 2q[i] and the request count n[i];
// each request is decided by the batch colocation rule on the state the earlier requests
// left, then its prefill joins the target's queue and it is one more request there.  The
// decode slacks are the caller's (the request's own decode is not live yet).
//   prep  one wavefront per request: domain, prev = argmax c, session_cached, follow-up,
//         whether prev is a candidate (passes the TPOT filter, or no instance does), the
//         cost on prev and the deadline -- none of it depends on the running state.
//   rank  per request, its best candidates on a state shortly before its decision (see
//         the speculative blocks below), many workgroups at once.
//   seq   ONE wavefront with 2q and n in LDS.  A cached follow-up whose prev is a
//         candidate sticks iff prev meets its deadline, which needs only prev's load: 64
//         requests are settled per step as in route_seq_kernel (the step's earlier
//         requests with the same prev add their costs); the first request not settled is
//         decided by rescoring its listed candidates on the current state.
//         The scores est2 x n are compared in 192 bits: over a batch both factors grow.
// ---------------------------------------------------------------------------------
typedef unsigned __int128 u128;
constexpr int SEQC_MAX_I = 4096;  // LDS: 2q (64 KB), n and the step counters (16 KB each)

struct SeqCRec {
  int32_t prev;
  int32_t flags;  // bit 0: in domain (apart from the instance state), 1: session cached,
                  // 2: follow-up, 3: prev is a candidate, 4: some instance passes the TPOT filter
  int32_t L;
  int32_t start;  // (rr_base + r) mod I
  i128 cost_prev;  // 2 x prefill_cost(req, c[prev])
  i128 thr;        // prev meets the deadline iff its doubled queue is at most thr
};

// floor(x / d) for 0 <= x < 2^128 and 0 < d < 2^32, by 32-bit digits
__device__ __forceinline__ u128 div128_u32(u128 x, uint32_t d) {
  u128 q = 0;
  uint64_t rem = 0;
#pragma unroll
  for (int k = 3; k >= 0; --k) {
    const uint64_t cur = (rem << 32) | uint32_t(x >> (32 * k));
    q |= u128(cur / d) << (32 * k);
    rem = cur % d;
  }
  return q;
}

__device__ __forceinline__ bool tpot_pass(int64_t slack, i128 cost2) {
  return slack >= NO_DECODE || cost2 <= i128(2) * slack;
}

__global__ __launch_bounds__(64 * RW) void route_seqc_prep_kernel(const int32_t *__restrict__ matched, int32_t n_req,
                                                                  int32_t I, const int32_t *__restrict__ prompt_len,
                                                                  const int32_t *__restrict__ hist_len,
                                                                  const int32_t *__restrict__ turn,
                                                                  const int64_t *__restrict__ slack, RouteParams p,
                                                                  uint64_t rr_base, SeqCRec *__restrict__ rec) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * RW + wave;
  if (r >= n_req) return;
  const int32_t *c = matched + int64_t(r) * I;
  const int64_t L = prompt_len[r];
  const int32_t hist = hist_len[r], tr = turn[r];
  bool ok = L >= 0 && L <= (int64_t(1) << 24) && hist >= 0 && tr >= 0;
  const int64_t max_c = ok ? L / p.B : -1;
  int32_t bc = -1, bi = 0x7FFFFFFF;
  bool any_pass = false;
  for (int32_t i = lane; i < I; i += 64) {
    const int32_t ci = c[i];
    if (ci < 0 || ci > max_c) ok = false;
    if (ci > bc) {
      bc = ci;
      bi = i;
    }
    if (ok && tpot_pass(slack[i], est2(p, L, ci, 0))) any_pass = true;
  }
  ok = __ballot(!ok) == 0;
  any_pass = __ballot(any_pass) != 0;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const int32_t oc = __shfl_xor(bc, m, 64), oi = __shfl_xor(bi, m, 64);
    if (oc > bc || (oc == bc && oi < bi)) {
      bc = oc;
      bi = oi;
    }
  }
  if (lane != 0) return;
  SeqCRec out;
  const i128 cost_prev = ok ? est2(p, L, bc, 0) : i128(0);
  const bool cached = ok && i128(p.B) * bc * p.hit_den > i128(p.hit_num) * hist;
  const bool prev_cand = ok && (!any_pass || tpot_pass(slack[bi], cost_prev));
  out.prev = ok ? bi : 0;
  out.flags = int32_t(ok) | (int32_t(cached) << 1) | (int32_t(tr != 0) << 2) | (int32_t(prev_cand) << 3) |
              (int32_t(any_pass) << 4);
  out.L = ok ? int32_t(L) : 0;
  out.start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));
  out.cost_prev = cost_prev;
  // (2q + cost_prev) x SLACK_den <= SLACK_num x 2 (b + a L), both sides integers and the
  // bound non-negative: 2q <= floor(bound / SLACK_den) - cost_prev; SLACK infinite: always
  const i128 bound = i128(p.slack_num) * (i128(2) * (i128(p.slo_b) + i128(p.slo_a) * (ok ? L : 0)));
  out.thr = p.slack_den == 0 ? (i128(1) << 126) : i128(div128_u32(u128(bound), uint32_t(p.slack_den))) - cost_prev;
  rec[r] = out;
}

// a * x for 0 <= a < 2^127, x < 2^32, as (high 128 bits, low 64 bits)
struct P192 {
  u128 hi;
  uint64_t lo;
};
__device__ __forceinline__ P192 mul192(i128 a, uint32_t x) {
  const u128 ua = u128(a);
  const uint64_t p0 = uint64_t(uint32_t(ua)) * x;                           // < 2^64
  const uint64_t p1 = uint64_t(uint32_t(uint64_t(ua) >> 32)) * x + (p0 >> 32);  // < 2^64
  const uint64_t lo = (p1 << 32) | uint32_t(p0);
  const uint64_t a_hi = uint64_t(ua >> 64);
  if (a_hi == 0) return P192{u128(p1 >> 32), lo};  // the usual case: a load below 2^64
  return P192{u128(a_hi) * x + (p1 >> 32), lo};
}
__device__ __forceinline__ bool less192(const P192 &a, const P192 &b) {
  return a.hi < b.hi || (a.hi == b.hi && a.lo < b.lo);
}
// (score, rotation distance) minimum with 192-bit scores; d = INT_MAX marks "none yet"
struct MinPD {
  P192 s;
  int32_t d;
};
__device__ __forceinline__ void min_pd(MinPD &a, const P192 &s, int32_t d) {
  if (d != 0x7FFFFFFF && (a.d == 0x7FFFFFFF || less192(s, a.s) || (!less192(a.s, s) && d < a.d))) {
    a.s = s;
    a.d = d;
  }
}
__device__ __forceinline__ void min_pd_xor(MinPD &a, int m) {
  P192 o;
  o.hi = u128(shfl_xor128(i128(a.s.hi), m));
  o.lo = (uint64_t(uint32_t(__shfl_xor(int(a.s.lo >> 32), m, 64))) << 32) |
         uint32_t(__shfl_xor(int(uint32_t(a.s.lo)), m, 64));
  min_pd(a, o, __shfl_xor(a.d, m, 64));
}

// DPP move of a 64-bit value from lane l - s of the same row (row_shr:s) or from the last lane
// of an earlier row (row_bcast); lanes without a source, or outside the row mask, keep v.
template <int CTRL, int RM>
__device__ __forceinline__ uint64_t dpp_or_own64(uint64_t v) {
  const int lo = __builtin_amdgcn_update_dpp(int(uint32_t(v)), int(uint32_t(v)), CTRL, RM, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(int(uint32_t(v >> 32)), int(uint32_t(v >> 32)), CTRL, RM, 0xF, false);
  return (uint64_t(uint32_t(hi)) << 32) | uint32_t(lo);
}
template <int CTRL, int RM>
__device__ __forceinline__ void dpp_min_key(uint64_t &k1, uint64_t &k0) {
  const uint64_t o1 = dpp_or_own64<CTRL, RM>(k1), o0 = dpp_or_own64<CTRL, RM>(k0);
  if (o1 < k1 || (o1 == k1 && o0 < k0)) {
    k1 = o1;
    k0 = o0;
  }
}
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  return (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v >> 32)), l))) << 32) |
         uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v)), l));
}

// Lexicographic minimum of (k1, k0) over lanes 0..N-1 (N = 64: the wavefront; N <= 16:
// within row 0) by DPP moves toward lane N - 1; every lane gets it.
template <int N>
__device__ __forceinline__ void wave_min_key(uint64_t &k1, uint64_t &k0) {
  if (N > 1) dpp_min_key<0x111, 0xF>(k1, k0);
  if (N > 2) dpp_min_key<0x112, 0xF>(k1, k0);
  if (N > 4) dpp_min_key<0x114, 0xF>(k1, k0);
  if (N > 8) dpp_min_key<0x118, 0xF>(k1, k0);
  if (N > 16) {
    dpp_min_key<0x142, 0xA>(k1, k0);  // row_bcast:15 into rows 1 and 3
    dpp_min_key<0x143, 0xC>(k1, k0);  // row_bcast:31 into rows 2 and 3
  }
  k1 = readlane64(k1, N - 1);
  k0 = readlane64(k0, N - 1);
}

// Minimum of (score, d) over lanes 0..N-1 (N = 64: the wavefront; N <= 16: within row 0);
// every lane gets it.  While every score is below 2^96 the pair is compared as two 64-bit
// words (score bits 32..95; score bits 0..31 and d) and reduced with DPP moves toward lane
// N - 1 (row_shr 1, 2, 4, 8, then row_bcast 15 and 31); otherwise with 192-bit shuffles.
template <int N>
__device__ __forceinline__ MinPD wave_min_pd(MinPD a) {
  const bool none = a.d == 0x7FFFFFFF;
  if (__ballot(!none && (a.s.hi >> 32) != 0) == 0) {
    uint64_t k1 = ~uint64_t(0), k0 = ~uint64_t(0);  // d < 2^31 - 1: no entry has k0 = ~0
    if (!none) {
      k1 = (uint64_t(a.s.hi) << 32) | (a.s.lo >> 32);
      k0 = (a.s.lo << 32) | uint32_t(a.d);
    }
    wave_min_key<N>(k1, k0);
    if (k0 == ~uint64_t(0)) return MinPD{{0, 0}, 0x7FFFFFFF};
    return MinPD{{u128(k1 >> 32), (k1 << 32) | (k0 >> 32)}, int32_t(uint32_t(k0))};
  }
  for (int m = N > 32 ? 32 : N / 2; m >= 1; m >>= 1) min_pd_xor(a, m);  // lanes 0..N-1 hold the minimum
  MinPD r;
  r.s.hi = u128(readlane128(i128(a.s.hi), 0));
  r.s.lo = readlane64(a.s.lo, 0);
  r.d = __builtin_amdgcn_readlane(a.d, 0);
  return r;
}

// ---------------------------------------------------------------------------------
// Speculative blocks.  A decision adds to one instance's queue and count, so it raises
// that instance's score and no other.  Requests are taken in blocks of SQW.  Launch L runs
// two kinds of workgroup on the state X_L it starts from (the queues and counts after
// blocks 0 .. L-2): ranking workgroups list, for every request of block L, its SQK best
// candidates on X_L; the deciding workgroup decides block L-1 starting from X_L and writes
// X_{L+1}.  When a request of block L is decided (launch L+1), the instances whose scores
// have changed since X_L are those updated by block L-1 and by the earlier requests of
// block L: at most 2 SQW - 1 < SQK.  So some listed candidate e* still has its X_L score,
// and every unlisted candidate x scores at least its X_L score, which is above e*'s (the
// keys (score, rotation distance) are distinct): the minimum over all candidates is the
// minimum over the list, rescored on the current state.  Nothing is approximated.
// ---------------------------------------------------------------------------------
constexpr int SQW = 32;       // requests per block
constexpr int SQK = 2 * SQW;  // listed candidates per request
constexpr int SQE = SQK / 64;  // listed candidates per lane when a request is decided
constexpr int SQT = 1024;     // threads per workgroup of the block kernel
constexpr int SQ_NP = SEQC_MAX_I;
static_assert(SQ_NP <= 4096, "rotation distances are packed in 12 bits");

struct SeqCWs {
  SeqCRec *recs;     // [n_req]
  uint32_t *l_inst;  // [2][SQW][SQK] listed instances, by block parity, request in block, rank
  i128 *l_cst;       // [2][SQW][SQK] their doubled prefill costs for the request
  uint32_t *l_cnt;   // [2][SQW] entries listed
  i128 *q2;          // [2][I] doubled queues; X_L is [L & 1]
  uint32_t *nr;      // [2][I] request counts
  int32_t *st;       // 1 iff the instance state given is in domain
};
inline uint64_t seqc_layout(int32_t n_req, int32_t I, SeqCWs *w, void *base) {
  uint64_t off = 0;
  auto take = [&](uint64_t bytes) {
    const uint64_t o = off;
    off = (off + bytes + 255) / 256 * 256;
    return o;
  };
  const uint64_t R = uint64_t(n_req < 1 ? 1 : n_req), NI = uint64_t(I < 1 ? 1 : I);
  const uint64_t o_rec = take(R * sizeof(SeqCRec)), o_li = take(4ull * 2 * SQW * SQK),
                 o_lc = take(16ull * 2 * SQW * SQK), o_ln = take(4ull * 2 * SQW), o_q = take(16 * 2 * NI),
                 o_n = take(4 * 2 * NI), o_st = take(4);
  if (w) {
    char *b = static_cast<char *>(base);
    w->recs = reinterpret_cast<SeqCRec *>(b + o_rec);
    w->l_inst = reinterpret_cast<uint32_t *>(b + o_li);
    w->l_cst = reinterpret_cast<i128 *>(b + o_lc);
    w->l_cnt = reinterpret_cast<uint32_t *>(b + o_ln);
    w->q2 = reinterpret_cast<i128 *>(b + o_q);
    w->nr = reinterpret_cast<uint32_t *>(b + o_n);
    w->st = reinterpret_cast<int32_t *>(b + o_st);
  }
  return off;
}

// X_0: the doubled queues and the counts given, and whether they are in domain.
__global__ __launch_bounds__(SQT) void route_seqc_init_kernel(int32_t I, const int64_t *__restrict__ q,
                                                              const int32_t *__restrict__ n_run, SeqCWs w) {
  int ok = 1;
  for (int32_t i = threadIdx.x; i < I; i += SQT) {
    const int64_t qi = q[i];
    const int32_t ni = n_run[i];
    if (qi < 0 || qi >= (int64_t(1) << 62) || ni < 0) ok = 0;
    w.q2[i] = i128(2) * qi;
    w.nr[i] = uint32_t(ni);
  }
  ok = __syncthreads_and(ok);
  if (threadIdx.x == 0) *w.st = ok;
}

// A candidate's key as three words compared in order (k2, k1, k0); all ones: no candidate.
struct Key3 {
  uint64_t k2, k1, k0;
};
__device__ __forceinline__ bool key_less(const Key3 &a, const Key3 &b) {
  return a.k2 < b.k2 || (a.k2 == b.k2 && (a.k1 < b.k1 || (a.k1 == b.k1 && a.k0 < b.k0)));
}
__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
  const int lo = __shfl(int(uint32_t(v)), src, 64), hi = __shfl(int(uint32_t(v >> 32)), src, 64);
  return (uint64_t(uint32_t(hi)) << 32) | uint32_t(lo);
}
__device__ __forceinline__ Key3 key_shfl(const Key3 &k, int src) {
  return Key3{shfl64(k.k2, src), shfl64(k.k1, src), shfl64(k.k0, src)};
}
// Compare-exchange with lane ^ j: this lane keeps the smaller key iff keep_min.
__device__ __forceinline__ void key_cx(Key3 &k, int j, bool keep_min) {
  const int lane = threadIdx.x & 63;
  const Key3 o = key_shfl(k, lane ^ j);
  if (key_less(o, k) == keep_min) k = o;
}
// The wavefront's 64 keys (one per lane) sorted ascending across the lanes (bitonic network).
__device__ __forceinline__ void key_sort64(Key3 &k) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1)
#pragma unroll
    for (int j = size >> 1; j > 0; j >>= 1) key_cx(k, j, ((lane & j) == 0) == ((lane & size) == 0));
}
// run and o sorted ascending: run becomes the 64 smallest of both, sorted ascending.
// min(run[l], o[63 - l]) are those 64 keys in bitonic order; a bitonic merge sorts them.
__device__ __forceinline__ void key_merge64(Key3 &run, const Key3 &o_rev) {
  const int lane = threadIdx.x & 63;
  if (key_less(o_rev, run)) run = o_rev;
#pragma unroll
  for (int j = 32; j > 0; j >>= 1) key_cx(run, j, (lane & j) == 0);
}

// Ranking: request j of block L, on X_L.  Every candidate's key is score x 2^12 + rotation
// distance (the score is below 2^160, so the key fits three words).  Each wavefront keeps
// the 64 smallest keys of its instances (w 64 + lane + 1024 m) sorted across its lanes;
// the 16 wavefronts' lists are then merged pairwise through LDS, and the SQK = 64 smallest
// keys overall are listed with their costs.  The list need not be in key order: the
// deciding wavefront rescores every listed candidate.
__device__ __forceinline__ void seqc_rank(int32_t L, const int32_t *__restrict__ matched, int32_t n_req, int32_t I,
                                          const int64_t *__restrict__ slack, const RouteParams &p, const SeqCWs &w,
                                          uint64_t *smem) {
  static_assert(SQK == 64 && SQT == 1024, "one listed candidate per lane, 16 wavefronts");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int32_t j = int32_t(blockIdx.x) - 1;
  const int32_t r = L * SQW + j;
  if (r >= n_req) return;  // whole workgroup
  const uint64_t le = uint64_t((L & 1) * SQW + j);
  const SeqCRec rec = w.recs[r];
  if (!*w.st || !(rec.flags & 1)) {  // out of domain: decided without a list
    if (tid == 0) w.l_cnt[le] = 0;
    return;
  }
  const int64_t Lr = rec.L;
  const int32_t start = rec.start;
  const bool any_pass = rec.flags & 16;
  const i128 *q2 = w.q2 + uint64_t(L & 1) * I;
  const uint32_t *nr = w.nr + uint64_t(L & 1) * I;
  const int32_t *c = matched + int64_t(r) * I;
  constexpr uint64_t ONES = ~uint64_t(0);
  Key3 run{ONES, ONES, ONES};
  for (int32_t base = wave * 64; base < I; base += SQT) {  // wavefront-uniform
    const int32_t i = base + lane;
    Key3 k{ONES, ONES, ONES};
    if (i < I) {
      const i128 cst = est2(p, Lr, c[i], 0);
      if (!any_pass || tpot_pass(slack[i], cst)) {
        const P192 s = mul192(q2[i] + cst, nr[i]);
        const uint64_t d = uint64_t(i >= start ? i - start : i - start + I);
        const uint64_t h0 = uint64_t(s.hi), h1 = uint64_t(s.hi >> 64);
        k.k0 = (s.lo << 12) | d;
        k.k1 = (s.lo >> 52) | (h0 << 12);
        k.k2 = (h0 >> 52) | (h1 << 12);  // below 2^44: no candidate's key is all ones
      }
    }
    key_sort64(k);
    if (base == wave * 64) {
      run = k;
    } else {
      key_merge64(run, key_shfl(k, 63 - lane));
    }
  }
  // pairwise merges: at level h, wavefront w < h takes the list of wavefront w + h
  Key3 *buf = reinterpret_cast<Key3 *>(smem);  // [8][64]
#pragma unroll
  for (int h = 8; h >= 1; h >>= 1) {
    if (wave >= h && wave < 2 * h) buf[(wave - h) * 64 + lane] = run;
    __syncthreads();
    if (wave < h) key_merge64(run, buf[wave * 64 + 63 - lane]);
    __syncthreads();
  }
  if (wave != 0) return;
  const bool listed = !(run.k2 == ONES && run.k1 == ONES && run.k0 == ONES);
  if (listed) {  // the listed entries are the first cnt lanes (keys ascending, padding last)
    int32_t inst = start + int32_t(run.k0 & 4095);
    inst = inst >= I ? inst - I : inst;
    w.l_inst[le * SQK + lane] = uint32_t(inst);
    w.l_cst[le * SQK + lane] = est2(p, Lr, c[inst], 0);
  }
  const int cnt = __popcll(__ballot(listed));
  if (lane == 0) w.l_cnt[le] = uint32_t(cnt);
}

// A request to decide with its record and list (entries lane + 64 h, h < SQE).
struct SeqLRow {
  SeqCRec rec;
  uint32_t cnt;
  uint32_t inst[SQE];
  i128 cst[SQE];
};
// The deciding workgroup's copy of block L-1 in LDS: records, list counts and lists.
struct SeqCStage {
  int32_t bs;           // the block's first request
  const SeqCRec *rec;   // [SQW]
  const uint32_t *cnt;  // [SQW]
  const uint32_t *inst;  // [SQW][SQK]
  const i128 *cst;       // [SQW][SQK]
};
__device__ __forceinline__ void seqc_lrow_load(int32_t r, int32_t re, const SeqCStage &sg, SeqLRow &row) {
  const int lane = threadIdx.x & 63;
  const int32_t x = (r < re ? r : re - 1) - sg.bs;  // clamped, unconditional loads: see seq_load
  row.rec = sg.rec[x];
  row.cnt = sg.cnt[x];
#pragma unroll
  for (int h = 0; h < SQE; ++h) {
    row.inst[h] = sg.inst[x * SQK + lane + 64 * h];
    row.cst[h] = sg.cst[x * SQK + lane + 64 * h];
  }
}

// Decide request r alone on the current state (wavefront 0; uniform branches).
__device__ __forceinline__ void seqc_list_decide(const SeqLRow &row, int32_t r, int32_t I, const RouteParams &p,
                                                 bool st_ok, i128 *q2, uint32_t *nr, int32_t *__restrict__ target,
                                                 uint8_t *__restrict__ branch) {
  const int lane = threadIdx.x & 63;
  const int32_t flags = uni(row.rec.flags);
  if (!st_ok || !(flags & 1)) {
    if (lane == 0) {
      target[r] = -1;
      branch[r] = SMETRIC_INVALID;
    }
    return;
  }
  const int32_t prev = uni(row.rec.prev);
  const bool cached = flags & 2, follow_up = flags & 4, prev_cand = flags & 8;
  // the listed instances' queues and counts are read with prev's queue, before the branch
  const int32_t start = uni(row.rec.start);
  const int32_t cnt = uni(int32_t(row.cnt));
  const i128 q_prev = q2[prev];
  const uint32_t n_prev = nr[prev];
  i128 a[SQE];
  uint32_t n[SQE], d[SQE];
  bool v[SQE], big = false;
  // Each lane's best one-word key, formed before any branch: while every listed queue is
  // below 2^64 and every score below 2^52, (score, d) is score 2^12 + d in one word.  The
  // ballot below cannot move into a branch, so the listed entries' loads are waited for
  // together with prev's, one LDS round trip for both.
  uint64_t k1w = ~uint64_t(0);
#pragma unroll
  for (int h = 0; h < SQE; ++h) {
    v[h] = lane + 64 * h < cnt;
    const int32_t i = v[h] ? int32_t(row.inst[h]) : 0;
    a[h] = q2[i] + row.cst[h];
    n[h] = nr[i];
    d[h] = uint32_t(i >= start ? i - start : i - start + I);
    const uint64_t lo = uint64_t(a[h]);
    const uint64_t p0 = uint64_t(uint32_t(lo)) * n[h];
    const uint64_t p1 = (lo >> 32) * n[h] + (p0 >> 32);  // score = p1 2^32 + low word of p0
    const bool b = (a[h] >> 64) != 0 || p1 >= (uint64_t(1) << 20);
    big |= v[h] && b;
    const uint64_t k = (p1 << 44) | (uint64_t(uint32_t(p0)) << 12) | d[h];
    k1w = v[h] && k < k1w ? k : k1w;
  }
  const bool one_word = __ballot(big) == 0;
  // the same on every lane (prev's queue and the record are); read as one scalar so that the
  // branches below are uniform ones, with no exec-mask bookkeeping
  const bool meets_prev = uni(int32_t(q_prev <= row.rec.thr)) != 0;
  int32_t t;
  uint8_t br;
  bool mine;  // this lane writes t's new queue and count (values it already holds)
  i128 q_new = 0;
  uint32_t n_new = 0;
  if (follow_up && cached && meets_prev && prev_cand) {
    t = prev;
    br = SMETRIC_STICK;
    mine = lane == 0;
    q_new = q_prev + row.rec.cost_prev;
    n_new = n_prev + 1;
  } else {
    int32_t dmin;
    bool wide = false;
#pragma unroll
    for (int h = 0; h < SQE; ++h) wide |= v[h] && (a[h] >> 64) != 0;
    if (one_word) {
      dmin = int32_t(uint32_t(wave_min_u64(k1w)) & 4095u);
    } else if (__ballot(wide) == 0) {  // every listed queue below 2^64: scores below 2^96, two words
      uint64_t k1 = ~uint64_t(0), k0 = ~uint64_t(0);
#pragma unroll
      for (int h = 0; h < SQE; ++h)
        if (v[h]) {
          const uint64_t lo = uint64_t(a[h]);
          const uint64_t p0 = uint64_t(uint32_t(lo)) * n[h];
          const uint64_t p1 = (lo >> 32) * n[h] + (p0 >> 32);  // score = p1 2^32 + low word of p0
          const uint64_t c0 = (p0 << 32) | d[h];
          if (p1 < k1 || (p1 == k1 && c0 < k0)) {
            k1 = p1;
            k0 = c0;
          }
        }
      wave_min_key<64>(k1, k0);
      dmin = int32_t(uint32_t(k0));
    } else {
      MinPD best{{0, 0}, 0x7FFFFFFF};
#pragma unroll
      for (int h = 0; h < SQE; ++h)
        if (v[h]) min_pd(best, mul192(a[h], n[h]), int32_t(d[h]));
      best = wave_min_pd<64>(best);
      dmin = best.d;
    }
    t = start + uni(dmin);  // start, d < I
    t = t >= I ? t - I : t;
    br = !follow_up ? SMETRIC_FIRST_TURN
                    : (!cached ? SMETRIC_EVICTED : (!meets_prev ? SMETRIC_MIGRATE : SMETRIC_MIGRATE_TPOT));
    mine = false;
#pragma unroll
    for (int h = 0; h < SQE; ++h)
      if (v[h] && int32_t(row.inst[h]) == t) {
        mine = true;
        q_new = a[h];  // its queue plus the request's cost there
        n_new = n[h] + 1;
      }
  }
  __builtin_amdgcn_wave_barrier();
  if (mine) {  // one lane: the listed instances are distinct
    q2[t] = q_new;
    nr[t] = n_new;
    target[r] = t;
    branch[r] = br;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// Deciding: block L-1 in steps of up to 64 requests, one per lane, as route_seq_kernel (a
// cached follow-up whose prev is a candidate sticks iff prev meets its deadline on its
// exact load: prev's queue plus the costs of the step's earlier requests with that prev);
// the first request not settled is decided by its list, and the next step starts after it.
// After two steps that settle nothing, the next 64 requests go one by one with their
// records and lists loaded D requests ahead.
template <int D>
__device__ __forceinline__ void seqc_decide_block(int32_t be, int32_t I, const RouteParams &p, const SeqCStage &sg,
                                                  bool st_ok, i128 *q2, uint32_t *nr, uint32_t *n_on,
                                                  int32_t *__restrict__ target, uint8_t *__restrict__ branch) {
  const int lane = threadIdx.x & 63;
  const int32_t bs = sg.bs;
  int32_t r0 = bs;
  int streak = 0;
  while (r0 < be) {
    if (streak >= 2) {
      const int32_t re = be - r0 < 64 ? be : r0 + 64;
      // ring slots are used in place (no register copies, which would have to wait for the
      // newest loads) and refilled unconditionally (clamped): a load under a branch is
      // waited for at the join
      SeqLRow ring[D];
#pragma unroll
      for (int d = 0; d < D; ++d) seqc_lrow_load(r0 + d, be, sg, ring[d]);
      for (int32_t r = r0; r < re; r += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
          if (r + d < re) seqc_list_decide(ring[d], r + d, I, p, st_ok, q2, nr, target, branch);
          seqc_lrow_load(r + d + D, be, sg, ring[d]);
        }
      }
      r0 = re;
      streak = 0;
      continue;
    }
    const int32_t nv = be - r0 < 64 ? be - r0 : 64;
    const int32_t r = r0 + lane;
    const SeqCRec rec = sg.rec[(r < be ? r : be - 1) - bs];
    const bool in = lane < nv;
    const bool ok = st_ok && (rec.flags & 1);
    const bool sticky = ok && (rec.flags & 2) && (rec.flags & 4) && (rec.flags & 8);
    const int32_t prev = rec.prev;
    const bool mine = in && sticky;
    if (mine) atomicAdd(&n_on[prev], 1u);
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    uint64_t todo = __ballot(mine && n_on[prev] > 1);
    __builtin_amdgcn_wave_barrier();
    if (mine) n_on[prev] = 0;
    i128 excl = 0;
    uint64_t group = 0;  // lanes with my prev (0: nobody else has it)
    while (todo) {
      const int32_t p0 = __builtin_amdgcn_readlane(prev, __builtin_ctzll(todo));
      const uint64_t m = __ballot(mine && prev == p0);
      todo &= ~m;
      i128 run = 0;
      for (uint64_t mm = m; mm; mm &= mm - 1) {
        const int l = __builtin_ctzll(mm);
        if (lane == l) {
          excl = run;
          group = m;
        }
        run += readlane128(rec.cost_prev, l);
      }
    }
    const i128 q_prev = (mine ? q2[prev] : i128(0)) + excl;
    bool settled = !ok;  // out of domain: settled, nothing queued
    uint8_t br = SMETRIC_INVALID;
    if (sticky && q_prev <= rec.thr) {
      settled = true;
      br = SMETRIC_STICK;
    }
    const uint64_t open = __ballot(in && !settled);
    const int32_t f = open ? __builtin_ctzll(open) : nv;  // requests [r0, r0 + f) are decided
    SeqLRow row;
    if (f < nv) seqc_lrow_load(r0 + f, be, sg, row);
    if (lane < f) {
      target[r] = ok ? prev : -1;
      branch[r] = br;
    }
    const uint64_t decided = f >= 64 ? ~uint64_t(0) : (uint64_t(1) << f) - 1;
    const uint64_t after_me = lane == 63 ? uint64_t(0) : ~((uint64_t(2) << lane) - 1);
    const bool last = mine && lane < f && (group & after_me & decided) == 0;
    const uint32_t added = group ? __popcll(group & decided) : 1;  // the group's requests decided here
    __builtin_amdgcn_wave_barrier();
    if (last) {
      q2[prev] = q_prev + rec.cost_prev;
      nr[prev] = nr[prev] + added;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    r0 += f;
    if (f < nv) {  // the first request not settled: decided by its list
      seqc_list_decide(row, r0, I, p, st_ok, q2, nr, target, branch);
      r0 += 1;
      streak = f == 0 ? streak + 1 : 0;
    }
  }
}

// Launch L: workgroup 0 decides block L-1 (L >= 1) and writes X_{L+1}; workgroups 1 ..
// rank the requests of block L (L < number of blocks).
constexpr int SQ_STAGE_WORDS = (SQW * SQK * 16 + SQW * int(sizeof(SeqCRec)) + SQW * SQK * 4 + SQW * 4 + 7) / 8;
__global__ __launch_bounds__(SQT) void route_seqc_block_kernel(int32_t L, const int32_t *__restrict__ matched,
                                                               int32_t n_req, int32_t I,
                                                               const int64_t *__restrict__ slack, RouteParams p,
                                                               SeqCWs w, int32_t *__restrict__ target,
                                                               uint8_t *__restrict__ branch) {
  // deciding: queues (16 B), counts and step counters per instance, then block L-1 staged
  // (costs, records, instances, counts); ranking: the merge buffer
  __shared__ uint64_t smem[3 * SQ_NP + SQ_STAGE_WORDS];
  if (blockIdx.x > 0) {
    seqc_rank(L, matched, n_req, I, slack, p, w, smem);
    return;
  }
  i128 *q2 = reinterpret_cast<i128 *>(smem);
  uint32_t *nr = reinterpret_cast<uint32_t *>(smem + 2 * SQ_NP);
  uint32_t *n_on = nr + SQ_NP;
  i128 *s_cst = reinterpret_cast<i128 *>(smem + 3 * SQ_NP);
  SeqCRec *s_rec = reinterpret_cast<SeqCRec *>(s_cst + SQW * SQK);
  uint32_t *s_inst = reinterpret_cast<uint32_t *>(s_rec + SQW);
  uint32_t *s_cnt = s_inst + SQW * SQK;
  const uint64_t sx = uint64_t(L & 1) * I, sy = uint64_t((L + 1) & 1) * I;
  for (int32_t i = threadIdx.x; i < I; i += SQT) {
    q2[i] = w.q2[sx + i];
    nr[i] = w.nr[sx + i];
    n_on[i] = 0;
  }
  const int32_t bs = (L - 1) * SQW, nb = L >= 1 ? (n_req - bs < SQW ? n_req - bs : SQW) : 0;
  const uint64_t le0 = uint64_t(((L - 1) & 1) * SQW);
  for (int32_t x = threadIdx.x; x < nb * SQK; x += SQT) {
    s_inst[x] = w.l_inst[le0 * SQK + x];
    s_cst[x] = w.l_cst[le0 * SQK + x];
  }
  for (int32_t x = threadIdx.x; x < nb; x += SQT) {
    s_rec[x] = w.recs[bs + x];
    s_cnt[x] = w.l_cnt[le0 + x];
  }
  __syncthreads();
  if (L >= 1 && threadIdx.x < 64) {
    const SeqCStage sg{bs, s_rec, s_cnt, s_inst, s_cst};
    seqc_decide_block<3>(bs + nb, I, p, sg, *w.st != 0, q2, nr, n_on, target, branch);
  }
  __syncthreads();
  for (int32_t i = threadIdx.x; i < I; i += SQT) {
    w.q2[sy + i] = q2[i];
    w.nr[sy + i] = nr[i];
  }
}

__global__ void route_seqc_final_kernel(int32_t I, int32_t slot, SeqCWs w, const int64_t *__restrict__ q,
                                        const int32_t *__restrict__ n_run, int64_t *__restrict__ q_out,
                                        int64_t *__restrict__ n_out) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= I) return;
  const bool ok = *w.st != 0;  // an invalid state is echoed as given
  if (q_out) {
    const i128 v = w.q2[uint64_t(slot) * I + i] >> 1;
    q_out[i] = !ok ? q[i] : (v > i128(INT64_MAX) ? INT64_MAX : int64_t(v));
  }
  if (n_out) n_out[i] = ok ? int64_t(w.nr[uint64_t(slot) * I + i]) : int64_t(n_run[i]);
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

// Requests routed one at a time: every running load stays below 2 q + (n_req + 1) x the
// largest doubled cost a request in domain can add (L <= 2^24, so n (2L - n) <= 2^48), and
// the deadline check multiplies it by SLACK's denominator.  The batch is accepted only when
// that product stays below 2^126, so no comparison of the online rules can overflow.
bool seq_loads_fit(const RouteParams &p, int32_t n_req) {
  const i128 cmax = i128(2) * p.c_lin * (int64_t(1) << 24) + i128(p.c_att) * (i128(1) << 48);
  const i128 worst = (i128(1) << 63) + i128(int64_t(n_req) + 1) * cmax;
  return worst < (i128(1) << 126) / i128(p.slack_den > 0 ? p.slack_den : 1);
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
  hipLaunchKernelGGL(route_kernel<0>, dim3((n_req + RW - 1) / RW), dim3(64 * RW), 0, stream, matched, n_req,
                     n_instances, prompt_len, hist_len, turn, q, rp, rr_base, target, branch, nullptr, 0, 0);
  return hip_rc(hipGetLastError());
}

extern "C" int smetric_route_loadaware(const int32_t *matched, int32_t n_req, int32_t n_instances,
                                       const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                                       const int64_t *q, const int64_t *load, int32_t margin_num,
                                       int32_t margin_den, const smetric_params *params, uint64_t rr_base,
                                       int32_t *target, uint8_t *branch, hipStream_t stream) {
  RouteParams rp;
  if (int rc = route_params(params, n_req, n_instances, rp)) return rc;
  if (margin_num < 0 || margin_den < 0) return SMETRIC_EINVAL;
  if (n_req == 0) return SMETRIC_OK;
  if (!matched || !prompt_len || !hist_len || !turn || !q || !load || !target || !branch) return SMETRIC_EINVAL;
  hipLaunchKernelGGL(route_kernel<1>, dim3((n_req + RW - 1) / RW), dim3(64 * RW), 0, stream, matched, n_req,
                     n_instances, prompt_len, hist_len, turn, q, rp, rr_base, target, branch, load, margin_num,
                     margin_den);
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

extern "C" int smetric_route_seq_coloc(const int32_t *matched, int32_t n_req, int32_t n_instances,
                                       const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                                       const int64_t *q, const int64_t *tpot_slack, const int32_t *n_running,
                                       const smetric_params *params, uint64_t rr_base, int32_t *target,
                                       uint8_t *branch, int64_t *q_out, int64_t *n_out, void *workspace,
                                       uint64_t ws_bytes, hipStream_t stream) {
  RouteParams rp;
  if (int rc = route_params(params, n_req, n_instances, rp)) return rc;
  if (n_instances > SEQC_MAX_I || !seq_loads_fit(rp, n_req)) return SMETRIC_EINVAL;
  if (!q || !tpot_slack || !n_running) return SMETRIC_EINVAL;
  if (n_req > 0 && (!matched || !prompt_len || !hist_len || !turn || !target || !branch)) return SMETRIC_EINVAL;
  const uint64_t need = seqc_layout(n_req, n_instances, nullptr, nullptr);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) || ws_bytes < need) return SMETRIC_EWORKSPACE;
  SeqCWs w;
  seqc_layout(n_req, n_instances, &w, workspace);
  if (n_req > 0)
    hipLaunchKernelGGL(route_seqc_prep_kernel, dim3((n_req + RW - 1) / RW), dim3(64 * RW), 0, stream, matched,
                       n_req, n_instances, prompt_len, hist_len, turn, tpot_slack, rp, rr_base, w.recs);
  hipLaunchKernelGGL(route_seqc_init_kernel, dim3(1), dim3(SQT), 0, stream, n_instances, q, n_running, w);
  const int32_t n_blk = (n_req + SQW - 1) / SQW;
  for (int32_t L = 0; L <= n_blk; ++L) {
    const int32_t rank = L < n_blk ? (n_req - L * SQW < SQW ? n_req - L * SQW : SQW) : 0;
    hipLaunchKernelGGL(route_seqc_block_kernel, dim3(1 + rank), dim3(SQT), 0, stream, L, matched, n_req,
                       n_instances, tpot_slack, rp, w, target, branch);
  }
  if (q_out || n_out)
    hipLaunchKernelGGL(route_seqc_final_kernel, dim3((n_instances + 255) / 256), dim3(256), 0, stream, n_instances,
                       (n_blk + 1) & 1, w, q, n_running, q_out, n_out);
  return hip_rc(hipGetLastError());
}

extern "C" int smetric_route_seq_coloc_ws_bytes(int32_t n_req, int32_t n_instances, uint64_t *ws_bytes) {
  if (n_req < 0 || n_instances < 1 || n_instances > SEQC_MAX_I || !ws_bytes) return SMETRIC_EINVAL;
  *ws_bytes = seqc_layout(n_req, n_instances, nullptr, nullptr);
  return SMETRIC_OK;
}

extern "C" int smetric_route_seq_ws_bytes(int32_t n_req, uint64_t *ws_bytes) {
  if (n_req < 0 || !ws_bytes) return SMETRIC_EINVAL;
  *ws_bytes = (uint64_t(n_req < 1 ? 1 : n_req) * sizeof(SeqRec) + 255) / 256 * 256;
  return SMETRIC_OK;
}

namespace smk {
namespace {

// The online route after its host checks: the pre-pass writes every request's record
// into recs (nothing there needs clearing), then one wavefront walks the batch.
int route_seq_launch(const int32_t *matched, int32_t n_req, int32_t n_instances, const int32_t *prompt_len,
                     const int32_t *hist_len, const int32_t *turn, const int64_t *q, const RouteParams &rp,
                     uint64_t rr_base, int32_t *target, uint8_t *branch, int64_t *q_out, SeqRec *recs,
                     hipStream_t stream) {
  if (n_req > 0)
    hipLaunchKernelGGL(route_seq_prep_kernel, dim3((n_req + RW - 1) / RW), dim3(64 * RW), 0, stream, matched, n_req,
                       n_instances, prompt_len, hist_len, turn, q, rp, rr_base, recs);
  const int kk = (n_instances + 63) / 64;
#define SEQ_LAUNCH(K, D)                                                                                       \
  hipLaunchKernelGGL((route_seq_kernel<K, D>), dim3(1), dim3(64), 0, stream, matched, n_req, n_instances,         \
                     q, rp, recs, target, branch, q_out)
  // prefetch depth D: D * (K + 4) vector loads in flight (K row words and a 64-byte
  // record per request) stay within the 63 the wait counter tracks
  if (kk <= 1) SEQ_LAUNCH(1, 8);
  else if (kk <= 2) SEQ_LAUNCH(2, 8);
  else if (kk <= 4) SEQ_LAUNCH(4, 7);
  else if (kk <= 8) SEQ_LAUNCH(8, 5);
  else if (kk <= 16) SEQ_LAUNCH(16, 3);
  else SEQ_LAUNCH(0, 8);
#undef SEQ_LAUNCH
  return hip_rc(hipGetLastError());
}

int route_seq_checks(const int32_t *matched, int32_t n_req, int32_t n_instances, const int32_t *prompt_len,
                     const int32_t *hist_len, const int32_t *turn, const int64_t *q, const smetric_params *params,
                     int32_t *target, uint8_t *branch, RouteParams &rp) {
  if (int rc = route_params(params, n_req, n_instances, rp)) return rc;
  if (n_instances > SEQ_MAX_I || !seq_loads_fit(rp, n_req)) return SMETRIC_EINVAL;
  if (!q) return SMETRIC_EINVAL;
  if (n_req > 0 && (!matched || !prompt_len || !hist_len || !turn || !target || !branch)) return SMETRIC_EINVAL;
  return SMETRIC_OK;
}

// Scratch of the allocation-free online route: one record per request, in a file-scope
// device array that every GPU the library runs on holds until the process ends.  Host
// code never passes the array's name to a kernel (on the host it is a stand-in, not a
// device address): each device's address is looked up once, with that device current,
// and kept.
constexpr int32_t SEQ_NOALLOC_MAX_REQ = 65536;
constexpr int SEQ_NOALLOC_MAX_DEVICES = 64;
static __device__ __align__(256) SeqRec seq_scratch[SEQ_NOALLOC_MAX_REQ];
std::mutex seq_scratch_mu;
SeqRec *seq_scratch_dev[SEQ_NOALLOC_MAX_DEVICES] = {};

int seq_scratch_ptr(SeqRec **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SEQ_NOALLOC_MAX_DEVICES) return SMETRIC_EHIP;
  std::lock_guard<std::mutex> lock(seq_scratch_mu);
  if (!seq_scratch_dev[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(seq_scratch)) != hipSuccess || !p) return SMETRIC_EHIP;
    seq_scratch_dev[dev] = static_cast<SeqRec *>(p);
  }
  *out = seq_scratch_dev[dev];
  return SMETRIC_OK;
}

}  // namespace
}  // namespace smk

extern "C" int smetric_route_seq(const int32_t *matched, int32_t n_req, int32_t n_instances,
                                 const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                                 const int64_t *q, const smetric_params *params, uint64_t rr_base,
                                 int32_t *target, uint8_t *branch, int64_t *q_out, void *workspace,
                                 uint64_t ws_bytes, hipStream_t stream) {
  RouteParams rp;
  if (int rc = route_seq_checks(matched, n_req, n_instances, prompt_len, hist_len, turn, q, params, target, branch,
                                rp))
    return rc;
  uint64_t need = 0;
  smetric_route_seq_ws_bytes(n_req, &need);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) || ws_bytes < need) return SMETRIC_EWORKSPACE;
  return route_seq_launch(matched, n_req, n_instances, prompt_len, hist_len, turn, q, rp, rr_base, target, branch,
                          q_out, static_cast<SeqRec *>(workspace), stream);
}

extern "C" int smetric_route_seq_noalloc_max_req(void) { return SEQ_NOALLOC_MAX_REQ; }

extern "C" int smetric_route_seq_noalloc(const int32_t *matched, int32_t n_req, int32_t n_instances,
                                         const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                                         const int64_t *q, const smetric_params *params, uint64_t rr_base,
                                         int32_t *target, uint8_t *branch, int64_t *q_out, hipStream_t stream) {
  RouteParams rp;
  if (int rc = route_seq_checks(matched, n_req, n_instances, prompt_len, hist_len, turn, q, params, target, branch,
                                rp))
    return rc;
  if (n_req > SEQ_NOALLOC_MAX_REQ) return SMETRIC_EWORKSPACE;
  SeqRec *recs = nullptr;
  if (int rc = seq_scratch_ptr(&recs)) return rc;
  return route_seq_launch(matched, n_req, n_instances, prompt_len, hist_len, turn, q, rp, rr_base, target, branch,
                          q_out, recs, stream);
}
