// The scoring template's comparison scorers: route every request to argmin_i f(req, i).
//
// Paper: Sec. 4.1 casts request routing as picking the instance with the lowest score f of
// its load and the request's KV$ hit; the motivating analysis of Sec. 4.1 and the baselines
// of Sec. 5 differ only in f -- load balance only (f = load), Dynamo's fewest tokens left to
// prefill, LMetric's product, the production scheduler's weighted sum of normalised load
// and miss ratio, and Preble's hit filter (more than half the prompt cached) in front of
// that weighted sum.  The exact integer forms are stated with smetric_route_score.
//
// Mapping to gfx950: one wavefront per request, as in the main route.  Lane l scores
// instances l, l + 64, ... (the loads of four of them issued together) and keeps the
// minimum of (score, rotation distance) -- and, for the hit filter, of (load, rotation
// distance) over the instances holding more than half the prompt; a butterfly across the
// wavefront finishes both and lane 0 writes the decision.  The weighted sum's normaliser (the
// cluster's largest load) is reduced once per workgroup into LDS.  Scores that fit 64 bits
// (load, tokens) stay 64-bit; the product and the weighted sum are formed in 128 bits.
#include <type_traits>

#include "common.h"

namespace smk {
namespace {

constexpr int SW = 4;  // waves per workgroup, one request each
constexpr int SU = 4;  // instances per lane whose loads are issued together
constexpr int32_t NONE = 0x7FFFFFFF;
typedef __int128 i128;

__device__ __forceinline__ int64_t shfl_xor_s(int64_t v, int m) {
  const int32_t lo = __shfl_xor(int32_t(uint32_t(uint64_t(v))), m, 64);
  const int32_t hi = __shfl_xor(int32_t(uint32_t(uint64_t(v) >> 32)), m, 64);
  return int64_t((uint64_t(uint32_t(hi)) << 32) | uint32_t(lo));
}
__device__ __forceinline__ i128 shfl_xor_s(i128 v, int m) {
  const uint64_t lo = uint64_t(shfl_xor_s(int64_t(uint64_t(v)), m));
  const uint64_t hi = uint64_t(shfl_xor_s(int64_t(uint64_t(v >> 64)), m));
  return i128((unsigned __int128)hi << 64 | lo);
}

// (s, d) replaces (bs, bd) when it is smaller, the rotation distance d breaking ties;
// d == NONE marks "no candidate yet"
template <typename S>
__device__ __forceinline__ void take_min(S &bs, int32_t &bd, S s, int32_t d) {
  if (d != NONE && (bd == NONE || s < bs || (s == bs && d < bd))) {
    bs = s;
    bd = d;
  }
}

// KIND: 0 load only, 1 tokens left, 2 product, 3 weighted sum, 4 hit filter + weighted sum
template <int KIND>
__global__ __launch_bounds__(64 * SW) void route_score_kernel(
    const int32_t *__restrict__ matched, int32_t n_req, int32_t I, const int32_t *__restrict__ prompt_len,
    const int64_t *__restrict__ q, const int32_t *__restrict__ load, int32_t B, int32_t lam_num,
    int32_t lam_den, uint64_t rr_base, int32_t *__restrict__ target, uint8_t *__restrict__ branch) {
  typedef typename std::conditional<(KIND <= 1), int64_t, i128>::type S;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int32_t lmax = 0;
  if (KIND >= 3) {  // the weighted sum normalises loads by the cluster's largest
    __shared__ int32_t s_max[SW];
    int32_t m = 0;
    for (int32_t i = threadIdx.x; i < I; i += 64 * SW) m = max(m, load[i]);
#pragma unroll
    for (int k = 32; k >= 1; k >>= 1) m = max(m, __shfl_xor(m, k, 64));
    if (lane == 0) s_max[wave] = m;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < SW; ++w) lmax = max(lmax, s_max[w]);
  }
  const int32_t r = blockIdx.x * SW + wave;
  if (r >= n_req) return;
  const int32_t *c = matched + int64_t(r) * I;
  const int64_t L = prompt_len[r];
  bool ok = L >= 0 && L <= (int64_t(1) << 24);
  const int64_t max_c = ok ? L / B : -1;
  const int32_t start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));
  // weighted sum times lam_den * Dl * Dc (Dl = max load or 1, Dc = L or 1): the load term
  // weighs l[i] by (lam_den - lam_num) Dc, the miss term weighs the new tokens by lam_num Dl
  const i128 w_load = i128(lam_den - lam_num) * (L > 0 ? L : 1);
  const i128 w_miss = i128(lam_num) * (lmax > 0 ? lmax : 1);

  S best_s = 0;
  int32_t best_d = NONE;
  int32_t hold_l = 0, hold_d = NONE;  // KIND 4: least loaded holder of more than half
  for (int32_t i0 = lane; i0 < I; i0 += 64 * SU) {
    int32_t cv[SU], lv[SU];
    int64_t qv[SU];
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int32_t ii = i0 + 64 * u < I ? i0 + 64 * u : I - 1;
      cv[u] = c[ii];
      qv[u] = q[ii];
      lv[u] = load[ii];
    }
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int32_t i = i0 + 64 * u;
      if (i >= I) break;
      const int32_t ci = cv[u], li = lv[u];
      const int64_t qi = qv[u];
      if (ci < 0 || ci > max_c || qi < 0 || qi >= (int64_t(1) << 62) || li < 0) ok = false;
      const int64_t n = L - int64_t(B) * ci;  // the request's new tokens on i
      S s;
      if (KIND == 0) s = li;
      else if (KIND == 1) s = int64_t(uint64_t(qi) + uint64_t(n));  // wraps only out of domain
      else if (KIND == 2) s = (i128(qi) + n) * li;
      else s = w_load * li + w_miss * n;
      const int32_t d = i >= start ? i - start : i - start + I;
      take_min(best_s, best_d, s, d);
      if (KIND == 4 && 2 * int64_t(B) * ci > L) take_min(hold_l, hold_d, li, d);
    }
  }
  ok = __ballot(!ok) == 0;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const S os = shfl_xor_s(best_s, m);
    const int32_t od = __shfl_xor(best_d, m, 64);
    take_min(best_s, best_d, os, od);
    if (KIND == 4) {
      const int32_t ol = __shfl_xor(hold_l, m, 64), ohd = __shfl_xor(hold_d, m, 64);
      take_min(hold_l, hold_d, ol, ohd);
    }
  }
  if (lane != 0) return;
  if (!ok) {
    target[r] = -1;
    branch[r] = SMETRIC_INVALID;
  } else if (KIND == 4 && hold_d != NONE) {
    target[r] = (start + hold_d) % I;
    branch[r] = SMETRIC_HIT_FILTER;
  } else {
    target[r] = (start + best_d) % I;
    branch[r] = SMETRIC_SCORED;
  }
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_route_score(int32_t kind, const int32_t *matched, int32_t n_req, int32_t n_instances,
                                   const int32_t *prompt_len, const int64_t *q, const int32_t *load,
                                   int32_t block_size, int32_t lam_num, int32_t lam_den, uint64_t rr_base,
                                   int32_t *target, uint8_t *branch, hipStream_t stream) {
  if (kind < SMETRIC_SCORE_LOAD || kind > SMETRIC_SCORE_HIT_FILTER || n_req < 0 || n_instances < 1 ||
      n_instances > 65536 || block_size < 2 || block_size > 256 || (block_size & 1))
    return SMETRIC_EINVAL;
  if ((kind == SMETRIC_SCORE_LINEAR || kind == SMETRIC_SCORE_HIT_FILTER) &&
      (lam_den <= 0 || lam_num < 0 || lam_num > lam_den))
    return SMETRIC_EINVAL;
  if (n_req == 0) return SMETRIC_OK;
  if (!matched || !prompt_len || !q || !load || !target || !branch) return SMETRIC_EINVAL;
  const dim3 grid((n_req + SW - 1) / SW), block(64 * SW);
  switch (kind) {
    case SMETRIC_SCORE_LOAD:
      hipLaunchKernelGGL(route_score_kernel<0>, grid, block, 0, stream, matched, n_req, n_instances, prompt_len,
                         q, load, block_size, lam_num, lam_den, rr_base, target, branch);
      break;
    case SMETRIC_SCORE_TOKENS:
      hipLaunchKernelGGL(route_score_kernel<1>, grid, block, 0, stream, matched, n_req, n_instances, prompt_len,
                         q, load, block_size, lam_num, lam_den, rr_base, target, branch);
      break;
    case SMETRIC_SCORE_PRODUCT:
      hipLaunchKernelGGL(route_score_kernel<2>, grid, block, 0, stream, matched, n_req, n_instances, prompt_len,
                         q, load, block_size, lam_num, lam_den, rr_base, target, branch);
      break;
    case SMETRIC_SCORE_LINEAR:
      hipLaunchKernelGGL(route_score_kernel<3>, grid, block, 0, stream, matched, n_req, n_instances, prompt_len,
                         q, load, block_size, lam_num, lam_den, rr_base, target, branch);
      break;
    default:
      hipLaunchKernelGGL(route_score_kernel<4>, grid, block, 0, stream, matched, n_req, n_instances, prompt_len,
                         q, load, block_size, lam_num, lam_den, rr_base, target, branch);
      break;
  }
  return hip_rc(hipGetLastError());
}
