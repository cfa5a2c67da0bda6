// Session reconstruction from block hashes (App. A).
//
// Paper: a request is the follow-up of an earlier request of the same user when its turn is
// larger by one and its block-hash sequence starts with the other's; chained together, such
// requests form a session.  Readings (smetric.h): requests in arrival order; the most recent
// qualifying request is the parent; the empty sequence is a prefix of every sequence; the
// session is the index of the chain's first request.
//
// Mapping to gfx950: a data-parallel join on one small hash table (two slots per request,
// L2-resident at trace sizes):
//   offer   one thread per request p: the slot of (user, turn + 1, block count, last key)
//           holds p (every request gets its own slot: no merging, one CAS per claim);
//   query   one wavefront per request r, lanes over its prefix lengths n = 0 .. nb_r: the
//           slots of (user_r, turn_r, n, key_r[n-1]) give the earlier requests whose whole
//           sequence is r's first n keys -- with chained keys (key j determines blocks 0..j)
//           one key comparison is the whole prefix test; the largest p < r wins;
//   roots   pointer jumping, ceil(log2 R) rounds (plus one to land in the output), so every
//           request reaches its chain's first request.
#include "common.h"

namespace smk {
namespace {

constexpr int TB = 256;

struct OfferSlot {
  uint64_t h;  // 0 = free; the triple's hash | 1 otherwise
  int32_t p;
  int32_t pad;
};

__device__ __forceinline__ uint64_t triple_hash(uint32_t user, int64_t turn, int64_t n, uint64_t last) {
  uint64_t x = mix64(last ^ 0x9E3779B97F4A7C15ull);
  x = mix64(x ^ (uint64_t(user) << 32 | uint32_t(turn)));
  x = mix64(x ^ uint64_t(n) * 0xC2B2AE3D27D4EB4Full);
  return x | 1;
}

__device__ __forceinline__ bool range_ok(const int64_t *blk_off, int32_t r, int64_t n_blocks, int64_t &b0,
                                         int64_t &nb) {
  b0 = blk_off[r];
  const int64_t b1 = blk_off[r + 1];
  nb = b1 - b0;
  return b0 >= 0 && b0 <= b1 && b1 <= n_blocks;
}

__global__ void offer_clear_kernel(OfferSlot *t, uint64_t ns) {
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < ns; i += stride) t[i] = OfferSlot{0, 0, 0};
}

__global__ __launch_bounds__(TB) void offer_kernel(const uint64_t *__restrict__ keys, const int64_t *__restrict__ blk_off,
                                                   int32_t n_req, int64_t n_blocks, const uint32_t *__restrict__ user,
                                                   const int32_t *__restrict__ turn, OfferSlot *t, uint64_t ns,
                                                   int32_t *status) {
  const int32_t p = int32_t(blockIdx.x) * TB + threadIdx.x;
  if (p >= n_req) return;
  int64_t b0, nb;
  if (!range_ok(blk_off, p, n_blocks, b0, nb) || turn[p] < 0) {
    if (status) atomicCAS(status, 0, SMETRIC_EINVAL);
    return;
  }
  const uint64_t h = triple_hash(user[p], int64_t(turn[p]) + 1, nb, nb > 0 ? keys[b0 + nb - 1] : 0);
  uint64_t s = h & (ns - 1);
  for (uint64_t step = 0; step < ns; ++step, s = (s + 1) & (ns - 1)) {
    if (atomicCAS(reinterpret_cast<unsigned long long *>(&t[s].h), 0ull, h) == 0ull) {
      t[s].p = p;
      return;
    }
  }
}

__global__ __launch_bounds__(TB) void query_kernel(const uint64_t *__restrict__ keys, const int64_t *__restrict__ blk_off,
                                                   int32_t n_req, int64_t n_blocks, const uint32_t *__restrict__ user,
                                                   const int32_t *__restrict__ turn, const OfferSlot *__restrict__ t,
                                                   uint64_t ns, int32_t *__restrict__ parent, int32_t *__restrict__ jump) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int32_t r = int32_t(blockIdx.x) * (TB / 64) + wave;
  if (r >= n_req) return;
  int64_t b0, nb;
  const int32_t tr = turn[r];
  if (!range_ok(blk_off, r, n_blocks, b0, nb) || tr < 0) {
    if (lane == 0) {
      parent[r] = -1;
      jump[r] = -1;
    }
    return;
  }
  const uint32_t u = user[r];
  int32_t best = -1;
  if (tr > 0) {
    for (int64_t n = lane; n <= nb; n += 64) {  // prefix length n: blocks 0 .. n-1
      const uint64_t last = n > 0 ? keys[b0 + n - 1] : 0;
      const uint64_t h = triple_hash(u, tr, n, last);
      uint64_t s = h & (ns - 1);
      for (uint64_t step = 0; step < ns; ++step, s = (s + 1) & (ns - 1)) {
        const uint64_t sh = t[s].h;
        if (sh == 0) break;
        if (sh != h) continue;
        const int32_t p = t[s].p;
        if (p >= r || p <= best) continue;
        // verify the triple itself (the hash is only a filter)
        const int64_t pb0 = blk_off[p], pnb = blk_off[p + 1] - pb0;
        if (user[p] == u && int64_t(turn[p]) + 1 == tr && pnb == n && (n == 0 || keys[pb0 + n - 1] == last))
          best = p;
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const int32_t o = __shfl_xor(best, m, 64);
      best = o > best ? o : best;
    }
  }
  if (lane == 0) {
    parent[r] = best;
    jump[r] = best >= 0 ? best : r;
  }
}

// One round of pointer jumping: a <- a[a] (invalid requests stay -1).
__global__ void jump_kernel(const int32_t *__restrict__ src, int32_t *__restrict__ dst, int32_t n_req) {
  const int32_t r = int32_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= n_req) return;
  const int32_t a = src[r];
  dst[r] = a < 0 ? -1 : src[a];
}

uint64_t offer_slots(int32_t n_req) {
  uint64_t ns = 64;
  while (ns < 2 * uint64_t(n_req < 1 ? 1 : n_req)) ns <<= 1;
  return ns;
}

// Workspace: the offer table, then one int32 per request for pointer jumping.
uint64_t jump_offset(int32_t n_req) { return (offer_slots(n_req) * sizeof(OfferSlot) + 255) / 256 * 256; }
uint64_t sessions_ws_bytes(int32_t n_req) {
  return jump_offset(n_req) + (uint64_t(n_req < 1 ? 1 : n_req) * 4 + 255) / 256 * 256;
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_sessions_ws_bytes(int32_t n_req, uint64_t *ws_bytes) {
  if (n_req < 0 || !ws_bytes) return SMETRIC_EINVAL;
  *ws_bytes = sessions_ws_bytes(n_req);
  return SMETRIC_OK;
}

extern "C" int smetric_sessions(const uint64_t *keys, const int64_t *blk_off, int32_t n_req, int64_t n_blocks,
                                const uint32_t *user, const int32_t *turn, int32_t *parent, int32_t *session,
                                int32_t *status, void *workspace, uint64_t ws_bytes, hipStream_t stream) {
  if (n_req < 0 || n_blocks < 0) return SMETRIC_EINVAL;
  if (n_req == 0) return SMETRIC_OK;
  if (!blk_off || !user || !turn || !parent || !session || (n_blocks > 0 && !keys)) return SMETRIC_EINVAL;
  const uint64_t need = sessions_ws_bytes(n_req);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) || ws_bytes < need) return SMETRIC_EWORKSPACE;
  const uint64_t ns = offer_slots(n_req);
  char *base = static_cast<char *>(workspace);
  OfferSlot *t = reinterpret_cast<OfferSlot *>(base);
  int32_t *jump = reinterpret_cast<int32_t *>(base + jump_offset(n_req));
  const int rgrid = (n_req + TB - 1) / TB;
  hipLaunchKernelGGL(offer_clear_kernel, dim3(int((ns + TB - 1) / TB < 4096 ? (ns + TB - 1) / TB : 4096)), dim3(TB), 0,
                     stream, t, ns);
  hipLaunchKernelGGL(offer_kernel, dim3(rgrid), dim3(TB), 0, stream, keys, blk_off, n_req, n_blocks, user, turn, t, ns,
                     status);
  hipLaunchKernelGGL(query_kernel, dim3((n_req + TB / 64 - 1) / (TB / 64)), dim3(TB), 0, stream, keys, blk_off, n_req,
                     n_blocks, user, turn, t, ns, parent, jump);
  // rounds: every chain is shorter than n_req, and each round doubles the distance covered
  int rounds = 1;
  while ((int64_t(1) << rounds) < int64_t(n_req)) ++rounds;
  int32_t *a = jump, *b = session;
  for (int k = 0; k < rounds; ++k) {
    hipLaunchKernelGGL(jump_kernel, dim3(rgrid), dim3(TB), 0, stream, a, b, n_req);
    int32_t *tmp = a;
    a = b;
    b = tmp;
  }
  // one more round lands the result in `session` (a round at the fixed point changes nothing)
  if (a != session) hipLaunchKernelGGL(jump_kernel, dim3(rgrid), dim3(TB), 0, stream, a, session, n_req);
  return hip_rc(hipGetLastError());
}
