// Block split + chained 64-bit block keys (K1).
//
// Paper: a prompt is identified at KV$-block granularity by its chained block hashes
// (Sec. 3.1; App. A).  The function is the SMH64-v1 reading stated in smetric.h:
// SplitMix64 constants, the NH digest of each block, a position salt, an affine chain
// s_j = M s_{j-1} + e_j and a finalised key.
//
// Mapping to gfx950: requests are cut into tiles of 64 blocks.
//  * B = 16 (the fast path): one workgroup of eight wavefronts per request, wavefront w
//    taking tiles w, w + 8, ... and loading its next tile while it hashes the current one,
//    so long prompts do not serialise on one wavefront.  Tokens are read as 16-byte
//    vectors, lane l of load u taking tokens [256u + 4l, 256u + 4l + 4) of the tile, so
//    every load instruction covers 1 KB of contiguous HBM.  Four lanes share a block;
//    each forms the NH products of its two token pairs and a quad reduction (DPP quad
//    permutes) yields the block digest.
//  * other even B: one wavefront per request; lane l digests block l of the tile.
//  Digests go through LDS so that lane l then owns block l of the tile; the chain is an
//  inclusive scan of affine maps x -> M x + e_l across the wavefront, done with DPP moves
//  (row shifts, then the row broadcasts) and per-lane powers of M.  A tile's carry-in composes the affine maps of
//  the tiles before it.  Because the chain is affine, this equals the sequential
//  definition exactly.
#include "common.h"

namespace smk {
namespace {

constexpr uint64_t GOLDEN = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t finalise(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
// Output t (0-based) of the SplitMix64 stream seeded with `seed`: the Weyl state after
// t+1 steps is seed + (t+1) * golden, so outputs can be formed independently.
__device__ __forceinline__ uint64_t splitmix_out(uint64_t seed, uint64_t t) {
  return finalise(seed + (t + 1) * GOLDEN);
}

template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  int lo = __builtin_amdgcn_mov_dpp(int(uint32_t(v)), CTRL, 0xF, 0xF, false);
  int hi = __builtin_amdgcn_mov_dpp(int(uint32_t(v >> 32)), CTRL, 0xF, 0xF, false);
  return (uint64_t(uint32_t(hi)) << 32) | uint32_t(lo);
}

__device__ __forceinline__ uint64_t readlane64u(uint64_t v, int l) {
  return (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v >> 32)), l))) << 32) |
         uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v)), l));
}

__device__ __forceinline__ uint64_t remap(uint64_t k) {
  if (k == KEY_EMPTY) return 1;
  if (k == KEY_TOMB) return KEY_TOMB - 1;
  return k;
}

struct ChainConsts {
  uint64_t M;
  uint64_t s_init;
  uint64_t Mpow[6];  // M^1, M^2, M^4, ..., M^32
  uint64_t Mlane;    // M^(lane+1)
  uint64_t Mrow;     // M^(lane % 16 + 1): joins a row to the last lane of the row before
  uint64_t Mhalf;    // M^(lane - 31) for lanes 32..63: joins them to lane 31
};

__device__ __forceinline__ uint64_t mpow(const uint64_t Mpow[6], uint32_t e) {
  uint64_t r = 1;
#pragma unroll
  for (int k = 0; k < 6; ++k)
    if ((e >> k) & 1) r *= Mpow[k];
  return r;
}

// The constants every lane shares (kernel arguments only: scalar registers).
__device__ ChainConsts chain_uniform(uint64_t seed, int B) {
  ChainConsts c;
  c.M = splitmix_out(seed, B) | 1ull;
  c.s_init = splitmix_out(seed, B + 1);
  uint64_t p = c.M;
  for (int k = 0; k < 6; ++k) {
    c.Mpow[k] = p;
    p *= p;
  }
  return c;
}
// This lane's powers, by binary exponentiation (exponents 1..64).
__device__ void chain_lanes(ChainConsts &c) {
  const uint32_t lane = threadIdx.x & 63;
  c.Mlane = lane == 63 ? c.Mpow[5] * c.Mpow[5] : mpow(c.Mpow, lane + 1);
  c.Mrow = mpow(c.Mpow, (lane & 15) + 1);
  c.Mhalf = mpow(c.Mpow, lane >= 32 ? lane - 31 : 1);
}
__device__ ChainConsts chain_consts(uint64_t seed, int B) {
  ChainConsts c = chain_uniform(seed, B);
  chain_lanes(c);
  return c;
}

// DPP move of a 64-bit value (both halves with the same control); lanes the control
// gives no source, and rows outside ROW_MASK, read 0.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ uint64_t dpp_take64(uint64_t v) {
  const int lo = __builtin_amdgcn_update_dpp(0, int(uint32_t(v)), CTRL, ROW_MASK, 0xF, true);
  const int hi = __builtin_amdgcn_update_dpp(0, int(uint32_t(v >> 32)), CTRL, ROW_MASK, 0xF, true);
  return (uint64_t(uint32_t(hi)) << 32) | uint32_t(lo);
}

// Inclusive scan of the affine maps x -> M x + v_l across the wavefront, in DPP only:
// returns sum_{k <= l} M^(l-k) v_k.  Distances 1, 2, 4, 8 inside each row of 16 lanes
// (row_shr), then rows 1 and 3 take the last lane of the row before (row_bcast:15), then
// lanes 32..63 take lane 31 (row_bcast:31).
__device__ __forceinline__ uint64_t affine_scan64(uint64_t v, const ChainConsts &cc) {
  v += cc.Mpow[0] * dpp_take64<0x111>(v);  // row_shr:1
  v += cc.Mpow[1] * dpp_take64<0x112>(v);  // row_shr:2
  v += cc.Mpow[2] * dpp_take64<0x114>(v);  // row_shr:4
  v += cc.Mpow[3] * dpp_take64<0x118>(v);  // row_shr:8
  v += cc.Mrow * dpp_take64<0x142, 0xA>(v);   // row_bcast:15 into rows 1 and 3
  v += cc.Mhalf * dpp_take64<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  return v;
}

// Given lane l's block digest for block j = j0 + l (valid when l < n_valid), finish the
// tile: salt, chain scan from `carry`, finalise, store.  Returns the chain state after
// the tile's last block (meaningful when the tile is full).
__device__ __forceinline__ uint64_t finish_tile(uint64_t d, int64_t j0, int n_valid, uint64_t carry,
                                                const ChainConsts &cc, uint64_t *out) {
  const int lane = threadIdx.x & 63;
  const int64_t j = j0 + lane;
  const uint64_t v = affine_scan64(lane < n_valid ? finalise(d + uint64_t(j)) : 0, cc);
  const uint64_t s = cc.Mlane * carry + v;  // s_j = M^(l+1) carry + sum_k M^(l-k) e_k
  if (lane < n_valid) out[lane] = remap(finalise(s));
  return uint64_t(__shfl(int64_t(s), 63, 64));
}

__device__ __forceinline__ bool request_ok(const int64_t *tok_off, const int64_t *blk_off, int r,
                                           int64_t n_tokens, int64_t n_blocks, int B, int64_t &t0,
                                           int64_t &b0, int64_t &nb) {
  t0 = tok_off[r];
  const int64_t t1 = tok_off[r + 1];
  b0 = blk_off[r];
  const int64_t b1 = blk_off[r + 1];
  nb = b1 - b0;
  return t0 >= 0 && t0 <= t1 && t1 <= n_tokens && b0 >= 0 && b0 <= b1 && b1 <= n_blocks &&
         nb == (t1 - t0) / B;
}

constexpr int WAVES = 1;  // wavefronts per workgroup of the generic kernel

// B = 16 fast path: one workgroup of NW wavefronts per request.  Step k covers tiles
// [k NW, k NW + NW): wavefront w digests tile k NW + w and scans it from a zero state;
// the tiles' aggregates meet in LDS, and wavefront w's carry-in is the step's carry
// advanced through the aggregates of the tiles before its own (x -> M^64 x + agg, as
// every tile before the request's last is full).  Each wavefront loads its next tile's
// tokens before working on the current one.
constexpr int HASH_NW = 8;  // wavefronts per request of the B = 16 kernel

struct Tile16 {
  int4 v[4];
};

__device__ __forceinline__ void load_tile16(const int32_t *x, int64_t tile, int64_t nb, int q, int lane, Tile16 &t) {
  const int64_t j0 = tile * 64;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int blk = 16 * u + (lane >> 2);
    if (j0 + blk < nb) __builtin_memcpy(&t.v[u], x + (j0 + blk) * 16 + 4 * q, 16);
    else t.v[u] = make_int4(0, 0, 0, 0);
  }
}

// COUNT: also the region partition's count pass -- every key adds one to its (partition
// chunk, table region) cell of `hist` (chunks of clen blocks, as the partition cuts them);
// a request's blocks meet at most two chunks unless it is longer than a chunk, so they are
// counted in LDS and added with one atomic per nonzero cell (the rare rest directly).
template <int NW, bool COUNT>
__global__ __launch_bounds__(64 * NW) void hash16_kernel(const int32_t *__restrict__ tokens,
                                                         int64_t n_tokens,
                                                         const int64_t *__restrict__ tok_off,
                                                         const int64_t *__restrict__ blk_off,
                                                         int32_t n_req, int64_t n_blocks,
                                                         uint64_t seed,
                                                         uint64_t *__restrict__ keys,
                                                         int32_t *status,
                                                         uint32_t *__restrict__ hist, uint64_t n_buckets,
                                                         uint64_t nb_inv, uint64_t clen, int *probe_err) {
  __shared__ uint64_t dig[NW][64];
  __shared__ uint64_t agg[NW];
  __shared__ unsigned int lh[COUNT ? 2 * NREG : 1];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x;
  int64_t t0, b0, nb;
  if (!request_ok(tok_off, blk_off, r, n_tokens, n_blocks, 16, t0, b0, nb)) {
    if (threadIdx.x == 0 && status) atomicCAS(status, 0, SMETRIC_EINVAL);
    // counting: this request's blocks are neither written nor counted, so the partition
    // must not run on the counts (it would place more blocks than it reserved)
    if (COUNT && threadIdx.x == 0) atomicCAS(probe_err, 0, SMETRIC_EINVAL);
    return;  // the whole workgroup leaves before any barrier
  }
  static_assert(NW == 2 || NW == 4 || NW == 8 || NW == 16, "the step's carries: an affine scan inside row 0");
  // The chain and digest constants depend on the seed and the lane only: wavefront 0 forms
  // them while every wavefront's first tile is in flight, and the others read them from LDS.
  // (the powers common to all lanes are formed by every wavefront in scalar registers)
  __shared__ uint64_t s_lane[3][64];  // M^(l+1), M^(l % 16 + 1), M^(l - 31)
  __shared__ uint32_t s_k[16];        // K[0 .. 15]
  const int q = lane & 3;
  const int32_t *x = tokens + t0;
  Tile16 cur, nxt;
  load_tile16(x, wave, nb, q, lane, cur);
  ChainConsts cc = chain_uniform(seed, 16);
  if (wave == 0) {
    chain_lanes(cc);
    s_lane[0][lane] = cc.Mlane;
    s_lane[1][lane] = cc.Mrow;
    s_lane[2][lane] = cc.Mhalf;
    if (lane < 16) s_k[lane] = uint32_t(splitmix_out(seed, lane));
  }
  __syncthreads();
  cc.Mlane = s_lane[0][lane];
  cc.Mrow = s_lane[1][lane];
  cc.Mhalf = s_lane[2][lane];
  // powers of a tile's map M^64: M64^1, ^2, ^4, ^8 for the scan over the waves' aggregates,
  // M64^wave for this wave's carry-in and M64^NW for the next step's
  const uint64_t M64 = cc.Mpow[5] * cc.Mpow[5], M128 = M64 * M64, M256 = M128 * M128, M512 = M256 * M256,
                 M1024 = M512 * M512;
  const uint64_t Mw = ((wave & 1) ? M64 : 1ull) * ((wave & 2) ? M128 : 1ull) * ((wave & 4) ? M256 : 1ull) *
                      ((wave & 8) ? M512 : 1ull);
  const uint64_t Mstep = NW == 2 ? M128 : (NW == 4 ? M256 : (NW == 8 ? M512 : M1024));
  // this lane's four offset constants: K[4q .. 4q+3], q = lane % 4
  const uint32_t k0 = s_k[4 * q + 0], k1 = s_k[4 * q + 1], k2 = s_k[4 * q + 2], k3 = s_k[4 * q + 3];
  const int64_t n_tiles = (nb + 63) / 64;
  uint64_t carry = cc.s_init;  // chain state before the step's first block
  const uint64_t c_lo = COUNT ? uint64_t(b0) / clen : 0, B1 = (c_lo + 1) * clen, B2 = B1 + clen;
  if (COUNT && threadIdx.x < 2 * NREG) lh[threadIdx.x] = 0;  // first used after the step's barrier
  for (int64_t step0 = 0; step0 < n_tiles; step0 += NW) {
    const int64_t tile = step0 + wave;
    load_tile16(x, tile + NW, nb, q, lane, nxt);
    const int64_t j0 = tile * 64;
    const int64_t left = nb - j0;
    const int n_valid = int(left <= 0 ? 0 : (left < 64 ? left : 64));
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int4 v = cur.v[u];
      uint64_t part = uint64_t(uint32_t(v.x) + k0) * uint64_t(uint32_t(v.y) + k1) +
                      uint64_t(uint32_t(v.z) + k2) * uint64_t(uint32_t(v.w) + k3);
      part += dpp64<0xB1>(part);  // quad_perm [1,0,3,2]
      part += dpp64<0x4E>(part);  // quad_perm [2,3,0,1]
      if (q == 0) dig[wave][16 * u + (lane >> 2)] = part;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    // local inclusive scan of the tile's affine maps from state 0
    const uint64_t v = affine_scan64(lane < n_valid ? finalise(dig[wave][lane] + uint64_t(j0 + lane)) : 0, cc);
    if (lane == 63) agg[wave] = v;
    __syncthreads();
    // inclusive scan of the tiles' aggregates over lanes 0..NW-1: lane w holds
    // sum_{k <= w} M64^(w-k) agg[k]; wave w starts from M64^w carry + (lane w-1's value)
    uint64_t a = lane < NW ? agg[lane] : 0;
    a += M64 * dpp_take64<0x111>(a);                   // row_shr:1
    if (NW > 2) a += M128 * dpp_take64<0x112>(a);      // row_shr:2
    if (NW > 4) a += M256 * dpp_take64<0x114>(a);      // row_shr:4
    if (NW > 8) a += M512 * dpp_take64<0x118>(a);      // row_shr:8
    const uint64_t before = wave == 0 ? 0 : readlane64u(a, wave - 1);
    const uint64_t c = Mw * carry + before;
    if (lane < n_valid) {
      const uint64_t key = remap(finalise(cc.Mlane * c + v));
      keys[b0 + j0 + lane] = key;
      if (COUNT) {
        const uint64_t b = uint64_t(b0 + j0 + lane);
        const uint32_t g = region_of(key, n_buckets, nb_inv);
        if (b < B2) atomicAdd(&lh[(b >= B1 ? NREG : 0) + g], 1u);
        else atomicAdd(&hist[(b / clen) * NREG + g], 1u);
      }
    }
    carry = Mstep * carry + readlane64u(a, NW - 1);  // used only when every tile of this step was full
    __syncthreads();
    cur = nxt;
  }
  if (COUNT && threadIdx.x < 2 * NREG) {  // the loop ended on a barrier: lh is complete
    const unsigned int v = lh[threadIdx.x];
    if (v) atomicAdd(&hist[(c_lo + threadIdx.x / NREG) * NREG + threadIdx.x % NREG], v);
  }
}

// Any even B in [2, 256].
__global__ __launch_bounds__(64 * WAVES) void hash_generic_kernel(
    const int32_t *__restrict__ tokens, int64_t n_tokens, const int64_t *__restrict__ tok_off,
    const int64_t *__restrict__ blk_off, int32_t n_req, int64_t n_blocks, int B, uint64_t seed,
    uint64_t *__restrict__ keys, int32_t *status) {
  __shared__ uint32_t K[256];
  for (int t = threadIdx.x; t < B; t += blockDim.x) K[t] = uint32_t(splitmix_out(seed, t));
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * WAVES + wave;
  if (r >= n_req) return;
  int64_t t0, b0, nb;
  if (!request_ok(tok_off, blk_off, r, n_tokens, n_blocks, B, t0, b0, nb)) {
    if (lane == 0 && status) atomicCAS(status, 0, SMETRIC_EINVAL);
    return;
  }
  const ChainConsts cc = chain_consts(seed, B);
  const int32_t *x = tokens + t0;
  uint64_t carry = cc.s_init;
  for (int64_t j0 = 0; j0 < nb; j0 += 64) {
    const int n_valid = int(nb - j0 < 64 ? nb - j0 : 64);
    uint64_t d = 0;
    if (lane < n_valid) {
      const int32_t *b = x + (j0 + lane) * B;
      for (int k = 0; k < B / 2; ++k)
        d += uint64_t(uint32_t(b[2 * k]) + K[2 * k]) * uint64_t(uint32_t(b[2 * k + 1]) + K[2 * k + 1]);
    }
    carry = finish_tile(d, j0, n_valid, carry, cc, keys + b0 + j0);
  }
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_hash_blocks(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_off,
                                   const int64_t *blk_off, int32_t n_req, int64_t n_blocks,
                                   int32_t block_size, uint64_t seed, uint64_t *keys,
                                   int32_t *status, hipStream_t stream) {
  if (n_req < 0 || n_tokens < 0 || n_blocks < 0 || block_size < 2 || block_size > 256 ||
      (block_size & 1))
    return SMETRIC_EINVAL;
  if (n_req == 0) return SMETRIC_OK;
  if (!tok_off || !blk_off || (n_tokens > 0 && !tokens) || (n_blocks > 0 && !keys))
    return SMETRIC_EINVAL;
  const dim3 grid((n_req + WAVES - 1) / WAVES), block(64 * WAVES);
  if (block_size == 16)
    hipLaunchKernelGGL((hash16_kernel<HASH_NW, false>), dim3(n_req), dim3(64 * HASH_NW), 0, stream, tokens, n_tokens, tok_off, blk_off,
                       n_req, n_blocks, seed, keys, status, static_cast<uint32_t *>(nullptr), uint64_t(0), uint64_t(0),
                       uint64_t(1), static_cast<int *>(nullptr));
  else
    hipLaunchKernelGGL(hash_generic_kernel, grid, block, 0, stream, tokens, n_tokens, tok_off,
                       blk_off, n_req, n_blocks, int(block_size), seed, keys, status);
  return hip_rc(hipGetLastError());
}

extern "C" int smetric_hash_partition(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_off,
                                      const int64_t *blk_off, int32_t n_req, int64_t n_blocks, int32_t block_size,
                                      uint64_t seed, uint64_t *keys, int32_t *status, const smetric_index *idx,
                                      void *probe, uint64_t probe_bytes, hipStream_t stream) {
  if (n_req < 0 || n_tokens < 0 || n_blocks < 0 || block_size < 2 || block_size > 256 || (block_size & 1))
    return SMETRIC_EINVAL;
  if (n_req > 0 && (!tok_off || (n_tokens > 0 && !tokens))) return SMETRIC_EINVAL;
  if (int rc = probe_state_args(idx, keys, blk_off, n_req, n_blocks, probe, probe_bytes)) return rc;
  ProbeView pv;
  probe_layout(n_blocks, &pv, probe);
  const DevIndex ix = dev_view(idx);  // geometry only
  const bool counted = block_size == 16 && n_req > 0;
  partition_head(pv, counted, stream);
  if (counted)
    hipLaunchKernelGGL((hash16_kernel<HASH_NW, true>), dim3(n_req), dim3(64 * HASH_NW), 0, stream, tokens, n_tokens,
                       tok_off, blk_off, n_req, n_blocks, seed, keys, status, pv.hist, ix.n_buckets, ix.nb_inv,
                       partition_chunk(uint64_t(n_blocks)), &pv.hdr->err);
  else if (n_req > 0)
    hipLaunchKernelGGL(hash_generic_kernel, dim3((n_req + WAVES - 1) / WAVES), dim3(64 * WAVES), 0, stream, tokens,
                       n_tokens, tok_off, blk_off, n_req, n_blocks, int(block_size), seed, keys, status);
  return partition_tail(ix, pv, keys, blk_off, n_req, uint64_t(n_blocks), counted, stream);
}

extern "C" int smetric_block_offsets(const int64_t *tok_off, int32_t n_req, int32_t block_size,
                                     int64_t *blk_off, int64_t *n_blocks) {
  if (n_req < 0 || block_size < 2 || block_size > 256 || (block_size & 1) || !tok_off ||
      !blk_off || !n_blocks)
    return SMETRIC_EINVAL;
  blk_off[0] = 0;
  for (int32_t r = 0; r < n_req; ++r) {
    const int64_t len = tok_off[r + 1] - tok_off[r];
    if (len < 0) return SMETRIC_EINVAL;
    blk_off[r + 1] = blk_off[r] + len / block_size;
  }
  *n_blocks = blk_off[n_req];
  return SMETRIC_OK;
}

extern "C" int smetric_version(void) { return (0 << 16) | 2; }
