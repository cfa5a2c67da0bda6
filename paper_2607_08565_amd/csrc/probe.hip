// Region-ordered probe of every block of a batch (K3, shared by match and insert).
//
// Paper: c_i is the prefix hit of the prompt in instance i's local KV$ (Sec. 4.1); after
// routing, the target caches every block (Sec. 2, 4.2).  Both steps ask the index the
// same question per block -- which instances hold this key -- so it is asked once.
//
// Mapping to gfx950.  Probes are random 128-byte reads over a table of several GB.  On
// MI355X such reads run at ~44 G lines/s while the lines in flight stay inside ~2 GiB and
// drop to 10-14 G lines/s over 4-9 GiB (the reach of the address-translation caches), so
// the batch's blocks are first partitioned by table region (NREG equal bucket ranges, each
// well inside that reach), with no global atomics:
//   requests  one wavefront per request checks the tiling and records each block's request
//   count     PART_WG workgroups, one contiguous chunk of blocks each: LDS histogram of
//             regions -> one row of the [chunk][region] matrix, plus region totals; a
//             key equal to a reserved value (the table's EMPTY or TOMB marker) is flagged
//   scan      one workgroup per region: its first position, then running offsets over
//             chunks -> first position of every (chunk, region) pair
//   scatter   each chunk again, one tile at a time: regrouped by region in LDS, then
//             (key, request) written as one contiguous run per region at its region-order
//             position, and the inverse index block -> position
//   probe     a fixed grid of FLAT_WG workgroups walks the region-ordered keys; all
//             workgroups advance through the regions together, so the live window slides
//             through the table.  One 128-byte bucket read (keys and values at once) per
//             bucket of the key's chain -- its home bucket, and when that is full the
//             buckets its displacement mask names -- gives a 64-bit holder descriptor,
//             written in region order.
// Requests must tile [0, n_blocks): blk_off[0] = 0, non-decreasing, blk_off[n_req] =
// n_blocks; otherwise the probe state is marked invalid (EINVAL).
#include "common.h"

namespace smk {
namespace {

constexpr int TB = WG_THREADS;

__global__ void zero_kernel(uint64_t *p, uint64_t n_words) {
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n_words; i += stride) p[i] = 0;
}

// two ranges cleared by one launch
__global__ void zero2_kernel(uint64_t *p, uint64_t n_words, uint64_t *p2, uint64_t n_words2) {
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n_words + n_words2; i += stride) {
    if (i < n_words) p[i] = 0;
    else p2[i - n_words] = 0;
  }
}

__global__ __launch_bounds__(64) void req_of_kernel(ProbeView pv, const int64_t *__restrict__ blk_off, int32_t n_req,
                                                    int64_t n_blocks) {
  const int r = blockIdx.x, lane = threadIdx.x;
  const int64_t b0 = blk_off[r], b1 = blk_off[r + 1];
  const bool ok = b0 >= 0 && b0 <= b1 && b1 <= n_blocks && (r > 0 || b0 == 0) && (r + 1 < n_req || b1 == n_blocks);
  if (!ok) {
    if (lane == 0) atomicCAS(&pv.hdr->err, 0, SMETRIC_EINVAL);
    return;
  }
  for (int64_t b = b0 + lane; b < b1; b += 64) pv.req_of[b] = uint32_t(r);
}

__device__ __forceinline__ void chunk_of(uint64_t n, uint64_t &lo, uint64_t &hi) {
  const uint64_t c = (n + PART_WG - 1) / PART_WG;
  lo = uint64_t(blockIdx.x) * c;
  hi = lo + c < n ? lo + c : n;
  if (lo > n) lo = n;
}

// Exclusive scan of one value per thread over a TB-thread workgroup; `wt` holds TB / 64
// wave totals.  Every thread returns its prefix; *total gets the sum.
__device__ __forceinline__ uint32_t wg_exclusive_scan(uint32_t v, uint32_t *wt, uint32_t *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) wt[wave] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < TB / 64; ++i) {
    const uint32_t t = wt[i];
    before += i < wave ? t : 0;
    all += t;
  }
  __syncthreads();  // wt may be reused by the caller
  *total = all;
  return before + x - v;
}

// Items per thread and per tile of the partition loops: U independent loads in flight.
constexpr int U = 8;
constexpr int TILE = U * TB;
// The scatter uses tiles of UW * TB blocks, so that each region's run per tile is longer.
constexpr int UW = 16;
constexpr int TILE_W = UW * TB;

__global__ __launch_bounds__(TB) void part_count_kernel(DevIndex ix, ProbeView pv, const uint64_t *__restrict__ keys,
                                                        uint64_t n) {
  __shared__ unsigned int h[NREG];
  for (int g = threadIdx.x; g < NREG; g += TB) h[g] = 0;
  __syncthreads();
  uint64_t lo, hi;
  chunk_of(n, lo, hi);
  bool bad = false;
  for (uint64_t t0 = lo; t0 < hi; t0 += TILE) {
    uint64_t k[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint64_t b = t0 + u * TB + threadIdx.x;
      k[u] = b < hi ? keys[b] : 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (t0 + u * TB + threadIdx.x < hi) {
        atomicAdd(&h[region_of(k[u], ix.n_buckets, ix.nb_inv)], 1u);
        bad |= k[u] == KEY_EMPTY || k[u] == KEY_TOMB;
      }
  }
  if (bad) atomicOr(&pv.hdr->bad_key, 1);
  __syncthreads();
  for (int g = threadIdx.x; g < NREG; g += TB) pv.hist[uint64_t(blockIdx.x) * NREG + g] = h[g];
}

// Workgroup g: first position of region g (the blocks of every region before it, summed
// over all chunks), then the running offsets of its chunks, and its own total.
static_assert(PART_WG == 4 * TB, "each thread of the scan covers 4 chunks");
__global__ __launch_bounds__(TB) void part_scan_kernel(ProbeView pv) {
  __shared__ uint32_t wt[TB / 64];
  __shared__ unsigned long long red[TB / 64];
  const int g = blockIdx.x, t = threadIdx.x;
  unsigned long long v = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    for (int i = 0; i < g; ++i) v += pv.hist[uint64_t(4 * t + j) * NREG + i];
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  if ((t & 63) == 0) red[t >> 6] = v;
  __syncthreads();
  unsigned long long off = 0;
#pragma unroll
  for (int i = 0; i < TB / 64; ++i) off += red[i];
  uint32_t c[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) c[j] = pv.hist[uint64_t(4 * t + j) * NREG + g];
  uint32_t total;
  uint32_t acc = wg_exclusive_scan(c[0] + c[1] + c[2] + c[3], wt, &total);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    pv.base[uint64_t(4 * t + j) * NREG + g] = off + acc;
    acc += c[j];
  }
  if (t == 0) pv.hdr->tot[g] = total;
  if (g == NREG - 1 && t == 0) pv.hdr->n = pv.hdr->err ? 0 : off + total;
}

// Workgroup w moves its chunk into region order one tile at a time: LDS counts and ranks
// per region, the tile regrouped by region in LDS, then each region's part written as one
// contiguous run after the previous tile's.
static_assert(NREG <= TB && NREG <= 256, "one region per thread, region ids in a byte");
__global__ __launch_bounds__(TB) void part_scatter_kernel(DevIndex ix, ProbeView pv, const uint64_t *__restrict__ keys,
                                                          uint64_t n) {
  __shared__ unsigned long long run[NREG];
  __shared__ uint32_t cnt[NREG], tstart[NREG], wt[TB / 64];
  __shared__ uint64_t skey[TILE_W];
  __shared__ uint32_t sblk[TILE_W], sreq[TILE_W];
  __shared__ uint8_t sg[TILE_W];
  if (pv.hdr->err) return;
  const int t = threadIdx.x;
  if (t < NREG) {
    run[t] = pv.base[uint64_t(blockIdx.x) * NREG + t];
    cnt[t] = 0;
  }
  __syncthreads();
  uint64_t lo, hi;
  chunk_of(n, lo, hi);
  for (uint64_t t0 = lo; t0 < hi; t0 += TILE_W) {
    uint64_t k[UW];
    uint32_t r[UW], rk[UW];
    uint8_t g[UW];
#pragma unroll
    for (int u = 0; u < UW; ++u) {
      const uint64_t b = t0 + u * TB + t;
      k[u] = b < hi ? keys[b] : 0;
      r[u] = b < hi ? pv.req_of[b] : 0;
    }
#pragma unroll
    for (int u = 0; u < UW; ++u) {
      g[u] = uint8_t(region_of(k[u], ix.n_buckets, ix.nb_inv));
      rk[u] = t0 + u * TB + t < hi ? atomicAdd(&cnt[g[u]], 1u) : 0;
    }
    __syncthreads();
    uint32_t total;
    const uint32_t before = wg_exclusive_scan(t < NREG ? cnt[t] : 0u, wt, &total);
    if (t < NREG) tstart[t] = before;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < UW; ++u) {
      const uint64_t b = t0 + u * TB + t;
      if (b < hi) {
        const uint32_t p = tstart[g[u]] + rk[u];
        skey[p] = k[u];
        sblk[p] = uint32_t(b);
        sreq[p] = r[u];
        sg[p] = g[u];
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < UW; ++u) {
      const uint32_t p = u * TB + t;
      if (p < total) {
        const uint32_t gg = sg[p];
        const uint64_t pos = run[gg] + (p - tstart[gg]);
        pv.part_key[pos] = skey[p];
        pv.part_req[pos] = sreq[p];
        pv.part_blk[pos] = sblk[p];
      }
    }
    __syncthreads();
    // the inverse map in block order through LDS (the keys' space is free now), so its
    // stores are coalesced rather than one line per lane
    uint32_t *sinv = reinterpret_cast<uint32_t *>(skey);
#pragma unroll
    for (int u = 0; u < UW; ++u) {
      const uint32_t p = u * TB + t;
      if (p < total) {
        const uint32_t gg = sg[p];
        sinv[sblk[p] - uint32_t(t0)] = uint32_t(run[gg] + (p - tstart[gg]));
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < UW; ++u) {
      const uint32_t p = u * TB + t;
      if (p < total) pv.inv[t0 + p] = sinv[p];
    }
    __syncthreads();
    if (t < NREG) {
      run[t] += cnt[t];
      cnt[t] = 0;
    }
    __syncthreads();
  }
}

// Probe bound.  The match reads a request's blocks only up to its first block that no
// instance holds (c[r][i] = the first block instance i misses, Sec. 4.1), so any block
// that no instance holds bounds the blocks worth probing.  Each request searches for one:
// BL lanes test BL evenly spaced blocks of the open interval (lo, hi) -- lo held by some
// instance (or -1), hi held by none (or the block count) -- and the interval shrinks to
// the first tested block held by none and the tested block before it.  It ends with hi
// held by none (or every tested block held, hi = the block count: nothing is skipped), so
// the first all-miss block lies at or before hi; with whole prompts cached, holding is
// monotone along a prompt and hi is exactly that block.  Blocks from hi on get their bit
// in the skip bitmap: the probe gives them the NONE descriptor without reading the table
// -- right for hi, never read by the match for later ones -- and the insert takes them as
// candidates, its placement turning any that exist (an entry whose ancestors were
// evicted) into a refresh.  Only when the insert cannot overflow the index whatever those
// blocks turn out to be (entries + blocks <= capacity), so that its all-or-nothing
// capacity check stays exact.
constexpr int BL = 4;  // lanes per request
// Workgroups of the probe kernel's grid (measured: 1,536 -- all resident at its register use -- beat 768, 1,024, 2,048, 3,072 and 4,096).
constexpr int PROBE_WG = 1536;
constexpr int PROBE_K = 2;  // keys per thread and iteration

// Is `key` in the table at all (any slot of its home chain)?
__device__ bool key_present(const DevIndex &ix, uint64_t key) {
  ChainWalk w = chain_start(home_bucket(key, ix.n_buckets), key_cls(key));
  bool had_empty;
  do {
    const BucketScan sc = scan_bucket(ix.slots + w.b * BUCKET_WORDS, key);
    if (sc.match) return true;
    had_empty = sc.empty != 0;
  } while (chain_next(ix, w, had_empty));
  return false;
}

__global__ __launch_bounds__(TB) void bound_kernel(DevIndex ix, ProbeView pv, const uint64_t *__restrict__ keys,
                                                   const int64_t *__restrict__ blk_off, int32_t n_req,
                                                   uint64_t n_blocks) {
  if (pv.hdr->err || pv.hdr->n != n_blocks || ix.hdr->n_entries + n_blocks > ix.capacity) return;
  const int lane = threadIdx.x & (BL - 1), gbase = (threadIdx.x & 63) & ~(BL - 1);
  const int64_t r = (int64_t(blockIdx.x) * TB + threadIdx.x) / BL;
  // a request whose range is not inside [0, n_blocks] is not bounded (its blocks are all probed)
  int64_t b0 = 0, nb = 0;
  if (r < n_req) {
    b0 = blk_off[r];
    const int64_t b1 = blk_off[r + 1];
    if (b0 < 0 || b1 < b0 || uint64_t(b1) > n_blocks) b0 = 0;
    else nb = b1 - b0;
  }
  int64_t lo = -1, hi = nb;
  uint32_t probes = 0;
  while (__ballot(hi - lo > 1) != 0) {  // whole wavefronts iterate together
    const int64_t gap = hi - lo - 1, cnt = gap < BL ? gap : BL;
    const bool mine = lane < cnt;
    const int64_t p = mine ? lo + (int64_t(lane) + 1) * (gap + 1) / (cnt + 1) : lo;
    const bool held = mine ? key_present(ix, keys[b0 + p]) : true;
    probes += mine;
    const uint32_t miss = uint32_t(__ballot(mine && !held) >> gbase) & ((1u << BL) - 1u);
    if (gap > 0) {
      if (miss) {
        const int t = __builtin_ctz(miss);
        hi = lo + (int64_t(t) + 1) * (gap + 1) / (cnt + 1);
        lo = t > 0 ? lo + int64_t(t) * (gap + 1) / (cnt + 1) : lo;
      } else {
        lo = lo + cnt * (gap + 1) / (cnt + 1);
      }
    }
  }
  // bits [b0 + hi, b0 + nb) of the (cleared) skip bitmap; edge words are shared with the
  // neighbouring requests
  const uint64_t s0 = uint64_t(b0 + hi), s1 = uint64_t(b0 + nb);
  if (s0 < s1)
    for (uint64_t w = s0 / 32 + lane; w <= (s1 - 1) / 32; w += BL) {
      const uint64_t lo_b = w * 32 > s0 ? w * 32 : s0, hi_b = (w + 1) * 32 < s1 ? (w + 1) * 32 : s1;
      const uint32_t bits = uint32_t(((uint64_t(1) << (hi_b - lo_b)) - 1) << (lo_b - w * 32));
      atomicOr(pv.skip + w, bits);
    }
  // counts for smetric_probe_stats: one atomic per request
  const unsigned long long skip = s0 < s1 ? s1 - s0 : 0;
#pragma unroll
  for (int d = 1; d < BL; d <<= 1) probes += __shfl_xor(probes, d, 64);
  if (lane == 0 && r < n_req) {
    if (s0 < s1) atomicAdd(&pv.hdr->n_skip, skip);
    if (probes) atomicAdd(&pv.hdr->n_search, (unsigned long long)probes);
  }
}

// Holder descriptor of a key, built bucket by bucket over the key's chain -- its home
// bucket, and only when that is full the buckets its displacement mask names.  A bucket's
// keys (its first 64 bytes) are read first; the value of a slot that holds the key is then
// read from the same line (an L2 hit), so a walk keeps only the keys in registers.
struct DescWalk {
  uint64_t key, first_slot;
  uint32_t cnt, first_inst;
  bool done;     // descriptor final
  bool pending;  // cw.b is the next bucket to fold
  uint64_t out;
  ChainWalk cw;
};

__device__ __forceinline__ void keys_load(const DevIndex &ix, uint64_t b, ulonglong2 kk[SLOTS / 2]) {
  const ulonglong2 *p = reinterpret_cast<const ulonglong2 *>(ix.slots + b * BUCKET_WORDS);
#pragma unroll
  for (int i = 0; i < SLOTS / 2; ++i) kk[i] = p[i];
}

__device__ __forceinline__ void desc_init(DescWalk &w, uint64_t key, uint64_t h) {
  w.key = key;
  w.cnt = 0;
  w.first_inst = 0;
  w.first_slot = 0;
  w.done = false;
  w.pending = false;
  w.out = 0;
  w.cw = chain_start(h, key_cls(key));
}

// Slots of bucket keys kk holding `key` (before the first EMPTY slot) and whether an EMPTY
// slot is there.
struct KeyScan {
  uint32_t match;
  bool empty;
};
__device__ __forceinline__ KeyScan scan_keys(const ulonglong2 kk[SLOTS / 2], uint64_t key) {
  uint32_t m = 0, e = 0;
#pragma unroll
  for (int i = 0; i < SLOTS / 2; ++i) {
    m |= (uint32_t(kk[i].x == key) << (2 * i)) | (uint32_t(kk[i].y == key) << (2 * i + 1));
    e |= (uint32_t(kk[i].x == KEY_EMPTY) << (2 * i)) | (uint32_t(kk[i].y == KEY_EMPTY) << (2 * i + 1));
  }
  if (e) m &= (e & (0u - e)) - 1u;
  return KeyScan{m, e != 0};
}

// The value word the fold of bucket b needs first: the first slot holding the key (slot 0
// when none does: a read of the same line, then unused).
__device__ __forceinline__ uint64_t first_val(const DevIndex &ix, uint64_t b, uint32_t match) {
  return ix.slots[b * BUCKET_WORDS + SLOTS + (match ? __builtin_ctz(match) : 0)];
}

// Fold bucket w.cw.b (its key matches and the first matching value) into the walk.
__device__ __forceinline__ void desc_fold(const DevIndex &ix, DescWalk &w, uint32_t match, uint64_t v0) {
  const uint64_t b = w.cw.b;
  bool first = true;
  while (match && !w.done) {
    const int s = __builtin_ctz(match);
    match &= match - 1;
    const uint64_t v = first ? v0 : ix.slots[b * BUCKET_WORDS + SLOTS + s];  // two or more: rare
    first = false;
    const uint32_t kind = val_kind(v);
    if (kind == HEADER) {
      w.out = make_desc(D_HOT, 0, val_rec(v));
      w.done = true;
    } else if (kind == PLAIN) {
      if (w.cnt == 0) {
        w.first_inst = val_inst(v);
        w.first_slot = b * SLOTS + s;
      }
      ++w.cnt;
    }
  }
}

__device__ __forceinline__ void desc_close(DescWalk &w) {
  if (w.done) return;
  w.done = true;
  w.out = w.cnt == 0 ? make_desc(D_NONE, 0, 0)
                     : (w.cnt == 1 ? make_desc(D_ONE, w.first_inst, w.first_slot) : make_desc(D_MANY, 0, 0));
}

// Each thread describes PK keys of the same iteration (positions i + u TB); a block past
// its request's probe bound gets NONE without a read.  All home buckets' keys are
// requested before any is examined, then all first matching values; a key whose home
// bucket is full (about a third at 3/4 occupancy) then reads its mask -- all masks
// requested together -- and the buckets the masks name (under a fifth of the keys) are
// read one per key per round.  Loads are unconditional: a lane with nothing to read for a
// key reads bucket 0 (or its mask), one line that stays cached.
template <int PK>
__global__ __launch_bounds__(TB) void probe_kernel(DevIndex ix, ProbeView pv) {
  const uint64_t n = pv.hdr->n;
  const uint64_t span = uint64_t(gridDim.x) * PK * TB;
  for (uint64_t i = uint64_t(blockIdx.x) * PK * TB + threadIdx.x; i < n; i += span) {
    uint64_t key[PK], h[PK];
    bool has[PK], skip[PK];
#pragma unroll
    for (int u = 0; u < PK; ++u) {
      const uint64_t q = i + uint64_t(u) * TB;
      has[u] = q < n;
      key[u] = pv.part_key[has[u] ? q : i];
    }
    uint32_t sw[PK], blk[PK];
#pragma unroll
    for (int u = 0; u < PK; ++u) {
      blk[u] = pv.part_blk[has[u] ? i + uint64_t(u) * TB : i];
      sw[u] = pv.skip[blk[u] >> 5];
    }
    DescWalk w[PK];
    bool any = false;
#pragma unroll
    for (int u = 0; u < PK; ++u) {
      skip[u] = !has[u] || ((sw[u] >> (blk[u] & 31)) & 1u);
      h[u] = home_bucket(key[u], ix.n_buckets);
      desc_init(w[u], key[u], h[u]);
      any |= !skip[u];
    }
    bool e[PK];
#pragma unroll
    for (int u = 0; u < PK; ++u) e[u] = true;  // a skipped block: no entries, as far as the walk goes
    if (any) {
      ulonglong2 kk[PK][SLOTS / 2];
#pragma unroll
      for (int u = 0; u < PK; ++u) keys_load(ix, skip[u] ? 0 : h[u], kk[u]);
      KeyScan sc[PK];
      uint64_t v[PK];
#pragma unroll
      for (int u = 0; u < PK; ++u) {
        sc[u] = scan_keys(kk[u], key[u]);
        v[u] = first_val(ix, skip[u] ? 0 : h[u], skip[u] ? 0u : sc[u].match);
      }
#pragma unroll
      for (int u = 0; u < PK; ++u)
        if (!skip[u]) {
          desc_fold(ix, w[u], sc[u].match, v[u]);
          e[u] = sc[u].empty;
        }
    }
    bool need[PK], any_need = false;
#pragma unroll
    for (int u = 0; u < PK; ++u) {
      need[u] = !w[u].done && !e[u];
      any_need |= need[u];
    }
    if (any_need) {
      uint32_t m[PK];
#pragma unroll
      for (int u = 0; u < PK; ++u) m[u] = mask_get(ix, need[u] ? h[u] : 0);
#pragma unroll
      for (int u = 0; u < PK; ++u) chain_set_mask(w[u].cw, m[u]);
    }
    bool pending = false;
#pragma unroll
    for (int u = 0; u < PK; ++u) {
      w[u].pending = need[u] && chain_next(ix, w[u].cw, false);
      if (!w[u].pending) desc_close(w[u]);
      pending |= w[u].pending;
    }
    while (pending) {
      uint64_t bb[PK];
      ulonglong2 kk[PK][SLOTS / 2];
#pragma unroll
      for (int u = 0; u < PK; ++u) {
        bb[u] = w[u].pending ? w[u].cw.b : 0;
        keys_load(ix, bb[u], kk[u]);
      }
      KeyScan sc[PK];
      uint64_t v[PK];
#pragma unroll
      for (int u = 0; u < PK; ++u) {
        sc[u] = scan_keys(kk[u], key[u]);
        v[u] = first_val(ix, bb[u], w[u].pending ? sc[u].match : 0u);
      }
      pending = false;
#pragma unroll
      for (int u = 0; u < PK; ++u)
        if (w[u].pending) {
          desc_fold(ix, w[u], sc[u].match, v[u]);
          w[u].pending = !w[u].done && chain_next(ix, w[u].cw, sc[u].empty);
          if (!w[u].pending) desc_close(w[u]);
          pending |= w[u].pending;
        }
    }
#pragma unroll
    for (int u = 0; u < PK; ++u)
      if (has[u]) pv.desc_p[i + uint64_t(u) * TB] = w[u].out;
  }
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_probe_ws_bytes(int64_t n_blocks, uint64_t *bytes) {
  if (n_blocks < 0 || n_blocks >= (int64_t(1) << 32) || !bytes) return SMETRIC_EINVAL;
  *bytes = probe_layout(n_blocks, nullptr, nullptr);
  return SMETRIC_OK;
}

namespace {
int probe_args(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
               int64_t n_blocks, void *probe, uint64_t probe_bytes) {
  if (!idx || !idx->slots || n_req < 0 || n_blocks < 0 || n_blocks >= (int64_t(1) << 32)) return SMETRIC_EINVAL;
  if (!blk_off || (n_blocks > 0 && !keys) || (n_req == 0 && n_blocks != 0)) return SMETRIC_EINVAL;
  if (!probe || (reinterpret_cast<uintptr_t>(probe) & 255) || probe_bytes < probe_layout(n_blocks, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  return SMETRIC_OK;
}
}  // namespace

namespace smk {
int probe_state_args(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                     int64_t n_blocks, void *probe, uint64_t probe_bytes) {
  return probe_args(idx, keys, blk_off, n_req, n_blocks, probe, probe_bytes);
}

void partition_head(ProbeView &pv, bool clear_hist, hipStream_t stream) {
  hipLaunchKernelGGL(zero2_kernel, dim3(16), dim3(TB), 0, stream, reinterpret_cast<uint64_t *>(pv.hdr),
                     uint64_t(sizeof(ProbeHdr) / 8), reinterpret_cast<uint64_t *>(pv.hist),
                     clear_hist ? uint64_t(PART_WG) * NREG / 2 : uint64_t(0));
}

int partition_tail(const DevIndex &ix, ProbeView &pv, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                   uint64_t n, bool counted, hipStream_t stream) {
  // launched after the hash in the fused call, so that the hash starts right after the clear
  if (n_req > 0)
    hipLaunchKernelGGL(req_of_kernel, dim3(n_req), dim3(64), 0, stream, pv, blk_off, n_req, int64_t(n));
  if (!counted) hipLaunchKernelGGL(part_count_kernel, dim3(PART_WG), dim3(TB), 0, stream, ix, pv, keys, n);
  hipLaunchKernelGGL(part_scan_kernel, dim3(NREG), dim3(TB), 0, stream, pv);
  hipLaunchKernelGGL(part_scatter_kernel, dim3(PART_WG), dim3(TB), 0, stream, ix, pv, keys, n);
  return hip_rc(hipGetLastError());
}
}  // namespace smk

extern "C" int smetric_probe_partition(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off,
                                       int32_t n_req, int64_t n_blocks, void *probe, uint64_t probe_bytes,
                                       hipStream_t stream) {
  if (int rc = probe_args(idx, keys, blk_off, n_req, n_blocks, probe, probe_bytes)) return rc;
  ProbeView pv;
  probe_layout(n_blocks, &pv, probe);
  const DevIndex ix = dev_view(idx);  // geometry only: the table's contents are not read here
  partition_head(pv, false, stream);
  return partition_tail(ix, pv, keys, blk_off, n_req, uint64_t(n_blocks), false, stream);
}

extern "C" int smetric_probe_lookup(const smetric_index *idx, void *probe, uint64_t probe_bytes,
                                    const uint64_t *keys, const int64_t *blk_off, int32_t n_req, int64_t n_blocks,
                                    hipStream_t stream) {
  if (!idx || !idx->slots || n_req < 0 || n_blocks < 0 || n_blocks >= (int64_t(1) << 32)) return SMETRIC_EINVAL;
  if (!blk_off || (n_blocks > 0 && !keys)) return SMETRIC_EINVAL;
  if (!probe || (reinterpret_cast<uintptr_t>(probe) & 255) || probe_bytes < probe_layout(n_blocks, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  ProbeView pv;
  probe_layout(n_blocks, &pv, probe);
  const DevIndex ix = dev_view(idx);
  const uint64_t nw = skip_words(uint64_t(n_blocks < 1 ? 1 : n_blocks));
  // the skip bitmap (whole 64-bit words: its allocation is rounded up to 256 bytes) and
  // the probe counters, one launch
  hipLaunchKernelGGL(zero2_kernel, dim3(nw / TB + 1 < 256 ? nw / TB + 1 : 256), dim3(TB), 0, stream,
                     reinterpret_cast<uint64_t *>(pv.skip), (nw + 1) / 2,
                     reinterpret_cast<uint64_t *>(&pv.hdr->n_skip), uint64_t(2));
  if (n_req > 0 && n_blocks > 0)
    hipLaunchKernelGGL(bound_kernel, dim3((uint64_t(n_req) * BL + TB - 1) / TB), dim3(TB), 0, stream, ix, pv, keys,
                       blk_off, n_req, uint64_t(n_blocks));
  hipLaunchKernelGGL(probe_kernel<PROBE_K>, dim3(PROBE_WG), dim3(TB), 0, stream, ix, pv);
  return hip_rc(hipGetLastError());
}

extern "C" int smetric_probe_stats(const void *probe, uint64_t probe_bytes, int64_t n_blocks, uint64_t *n_probed,
                                   uint64_t *n_search, hipStream_t stream) {
  if (n_blocks < 0 || n_blocks >= (int64_t(1) << 32) || !n_probed || !n_search) return SMETRIC_EINVAL;
  if (!probe || (reinterpret_cast<uintptr_t>(probe) & 255) || probe_bytes < probe_layout(n_blocks, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  ProbeView pv;
  probe_layout(n_blocks, &pv, const_cast<void *>(probe));
  ProbeHdr h;
  if (hipMemcpyAsync(&h, pv.hdr, sizeof(h), hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return SMETRIC_EHIP;
  *n_probed = h.n >= h.n_skip ? h.n - h.n_skip : 0;
  *n_search = h.n_search;
  return SMETRIC_OK;
}

extern "C" int smetric_probe(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                             int64_t n_blocks, void *probe, uint64_t probe_bytes, hipStream_t stream) {
  if (int rc = smetric_probe_partition(idx, keys, blk_off, n_req, n_blocks, probe, probe_bytes, stream)) return rc;
  return smetric_probe_lookup(idx, probe, probe_bytes, keys, blk_off, n_req, n_blocks, stream);
}
