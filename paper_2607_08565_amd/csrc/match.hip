// Index probe + first-miss reduction (K3 + K4).
//
// Paper: the router scores instance i by c_i, the prefix hit length of the request's
// prompt in instance i's local KV$ (Sec. 4.1, scoring template), measured at KV$-block
// granularity (Sec. 3.1).  Here c[r][i] = the number of leading blocks of request r
// whose keys instance i holds; an instance drops out at its first missing block.
//
// Mapping to gfx950: one wavefront per request.  The request is walked in chunks of 64
// blocks; lane l probes block j0+l (one 128-byte bucket line per probe, more only when
// a chain spills into the next bucket), collecting the block's holder set as one of
//   NONE, LIST (<= 8 plain holders, kept in registers), HOT (bitmap record in the pool)
//   or LONG (more plain holders than fit the list; re-walked on demand).
// The alive set then shrinks block by block:
//   * NARROW (<= 64 alive): lane t keeps alive instance a_t; per chunk and per alive
//     instance, every lane tests membership in its own block and one ballot finds the
//     first missing block.  This is the common case (a session's private blocks).
//   * WIDE (more alive, e.g. a shared system prefix): the alive bitmap lives in registers,
//     WPL 64-bit words per lane; holder bitmaps of 8 blocks are fetched ahead, then
//     ANDed in block order.  Once <= 64 remain the wave switches to NARROW.
// The output row is zeroed first; an instance is written again only when it drops after
// block 0 or survives to the end.
#include "common.h"

namespace smk {
namespace {

constexpr int MW = 1;        // waves per workgroup
constexpr int LIST_MAX = 8;  // plain holders kept per probe
enum HKind : uint32_t { H_NONE = 0, H_LIST = 1, H_HOT = 2, H_LONG = 3 };

struct Holders {
  uint32_t kind;
  uint32_t h[LIST_MAX];  // LIST members (0xFFFFFFFF when unused)
  uint64_t rec;          // HOT: pool record
};

__device__ __forceinline__ void load_keys(const uint64_t *bk, uint64_t k[SLOTS]) {
  const ulonglong2 *p = reinterpret_cast<const ulonglong2 *>(bk);
#pragma unroll
  for (int i = 0; i < SLOTS / 2; ++i) {
    ulonglong2 v = p[i];
    k[2 * i] = v.x;
    k[2 * i + 1] = v.y;
  }
}

// Walk key's chain and collect its holders.
__device__ Holders probe(const DevIndex &ix, uint64_t key) {
  Holders H;
  H.kind = H_NONE;
  H.rec = 0;
#pragma unroll
  for (int i = 0; i < LIST_MAX; ++i) H.h[i] = 0xFFFFFFFFu;
  uint32_t cnt = 0;
  ChainWalk w = chain_start(home_bucket(key, ix.n_buckets), key_cls(key));
  bool had_empty;
  do {
    const uint64_t *bk = ix.slots + w.b * BUCKET_WORDS;
    uint64_t k[SLOTS];
    load_keys(bk, k);
    uint32_t mm = 0, em = 0;
#pragma unroll
    for (int s = 0; s < SLOTS; ++s) {
      mm |= uint32_t(k[s] == key) << s;
      em |= uint32_t(k[s] == KEY_EMPTY) << s;
    }
    if (em) mm &= (em & (0u - em)) - 1u;  // only slots before the first empty one
    while (mm) {
      const int s = __builtin_ctz(mm);
      mm &= mm - 1;
      const uint64_t v = bk[SLOTS + s];
      const uint32_t kind = val_kind(v);
      if (kind == HEADER) {
        H.kind = H_HOT;
        H.rec = val_rec(v);
        return H;
      }
      if (kind == PLAIN) {
        const uint32_t inst = val_inst(v);
#pragma unroll
        for (int i = 0; i < LIST_MAX; ++i)
          if (cnt == uint32_t(i)) H.h[i] = inst;
        ++cnt;
      }
    }
    had_empty = em != 0;
  } while (chain_next(ix, w, had_empty));
  H.kind = cnt == 0 ? H_NONE : (cnt <= LIST_MAX ? H_LIST : H_LONG);
  return H;
}

// Is (key, inst) a plain entry?  Used for LONG holder sets only.
__device__ bool chain_has(const DevIndex &ix, uint64_t key, uint32_t inst) {
  ChainWalk cw = chain_start(home_bucket(key, ix.n_buckets), key_cls(key));
  bool had_empty;
  do {
    const uint64_t *bk = ix.slots + cw.b * BUCKET_WORDS;
    had_empty = false;
    for (int s = 0; s < SLOTS; ++s) {
      const uint64_t k = bk[s];
      if (k == KEY_EMPTY) {
        had_empty = true;
        break;
      }
      if (k == key) {
        const uint64_t v = bk[SLOTS + s];
        if (val_kind(v) == PLAIN && val_inst(v) == inst) return true;
      }
    }
  } while (chain_next(ix, cw, had_empty));
  return false;
}

// OR into `m` the bits of every plain holder of `key` that fall in word w.
__device__ uint64_t chain_word(const DevIndex &ix, uint64_t key, int w) {
  uint64_t m = 0;
  ChainWalk cw = chain_start(home_bucket(key, ix.n_buckets), key_cls(key));
  bool had_empty;
  do {
    const uint64_t *bk = ix.slots + cw.b * BUCKET_WORDS;
    had_empty = false;
    for (int s = 0; s < SLOTS; ++s) {
      const uint64_t k = bk[s];
      if (k == KEY_EMPTY) {
        had_empty = true;
        break;
      }
      if (k == key) {
        const uint64_t v = bk[SLOTS + s];
        if (val_kind(v) == PLAIN && int(val_inst(v) >> 6) == w) m |= uint64_t(1) << (val_inst(v) & 63);
      }
    }
  } while (chain_next(ix, cw, had_empty));
  return m;
}

__device__ __forceinline__ bool holds(const DevIndex &ix, const Holders &H, uint64_t key, uint32_t a) {
  switch (H.kind) {
    case H_LIST: {
      bool hit = false;
#pragma unroll
      for (int i = 0; i < LIST_MAX; ++i) hit |= H.h[i] == a;
      return hit;
    }
    case H_HOT:
      return (ix.pool[H.rec * uint64_t(ix.words) + (a >> 6)] >> (a & 63)) & 1;
    case H_LONG:
      return chain_has(ix, key, a);
    default:
      return false;
  }
}

__device__ __forceinline__ uint64_t rdl64(uint64_t v, int src) {
  const uint32_t lo = __builtin_amdgcn_readlane(uint32_t(v), src);
  const uint32_t hi = __builtin_amdgcn_readlane(uint32_t(v >> 32), src);
  return (uint64_t(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
  const uint32_t lo = uint32_t(__shfl(int(uint32_t(v)), src, 64));
  const uint32_t hi = uint32_t(__shfl(int(uint32_t(v >> 32)), src, 64));
  return (uint64_t(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int mask) {
  const uint32_t lo = uint32_t(__shfl_xor(int(uint32_t(v)), mask, 64));
  const uint32_t hi = uint32_t(__shfl_xor(int(uint32_t(v >> 32)), mask, 64));
  return (uint64_t(hi) << 32) | lo;
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

// Holder word w of block `src` (a lane of the current chunk) in WIDE mode.
__device__ __forceinline__ uint64_t holder_word(const DevIndex &ix, uint32_t kind, uint64_t rec,
                                                const uint32_t hl[LIST_MAX], uint64_t key, int w) {
  if (w >= ix.words) return 0;
  if (kind == H_HOT) return ix.pool[rec * uint64_t(ix.words) + w];
  if (kind == H_LIST) {
    uint64_t m = 0;
#pragma unroll
    for (int i = 0; i < LIST_MAX; ++i)
      if (hl[i] != 0xFFFFFFFFu && int(hl[i] >> 6) == w) m |= uint64_t(1) << (hl[i] & 63);
    return m;
  }
  if (kind == H_LONG) return chain_word(ix, key, w);
  return 0;
}

// Holder set of a block from its probe descriptor; MANY re-walks the chain.
__device__ __forceinline__ Holders decode(const DevIndex &ix, uint64_t d, uint64_t key) {
  Holders H;
  H.kind = H_NONE;
  H.rec = 0;
#pragma unroll
  for (int i = 0; i < LIST_MAX; ++i) H.h[i] = 0xFFFFFFFFu;
  switch (desc_kind(d)) {
    case D_ONE:
      H.kind = H_LIST;
      H.h[0] = desc_inst(d);
      break;
    case D_HOT:
      H.kind = H_HOT;
      H.rec = desc_x(d);
      break;
    case D_MANY:
      H = probe(ix, key);
      break;
    default:
      break;
  }
  return H;
}

// DESC = false: probe each block's chain here (early exit after the first all-miss
// chunk).  DESC = true: read the descriptors written by the region-ordered probe.
template <int WPL, bool DESC>
__global__ __launch_bounds__(64 * MW) void match_kernel(DevIndex ix, const uint64_t *__restrict__ keys,
                                                        const int64_t *__restrict__ blk_off,
                                                        int32_t n_req, int64_t n_blocks,
                                                        int32_t *__restrict__ matched,
                                                        const uint64_t *__restrict__ desc,
                                                        const uint32_t *__restrict__ inv,
                                                        const ProbeHdr *__restrict__ ph) {
  __shared__ int32_t nlist[MW][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * MW + wave;
  if (r >= n_req) return;
  const int I = ix.n_inst;
  int32_t *row = matched + int64_t(r) * I;
  for (int i = lane; i < I; i += 64) row[i] = 0;
  const int64_t b0 = blk_off[r], b1 = blk_off[r + 1];
  if (!(b0 >= 0 && b0 <= b1 && b1 <= n_blocks) || (DESC && ph->err)) {
    if (lane == 0) set_status(ix.hdr, SMETRIC_EINVAL);
    return;
  }
  const int64_t nb = b1 - b0;
  if (nb == 0) return;

  enum { M_ALL, M_NARROW, M_WIDE, M_DONE };
  int mode = M_ALL;
  int my_inst = -1;   // NARROW: this lane's alive instance
  uint64_t A[WPL];    // WIDE: alive words lane + 64 t (WPL = 1: word wl, in every lane group)
#pragma unroll
  for (int t = 0; t < WPL; ++t) A[t] = 0;
  // WPL = 1 (at most 4,096 instances): the wavefront is cut into groups of lpb lanes (the
  // least power of two >= the bitmap's words); lane (sub, wl) handles word wl of the
  // group's block, so one load instruction fetches the words of bpl = 64 / lpb blocks
  // (4 at 1,024 instances) and every lane group keeps a copy of the alive words.
  const int words = ix.words;
  const int lpb = WPL > 1 ? 64 : (words <= 1 ? 1 : 1 << (32 - __builtin_clz(uint32_t(words - 1))));
  const int bpl = 64 / lpb, sub = lane / lpb, wl = lane % lpb;

  // DESC: descriptors are fetched PF chunks at a time -- positions, then all PF gathers
  // at once -- since a chunk's own work rarely touches memory and the walk is otherwise
  // one round trip per chunk
  constexpr int PF = DESC ? 8 : 1;
  uint64_t dq[PF];
  int left = 0;
  for (int64_t j0 = 0; j0 < nb && mode != M_DONE; j0 += 64) {
    const int64_t j = j0 + lane;
    const bool valid = j < nb;
    if (DESC && left == 0) {
      // indexes clamped to the request's last block, so that the loads need no branches
      // (a branch around a load makes the compiler wait for it on the spot)
      uint32_t at[PF];
#pragma unroll
      for (int k = 0; k < PF; ++k) at[k] = inv[b0 + (j + 64 * k < nb ? j + 64 * k : nb - 1)];
#pragma unroll
      for (int k = 0; k < PF; ++k) dq[k] = desc[at[k]];
#pragma unroll
      for (int k = 0; k < PF; ++k) dq[k] = j + 64 * k < nb ? dq[k] : 0;
      left = PF;
    }
    const uint64_t d_cur = dq[0];
#pragma unroll
    for (int k = 0; k + 1 < PF; ++k) dq[k] = dq[k + 1];
    --left;
    // DESC, NARROW, and every descriptor of the chunk NONE or ONE (a session's private
    // blocks, the common case): "held by a" is read off the descriptor, nothing decoded
    const bool simple = DESC && mode == M_NARROW && !__ballot(valid && desc_kind(d_cur) >= D_MANY);
    Holders H;
    uint64_t key = 0;
    if (valid && !simple) {
      if (DESC) {
        const uint64_t d = d_cur;
        if (desc_kind(d) == D_MANY) key = keys[b0 + j];
        H = decode(ix, d, key);
      } else {
        key = keys[b0 + j];
        H = probe(ix, key);
      }
    } else {
      H.kind = H_NONE;
      H.rec = 0;
#pragma unroll
      for (int i = 0; i < LIST_MAX; ++i) H.h[i] = 0xFFFFFFFFu;
    }
    int jj = 0;
    if (mode == M_ALL) {
      // block 0 fixes the first alive set; everyone else already has c = 0
      const uint32_t kind0 = __builtin_amdgcn_readfirstlane(H.kind);
      if (kind0 == H_NONE) return;
      if (kind0 == H_LIST) {
#pragma unroll
        for (int i = 0; i < LIST_MAX; ++i) {
          const uint32_t v = __builtin_amdgcn_readlane(H.h[i], 0);
          if (lane == i) my_inst = v == 0xFFFFFFFFu ? -1 : int(v);
        }
        mode = M_NARROW;
      } else {
        const uint64_t rec0 = rdl64(H.rec, 0), key0 = rdl64(key, 0);
        uint32_t hl0[LIST_MAX];
#pragma unroll
        for (int i = 0; i < LIST_MAX; ++i) hl0[i] = 0xFFFFFFFFu;
        if constexpr (WPL == 1) {
          A[0] = holder_word(ix, kind0, rec0, hl0, key0, wl);
        } else {
#pragma unroll
          for (int t = 0; t < WPL; ++t) A[t] = holder_word(ix, kind0, rec0, hl0, key0, lane + 64 * t);
        }
        mode = M_WIDE;
      }
      jj = 1;
    }

    if (WPL == 1 && mode == M_WIDE) {
      // groups of GQ loads (GQ x bpl blocks, one round trip); the words of each block are
      // then ANDed in block order, each fetched from its lane group with a shuffle
      constexpr int GQ = 8;
      while (jj < 64 && mode == M_WIDE) {
        uint64_t hq[GQ];
        uint32_t kq[GQ];
#pragma unroll
        for (int q = 0; q < GQ; ++q) {
          const int b = jj + q * bpl + sub;
          const int src = b < 64 ? b : 63;
          const uint32_t kd = uint32_t(__shfl(int(H.kind), src, 64));
          const uint64_t rc = shfl64(H.rec, src);
          kq[q] = (b < 64 && j0 + b < nb) ? kd : uint32_t(H_NONE);
          // no branch around the load: a non-HOT block reads record 0 (always present)
          hq[q] = ix.pool[(kq[q] == H_HOT ? rc : 0) * uint64_t(words) + uint64_t(wl < words ? wl : 0)];
        }
#pragma unroll
        for (int q = 0; q < GQ; ++q) {
          if (kq[q] != H_HOT || wl >= words) hq[q] = 0;
          if (__ballot(kq[q] == H_LIST || kq[q] == H_LONG)) {  // rare: plain holders
            const int b = jj + q * bpl + sub;
            const int src = b < 64 ? b : 63;
            uint32_t hl[LIST_MAX];
#pragma unroll
            for (int i = 0; i < LIST_MAX; ++i) hl[i] = uint32_t(__shfl(int(H.h[i]), src, 64));
            const uint64_t k = shfl64(key, src);
            if (kq[q] == H_LIST || kq[q] == H_LONG) hq[q] = holder_word(ix, kq[q], 0, hl, k, wl);
          }
        }
        const int nblk = GQ * bpl < 64 - jj ? GQ * bpl : 64 - jj;
        // the group's blocks at once: lane (sub, wl) ANDs its words over the loads, the lane
        // groups then combine theirs, so every lane holds word wl of the intersection of the
        // group's blocks in this chunk (one past the request's end reads as empty, so the
        // survivors are written below); if every alive instance holds them all, nobody drops
        // here and the block-by-block AND is skipped
        uint64_t all = ~uint64_t(0);
#pragma unroll
        for (int q = 0; q < GQ; ++q) all &= jj + q * bpl + sub < 64 ? hq[q] : ~uint64_t(0);
        for (int d = lpb; d < 64; d <<= 1) all &= shfl_xor64(all, d);
        if (!__ballot((A[0] & ~all) != 0)) {
          jj += nblk;
          continue;
        }
#pragma unroll
        for (int q = 0; q < GQ; ++q) {
          for (int s2 = 0; s2 < bpl; ++s2) {
            const int t = q * bpl + s2;
            if (t >= nblk) break;
            const uint64_t x = shfl64(hq[q], s2 * lpb + wl);
            const uint64_t n = A[0] & x;
            uint64_t d = A[0] & ~n;
            A[0] = n;
            const int64_t jb = j0 + jj + t;
            if (sub == 0) {
              while (d) {  // blocks past the end count as misses: survivors get nb
                const int bit = __builtin_ctzll(d);
                d &= d - 1;
                row[wl * 64 + bit] = int32_t(jb < nb ? jb : nb);
              }
            }
          }
        }
        jj += nblk;
        const uint32_t cnt = sub == 0 ? uint32_t(__popcll(A[0])) : 0u;
        const uint32_t n_alive = wave_sum(cnt);
        if (n_alive == 0) {
          mode = M_DONE;
        } else if (n_alive <= 64) {
          // hand the survivors to lanes: exclusive prefix of the lead group's counts
          uint32_t pre = cnt;
#pragma unroll
          for (int d = 1; d < 64; d <<= 1) {
            const uint32_t t = __shfl_up(pre, d, 64);
            if (lane >= d) pre += t;
          }
          pre -= cnt;
          uint64_t a = sub == 0 ? A[0] : 0;
          while (a) {
            const int bit = __builtin_ctzll(a);
            a &= a - 1;
            nlist[wave][pre++] = wl * 64 + bit;
          }
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
          my_inst = lane < int(n_alive) ? nlist[wave][lane] : -1;
          __builtin_amdgcn_wave_barrier();
          mode = M_NARROW;
        }
      }
    }

    if (WPL > 1 && mode == M_WIDE) {
      // block by block, G blocks' holder words fetched ahead of the AND chain
      constexpr int G = WPL >= 8 ? 1 : 8 / WPL;
      while (jj < 64 && mode == M_WIDE) {
        uint64_t hw[G][WPL];
        uint32_t kinds[G];
        // bitmap words of all G blocks requested at once, with no branch around the loads
        // (a non-HOT block reads record 0, always present, and discards it), so the
        // group costs one round trip
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const int src = jj + g < 64 ? jj + g : 63;
          const bool in = jj + g < 64 && j0 + jj + g < nb;
          kinds[g] = in ? __builtin_amdgcn_readlane(H.kind, src) : uint32_t(H_NONE);
          const uint64_t rec = kinds[g] == H_HOT ? rdl64(H.rec, src) : 0;
#pragma unroll
          for (int t = 0; t < WPL; ++t) {
            const int w = lane + 64 * t;
            hw[g][t] = ix.pool[rec * uint64_t(ix.words) + uint64_t(w < ix.words ? w : 0)];
          }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
          if (kinds[g] == H_HOT) {
#pragma unroll
            for (int t = 0; t < WPL; ++t)
              if (lane + 64 * t >= ix.words) hw[g][t] = 0;
          } else {
            const int src = jj + g < 64 ? jj + g : 63;
            const uint64_t k = rdl64(key, src);
            uint32_t hl[LIST_MAX];
#pragma unroll
            for (int i = 0; i < LIST_MAX; ++i) hl[i] = __builtin_amdgcn_readlane(H.h[i], src);
#pragma unroll
            for (int t = 0; t < WPL; ++t) hw[g][t] = holder_word(ix, kinds[g], 0, hl, k, lane + 64 * t);
          }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const int64_t jb = j0 + jj + g;
          if (jj + g < 64) {
#pragma unroll
            for (int t = 0; t < WPL; ++t) {
              const uint64_t n = A[t] & hw[g][t];
              uint64_t d = A[t] & ~n;
              A[t] = n;
              const int w = lane + 64 * t;
              while (d) {  // blocks past the end count as misses: survivors get nb
                const int bit = __builtin_ctzll(d);
                d &= d - 1;
                row[w * 64 + bit] = int32_t(jb < nb ? jb : nb);
              }
            }
          }
        }
        jj += G;
        uint32_t cnt = 0;
#pragma unroll
        for (int t = 0; t < WPL; ++t) cnt += __popcll(A[t]);
        const uint32_t n_alive = wave_sum(cnt);
        if (n_alive == 0) {
          mode = M_DONE;
        } else if (n_alive <= 64) {
          // hand the survivors to lanes: exclusive prefix of per-lane counts
          uint32_t pre = cnt;
#pragma unroll
          for (int d = 1; d < 64; d <<= 1) {
            const uint32_t t = __shfl_up(pre, d, 64);
            if (lane >= d) pre += t;
          }
          pre -= cnt;
#pragma unroll
          for (int t = 0; t < WPL; ++t) {
            uint64_t a = A[t];
            while (a) {
              const int bit = __builtin_ctzll(a);
              a &= a - 1;
              nlist[wave][pre++] = (lane + 64 * t) * 64 + bit;
            }
          }
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
          my_inst = lane < int(n_alive) ? nlist[wave][lane] : -1;
          __builtin_amdgcn_wave_barrier();
          mode = M_NARROW;
        }
      }
    }

    if (mode == M_NARROW && jj < 64) {
      // every alive instance: first block of the chunk (at or after jj) it does not hold
      uint64_t alive = __ballot(my_inst >= 0);
      // simple chunks: the lane's single holder, or none (-1)
      const int32_t one = (valid && desc_kind(d_cur) == D_ONE) ? int32_t(desc_inst(d_cur)) : -1;
      while (alive) {
        const int t = __builtin_ctzll(alive);
        alive &= alive - 1;
        const uint32_t a = __builtin_amdgcn_readlane(uint32_t(my_inst), t);
        const bool held = lane < jj || (simple ? one == int32_t(a) : (valid && holds(ix, H, key, a)));
        const uint64_t miss = __ballot(!held);
        if (miss) {
          const int f = __builtin_ctzll(miss);
          if (lane == t) {
            row[a] = int32_t(j0 + f < nb ? j0 + f : nb);
            my_inst = -1;
          }
        }
      }
      if (!__ballot(my_inst >= 0)) mode = M_DONE;
    }
  }
  // survivors of a request whose block count is a multiple of 64
  if (mode == M_NARROW) {
    if (my_inst >= 0) row[my_inst] = int32_t(nb);
  } else if (mode == M_WIDE) {
#pragma unroll
    for (int t = 0; t < WPL; ++t) {
      uint64_t a = (WPL > 1 || sub == 0) ? A[t] : 0;  // WPL = 1: the lead lane group's copy
      const int w = WPL > 1 ? lane + 64 * t : wl;
      while (a) {
        const int bit = __builtin_ctzll(a);
        a &= a - 1;
        row[w * 64 + bit] = int32_t(nb);
      }
    }
  }
}

template <bool DESC>
int launch_match(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                 int64_t n_blocks, int32_t *matched, const uint64_t *desc, const uint32_t *inv, const ProbeHdr *ph,
                 hipStream_t stream) {
  const DevIndex ix = dev_view(idx);
  const dim3 grid((n_req + MW - 1) / MW), block(64 * MW);
  const int wpl = (ix.words + 63) / 64;
  if (wpl <= 1)
    hipLaunchKernelGGL((match_kernel<1, DESC>), grid, block, 0, stream, ix, keys, blk_off, n_req, n_blocks, matched, desc, inv, ph);
  else if (wpl <= 2)
    hipLaunchKernelGGL((match_kernel<2, DESC>), grid, block, 0, stream, ix, keys, blk_off, n_req, n_blocks, matched, desc, inv, ph);
  else if (wpl <= 4)
    hipLaunchKernelGGL((match_kernel<4, DESC>), grid, block, 0, stream, ix, keys, blk_off, n_req, n_blocks, matched, desc, inv, ph);
  else if (wpl <= 8)
    hipLaunchKernelGGL((match_kernel<8, DESC>), grid, block, 0, stream, ix, keys, blk_off, n_req, n_blocks, matched, desc, inv, ph);
  else
    hipLaunchKernelGGL((match_kernel<16, DESC>), grid, block, 0, stream, ix, keys, blk_off, n_req, n_blocks, matched, desc, inv, ph);
  return hip_rc(hipGetLastError());
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_match(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off,
                             int32_t n_req, int64_t n_blocks, int32_t *matched, hipStream_t stream) {
  if (!idx || n_req < 0 || n_blocks < 0) return SMETRIC_EINVAL;
  if (n_req == 0) return SMETRIC_OK;
  if (!blk_off || !matched || (n_blocks > 0 && !keys) || !idx->slots) return SMETRIC_EINVAL;
  return launch_match<false>(idx, keys, blk_off, n_req, n_blocks, matched, nullptr, nullptr, nullptr, stream);
}

extern "C" int smetric_match_probed(const smetric_index *idx, const void *probe, uint64_t probe_bytes,
                                    const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                                    int64_t n_blocks, int32_t *matched, hipStream_t stream) {
  if (!idx || n_req < 0 || n_blocks < 0 || n_blocks >= (int64_t(1) << 32)) return SMETRIC_EINVAL;
  if (n_req == 0) return SMETRIC_OK;
  if (!blk_off || !matched || (n_blocks > 0 && !keys) || !idx->slots) return SMETRIC_EINVAL;
  if (!probe || (reinterpret_cast<uintptr_t>(probe) & 255) || probe_bytes < probe_layout(n_blocks, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  ProbeView pv;
  probe_layout(n_blocks, &pv, const_cast<void *>(probe));
  return launch_match<true>(idx, keys, blk_off, n_req, n_blocks, matched, pv.desc_p, pv.inv, pv.hdr, stream);
}
