// Global block index in HBM: layout, insert (K2 + K7), evict (K6), dump, stats.
//
// Paper: the router consults each instance's local KV$ contents ("kvc", Sec. 4.1) to get
// the prefix hit c_i; the structure is not described.  The index here is the set of
// entries (key, instance) with the producing session and the last epoch; after a batch
// is routed every full block of each prompt is entered on its target (the target's
// prefill caches the prompt, Sec. 2 and 4.2), and a fraction of the oldest entries can be
// evicted (local tiers evict, Sec. 2 and 4.2 "session_cached").
//
// Layout of the caller's buffer:
//   [0, 256)                 IndexHdr: entry count, sticky status, pool use
//   slots                    n_buckets x 128 B: keys[8] then values[8]
//   pool                     n_records x bitmap_words x 8 B: holder bitmaps
//   masks                    n_buckets x 16 bits: each chain start's displacement mask
// A key normally owns one PLAIN slot per holder in its home chain (linear probing over
// buckets from home_bucket(key)).  When a key gains more than T holders its plain slots
// are replaced by one HEADER slot pointing at a bitmap record, and every holder becomes a
// MEMBER slot found from member_bucket(key, inst); probes of the key then read one
// bucket line plus the bitmap instead of walking T+ slots.  If the pool runs out, keys
// simply stay plain.  Slots are only ever claimed (EMPTY -> key by compare-and-swap) or
// turned into tombstones, so every slot of a key lies before the first EMPTY slot of its
// chain.  Eviction selects the oldest entries by (epoch, key, instance) digit by digit
// over a gathered copy of the entries, then turns them into tombstones in place, or --
// once tombstones would take too many slots -- rebuilds the table from the survivors.
//
// Insert pipeline (no sort, no host synchronisation):
//   clear      scratch dedupe table
//   probe      per pair (r, j): validate; find (key, target) -> refresh position, or
//              enter the pair in the dedupe table keyed by (key, instance), keeping the
//              lowest request index (atomic min), and list each distinct new pair once
//   check      one thread: first error -> EINVAL/EFULL, nothing changes; else count
//   refresh    epoch = max(old, epoch) for existing entries
//   place      each distinct new pair claims a slot; the thread whose slot becomes the
//              key's (T+1)-th plain slot -- unique, since claims fill a chain in order --
//              queues the key for conversion
//   spill      queued keys get a bitmap record, member slots, a header and tombstones
#include <rocprim/device/device_radix_sort.hpp>

#include "common.h"

namespace smk {
namespace {

constexpr int TB = 256;
constexpr int MAX_GRID = 4096;

inline uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }
inline int grid_for(uint64_t n) {
  const uint64_t g = (n + TB - 1) / TB;
  return int(g < 1 ? 1 : (g > MAX_GRID ? MAX_GRID : g));
}

__global__ void fill_kernel(uint64_t *p, uint64_t n_words, uint64_t value) {
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n_words; i += stride) p[i] = value;
}

__global__ void set_int_kernel(int *p, int v) { *p = v; }

__global__ void unset_values_kernel(uint64_t *slots, uint64_t n_buckets) {
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t b = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; b < n_buckets; b += stride) {
    ulonglong2 *v = reinterpret_cast<ulonglong2 *>(slots + b * BUCKET_WORDS + SLOTS);
#pragma unroll
    for (int i = 0; i < SLOTS / 2; ++i) v[i] = make_ulonglong2(VAL_UNSET, VAL_UNSET);
  }
}

int fill(void *p, uint64_t bytes, uint64_t value, hipStream_t s) {
  const uint64_t n = bytes / 8;
  if (n == 0) return SMETRIC_OK;
  hipLaunchKernelGGL(fill_kernel, dim3(grid_for(n)), dim3(TB), 0, s, static_cast<uint64_t *>(p), n, value);
  return hip_rc(hipGetLastError());
}

struct Layout {
  int32_t words, threshold;
  uint64_t n_records, n_buckets, slots_off, pool_off, bytes;
};

// n_slots = 0: the table holds capacity entries (plus converted keys' headers and
// tombstones) at <= 3/4 occupancy.  Otherwise the caller fixes the slot count (rounded up
// to whole buckets), which must leave at least 1/16 of the slots free at capacity.
bool layout_for(uint64_t capacity, int32_t n_inst, uint64_t n_slots, Layout &L) {
  if (capacity == 0 || capacity > (uint64_t(1) << 40) || n_inst < 1 || n_inst > 65536) return false;
  if (n_slots > (uint64_t(1) << 41)) return false;
  L.words = bitmap_words_for(n_inst);
  L.threshold = threshold_for(n_inst);
  uint64_t rec = capacity / 256;
  if (rec < 64) rec = 64;
  const uint64_t rec_max = capacity / uint64_t(L.threshold + 1) + 1;
  if (rec > rec_max) rec = rec_max;
  L.n_records = rec;
  // slots: live entries plus headers/tombstones of converted keys, at <= 3/4 occupancy
  const uint64_t slots = capacity + uint64_t(L.threshold) * rec;
  if (n_slots == 0) {
    L.n_buckets = (slots * 4 / 3 + SLOTS - 1) / SLOTS + 1;
  } else {
    L.n_buckets = (n_slots + SLOTS - 1) / SLOTS;
    if (slots * 16 > L.n_buckets * SLOTS * 15) return false;
  }
  L.slots_off = sizeof(IndexHdr);
  L.pool_off = L.slots_off + L.n_buckets * BUCKET_WORDS * 8;
  // then the displacement masks, one byte per bucket (dev_view finds them after the pool)
  L.bytes = round_up(L.pool_off + L.n_records * uint64_t(L.words) * 8 + mask_bytes(L.n_buckets), 256);
  return true;
}

int attach(smetric_index *idx, void *mem, uint64_t mem_bytes, uint64_t capacity, int32_t n_inst, uint64_t n_slots) {
  Layout L;
  if (!idx || !mem || !layout_for(capacity, n_inst, n_slots, L) || mem_bytes < L.bytes ||
      (reinterpret_cast<uintptr_t>(mem) & 255))
    return SMETRIC_EINVAL;
  char *base = static_cast<char *>(mem);
  idx->mem = mem;
  idx->mem_bytes = mem_bytes;
  idx->capacity = capacity;
  idx->n_instances = n_inst;
  idx->bitmap_words = L.words;
  idx->spill_threshold = L.threshold;
  idx->reserved0 = 0;
  idx->n_buckets = L.n_buckets;
  idx->n_records = L.n_records;
  idx->slots = reinterpret_cast<uint64_t *>(base + L.slots_off);
  idx->pool = reinterpret_cast<uint64_t *>(base + L.pool_off);
  idx->hdr = base;
  return SMETRIC_OK;
}

// ---------------------------------------------------------------------------------
// Table primitives
// ---------------------------------------------------------------------------------
struct Found {
  int64_t slot;  // bucket * SLOTS + s, or -1
  uint64_t val;
};

// Find the entry (key, inst), looking through a bitmap record when the key has one.
__device__ Found find_member(const DevIndex &ix, uint64_t key, uint32_t inst) {
  ChainWalk w = chain_start(member_bucket(key, inst, ix.n_buckets, ix.nb_inv), member_cls(key, inst));
  bool had_empty;
  do {
    const uint64_t m = w.b;
    const uint64_t *mk = ix.slots + m * BUCKET_WORDS;
    const BucketScan sc = scan_bucket(mk, key);
    uint32_t mm = sc.match;
    while (mm) {
      const int t = __builtin_ctz(mm);
      mm &= mm - 1;
      const uint64_t v = mk[SLOTS + t];
      if (val_kind(v) == MEMBER && val_inst(v) == inst) return Found{int64_t(m * SLOTS + t), v};
    }
    had_empty = sc.empty != 0;
  } while (chain_next(ix, w, had_empty));
  return Found{-1, 0};
}

__device__ Found find_entry(const DevIndex &ix, uint64_t key, uint32_t inst) {
  ChainWalk w = chain_start(home_bucket(key, ix.n_buckets), key_cls(key));
  bool had_empty;
  do {
    const uint64_t b = w.b;
    const uint64_t *bk = ix.slots + b * BUCKET_WORDS;
    const BucketScan sc = scan_bucket(bk, key);
    uint32_t mm = sc.match;
    while (mm) {
      const int s = __builtin_ctz(mm);
      mm &= mm - 1;
      const uint64_t v = bk[SLOTS + s];
      const uint32_t kind = val_kind(v);
      if (kind == PLAIN && val_inst(v) == inst) return Found{int64_t(b * SLOTS + s), v};
      if (kind == HEADER) {
        const uint64_t bw = ix.pool[val_rec(v) * uint64_t(ix.words) + (inst >> 6)];
        if (!((bw >> (inst & 63)) & 1)) return Found{-1, 0};
        return find_member(ix, key, inst);
      }
    }
    had_empty = sc.empty != 0;
  } while (chain_next(ix, w, had_empty));
  return Found{-1, 0};
}

__device__ __forceinline__ uint64_t *val_ptr(const DevIndex &ix, int64_t slot) {
  return ix.slots + (slot / SLOTS) * BUCKET_WORDS + SLOTS + (slot % SLOTS);
}

// Walk the chain from bucket b and claim its first EMPTY slot for `key`.  With
// want_header, stop instead at a HEADER slot of `key` (the key has a bitmap record).
// `same` counts slots holding `key` ahead of the claimed one.  Plain loads may see a
// stale EMPTY; the compare-and-swap then fails and returns the slot's real key, and
// slots never return to EMPTY, so the count is exact.
// With max_same, the walk gives up (capped) once it has seen max_same slots of `key`
// ahead of any free slot: that key is about to get a bitmap record, and its remaining
// new holders are entered after the conversion instead of piling up plain slots that
// would all turn into tombstones.
// With want_inst, a PLAIN slot of (key, want_inst) met on the way ends the walk instead
// (existing): the pair is already an entry.
struct Claim {
  int64_t slot;      // claimed slot, or -1
  int64_t header;    // HEADER slot of key when found, else -1
  int64_t existing;  // PLAIN slot of (key, want_inst) when found, else -1
  uint32_t same;
  bool capped;
};
constexpr uint32_t NO_INST = 0xFFFFFFFFu;
__device__ Claim claim_slot(const DevIndex &ix, uint64_t b, uint64_t key, uint32_t cls, bool want_header,
                            uint32_t max_same = 0xFFFFFFFFu, uint32_t want_inst = NO_INST) {
  Claim c{-1, -1, -1, 0, false};
  const uint64_t h = b;  // the chain start whose displacement mask records the claim
  for (uint64_t step = 0; step < ix.n_buckets; ++step, b = next_bucket(b, ix.n_buckets)) {
    uint64_t *bk = ix.slots + b * BUCKET_WORDS;
    const BucketScan sc = scan_bucket(bk, key);
    if (want_header || want_inst != NO_INST) {
      uint32_t mm = sc.match;
      while (mm) {
        const int s = __builtin_ctz(mm);
        mm &= mm - 1;
        const uint64_t v = bk[SLOTS + s];
        if (want_header && val_kind(v) == HEADER) {
          c.header = int64_t(b * SLOTS + s);
          return c;
        }
        if (val_kind(v) == PLAIN && val_inst(v) == want_inst) {
          c.existing = int64_t(b * SLOTS + s);
          return c;
        }
      }
    }
    if (!sc.empty) {
      c.same += __popc(sc.match);
      if (c.same >= max_same) {
        c.capped = true;
        return c;
      }
      continue;
    }
    // slots before the first EMPTY are final; try the EMPTY ones in order
    const int first = __builtin_ctz(sc.empty);
    c.same += __popc(sc.match & ((1u << first) - 1u));
    for (int s = first; s < SLOTS; ++s) {
      if (c.same >= max_same) {
        c.capped = true;
        return c;
      }
      const uint64_t k = atomicCAS(reinterpret_cast<unsigned long long *>(&bk[s]), KEY_EMPTY, key);
      if (k == KEY_EMPTY) {
        c.slot = int64_t(b * SLOTS + s);
        mask_note(ix, h, b, cls);
        return c;
      }
      if (k == key) {  // claimed meanwhile by another pair of the same key (never this pair)
        if (want_header && val_kind(__hip_atomic_load(&bk[SLOTS + s], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) == HEADER) {
          c.header = int64_t(b * SLOTS + s);  // cannot happen: headers predate this kernel
          return c;
        }
        ++c.same;
      }
    }
  }
  return c;
}

// epoch = max(old, epoch) of the entry at `slot` (kind and instance given), session kept
// (an existing pair).
__device__ __forceinline__ void refresh_at(const DevIndex &ix, int64_t slot, uint32_t kind, uint32_t inst,
                                           uint32_t epoch) {
  raise_epoch_at(val_ptr(ix, slot), kind, inst, epoch);
}

// Enter a pair that is not known to be an entry (one per pair and call: pairs are
// distinct).  Returns PLACED, REFRESHED (it was an entry: its epoch is raised instead),
// DEFERRED (capped: enter it again after the key's conversion, uncapped) or FAILED (no
// free slot).  trigger is set when the slot is the key's (T+1)-th plain slot, the last
// one a key gets before its conversion.
enum Placed { PLACED = 0, DEFERRED = 1, FAILED = 2, REFRESHED = 3 };
__device__ int place_new(const DevIndex &ix, uint64_t key, uint32_t inst, uint32_t epoch, uint32_t sess,
                         bool &trigger, bool capped) {
  trigger = false;
  const Claim c = claim_slot(ix, home_bucket(key, ix.n_buckets), key, key_cls(key), true,
                             capped ? uint32_t(ix.threshold) + 1 : 0xFFFFFFFFu, inst);
  if (c.existing >= 0) {
    refresh_at(ix, c.existing, PLAIN, inst, epoch);
    return REFRESHED;
  }
  if (c.header >= 0) {
    const uint64_t rec = val_rec(*val_ptr(ix, c.header));
    const unsigned long long old = atomicOr(
        reinterpret_cast<unsigned long long *>(&ix.pool[rec * uint64_t(ix.words) + (inst >> 6)]), 1ull << (inst & 63));
    if ((old >> (inst & 63)) & 1) {  // already a member
      const Found f = find_member(ix, key, inst);
      if (f.slot < 0) return FAILED;
      refresh_at(ix, f.slot, MEMBER, inst, epoch);
      return REFRESHED;
    }
    const Claim m = claim_slot(ix, member_bucket(key, inst, ix.n_buckets, ix.nb_inv), key, member_cls(key, inst), false);
    if (m.slot < 0) return FAILED;
    *val_ptr(ix, m.slot) = make_val(inst, MEMBER, epoch, sess);
    return PLACED;
  }
  if (c.capped) return DEFERRED;
  if (c.slot < 0) return FAILED;
  *val_ptr(ix, c.slot) = make_val(inst, PLAIN, epoch, sess);
  trigger = c.same == uint32_t(ix.threshold);
  return PLACED;
}

// A REFRESHED pair was counted as new by the capacity check: take it back, one atomic
// per wavefront.
__device__ __forceinline__ void uncount_refreshed(const DevIndex &ix, bool refreshed) {
  const uint64_t m = __ballot(refreshed);
  if (m && (threadIdx.x & 63) == uint32_t(__builtin_ctzll(m)))
    atomicAdd(&ix.hdr->n_entries, 0ull - (unsigned long long)__popcll(m));
}

// Replace the plain slots of `key` by a bitmap record (one thread per key).
__device__ bool spill_key(const DevIndex &ix, uint64_t key) {
  const unsigned long long rec = atomicAdd(reinterpret_cast<unsigned long long *>(&ix.hdr->rec_used), 1ull);
  if (rec >= ix.n_records) return true;  // pool exhausted: the key stays plain
  uint64_t *bm = ix.pool + rec * uint64_t(ix.words);
  int64_t first = -1;
  uint64_t b = home_bucket(key, ix.n_buckets);
  for (uint64_t step = 0; step < ix.n_buckets; ++step) {
    uint64_t *bk = ix.slots + b * BUCKET_WORDS;
    bool end = false;
    for (int s = 0; s < SLOTS; ++s) {
      const uint64_t k = bk[s];
      if (k == KEY_EMPTY) {
        end = true;
        break;
      }
      if (k != key) continue;
      const uint64_t v = bk[SLOTS + s];
      if (val_kind(v) != PLAIN) continue;
      const uint32_t inst = val_inst(v);
      bm[inst >> 6] |= 1ull << (inst & 63);
      const Claim m = claim_slot(ix, member_bucket(key, inst, ix.n_buckets, ix.nb_inv), key, member_cls(key, inst), false);
      if (m.slot < 0) return false;
      *val_ptr(ix, m.slot) = make_val(inst, MEMBER, val_epoch(v), val_session(v));
      if (first < 0) {
        first = int64_t(b * SLOTS + s);
        bk[SLOTS + s] = header_val(rec);
      } else {
        bk[s] = KEY_TOMB;
      }
    }
    if (end) break;
    b = (b + 1 == ix.n_buckets) ? 0 : b + 1;
  }
  return true;
}

// ---------------------------------------------------------------------------------
// Insert
// ---------------------------------------------------------------------------------
struct WsHdr {
  unsigned long long n_new;    // distinct new pairs listed
  unsigned long long n_pairs;  // pairs over all request ranges
  unsigned long long n_trig;   // keys queued for conversion
  int err;                     // first input error seen by the probe
  int abort;                   // set by the check: leave the index unchanged
  unsigned long long n_cand;   // pairs absent before the batch (region-ordered insert)
  unsigned long long n_dd;     // dedupe slots in use (a power of two)
  unsigned long long n_def;    // new pairs deferred until their key's conversion
  unsigned long long nsub;     // region-ordered insert: bins per region (a power of two)
  unsigned long long n_dd2;    // region-ordered insert: fallback pair-table slots in use
  unsigned long long n_over;   // region-ordered insert: candidates in bins too large for LDS
  int req_bad;                 // region-ordered insert: some request's target or session is invalid
  int inl;                     // region-ordered insert: refreshes done by the classify pass
  unsigned long long pad[21];
};
static_assert(sizeof(WsHdr) == 256, "ws header size");

// Dedupe table slot: the pair's key and (inst + 1) << 32 | lowest request index, both in
// one 16-byte slot so a pair costs one line; all-zero = free.
struct DSlot {
  uint64_t key;
  uint64_t w2;
};
__device__ __forceinline__ uint32_t dd_inst(uint64_t w2) { return uint32_t(w2 >> 32) - 1; }
__device__ __forceinline__ uint32_t dd_req(uint64_t w2) { return uint32_t(w2); }

// Candidate of the region-ordered insert: an absent pair, as it enters the dedupe.
struct Cand {
  uint64_t key;
  uint64_t w2;  // same encoding as DSlot::w2
};

// Distinct new pair of the region-ordered insert, in bin order (key KEY_EMPTY: a dropped
// duplicate).  w2 as in DSlot, or NP_FALLBACK | h: the pair went through the fallback
// pair table and dd[h].w2 holds its final (lowest) request.
struct NewPair {
  uint64_t key;
  uint64_t w2;
};
constexpr uint64_t NP_FALLBACK = uint64_t(1) << 63;
__device__ __forceinline__ uint64_t np_w2(const NewPair &e, const DSlot *dd) {
  return (e.w2 & NP_FALLBACK) ? dd[e.w2 & ~NP_FALLBACK].w2 : e.w2;
}

// Binning of the region-ordered insert's candidates: bins are NREG x nsub equal ranges of
// home buckets, so every candidate of a key -- and of a (key, instance) pair -- lies in
// one bin, and a bin is deduplicated in LDS by one workgroup.
constexpr int KCH = 32;                     // chunks per region of the bin partition
// The classify pass runs INS_WG workgroups (as many as the device holds at its register
// use), each filling one candidate segment.
constexpr int INS_WG = 1024;
// Workgroups of the placement's grid.
constexpr int PLACE_WG = 4096;
inline uint64_t ins_segment(uint64_t n) {
  const uint64_t span = uint64_t(INS_WG) * WG_THREADS;
  return (n + span - 1) / span * WG_THREADS;
}
constexpr int SEG_PER_CH = INS_WG / KCH;    // classify segments per chunk
constexpr int NSUB_MAX = 1024;              // bins per region, at most
constexpr int NBIN_MAX = NREG * NSUB_MAX;
constexpr int BIN_TARGET = 1536;            // nsub keeps the mean bin at or below this
constexpr int DT = 4096;                    // slots of a bin's LDS pair table
constexpr int BIN_CAP = 3072;               // larger bins use the fallback pair table
static_assert(INS_WG % KCH == 0 && SEG_PER_CH <= 64, "chunk = whole classify segments");
static_assert(BIN_CAP + WG_THREADS < DT, "an LDS pair table never fills");

struct InsWs {
  WsHdr *hdr;
  uint64_t *pos;    // per block: slot + 1 of an entry to refresh, 0 = none
  DSlot *dd;        // dedupe table (region-ordered insert: fallback pair table)
  uint64_t *list;   // dedupe slots of distinct new pairs
  uint64_t *trig;   // keys queued for conversion
  uint64_t *def;    // list positions of deferred new pairs
  Cand *cand;       // region-ordered insert: absent pairs, one segment per workgroup,
                    // cut into one part per region
  uint32_t *cand_cnt;  // [INS_WG] candidates in each segment
  uint32_t *ctot;   // [NREG][KCH] candidates in each chunk of the bin partition
  uint32_t *soff;   // [INS_WG][NREG] offset of each (segment, region) part in its segment
  uint32_t *rcnt;   // [INS_WG][NREG] candidates in each part
  uint32_t *hist2;  // [NREG][KCH][NSUB_MAX] candidates of each bin in each chunk
  uint32_t *base2;  // [NREG][KCH][NSUB_MAX] first bin-order position of each (chunk, bin)
  uint32_t *bstart; // [NBIN_MAX + 1] first bin-order position of each bin
  uint32_t *bdist;  // [NBIN_MAX] distinct new pairs of each bin
  Cand *bcand;      // candidates in bin order
  NewPair *np;      // bin order: distinct new pairs
  uint64_t n_dedupe;
  uint64_t list_cap;  // entries in list and trig
  uint64_t seg;       // segment length of the region-ordered insert
};

uint64_t dedupe_size(int64_t n_blocks) {
  uint64_t n = 64;
  while (n < 2 * uint64_t(n_blocks)) n <<= 1;
  return n;
}

uint64_t insert_ws_layout(int64_t n_blocks, InsWs *ws, void *base) {
  const uint64_t n = uint64_t(n_blocks < 1 ? 1 : n_blocks);
  const uint64_t nd = dedupe_size(n_blocks);
  const uint64_t seg = ins_segment(n), seg_n = seg * INS_WG;
  const uint64_t nl = seg_n > n ? seg_n : n;
  uint64_t off = 0;
  auto take = [&](uint64_t bytes) {
    const uint64_t o = off;
    off = round_up(off + bytes, 256);
    return o;
  };
  const uint64_t o_hdr = take(sizeof(WsHdr));
  const uint64_t o_pos = take(8 * n);
  const uint64_t o_dd = take(16 * nd);
  const uint64_t o_list = take(8 * nl);
  const uint64_t o_trig = take(8 * nl);
  const uint64_t o_def = take(8 * nl);
  const uint64_t o_cand = take(sizeof(Cand) * seg_n);
  const uint64_t o_cc = take(4ull * INS_WG);
  const uint64_t o_ct = take(4ull * NREG * KCH);
  const uint64_t o_soff = take(4ull * INS_WG * NREG);
  const uint64_t o_rcnt = take(4ull * INS_WG * NREG);
  const uint64_t o_h2 = take(4ull * NREG * KCH * NSUB_MAX);
  const uint64_t o_b2 = take(4ull * NREG * KCH * NSUB_MAX);
  const uint64_t o_bs = take(4ull * (NBIN_MAX + 1));
  const uint64_t o_bd = take(4ull * NBIN_MAX);
  const uint64_t o_bc = take(sizeof(Cand) * n);
  const uint64_t o_np = take(sizeof(NewPair) * n);
  if (ws) {
    char *b = static_cast<char *>(base);
    ws->hdr = reinterpret_cast<WsHdr *>(b + o_hdr);
    ws->pos = reinterpret_cast<uint64_t *>(b + o_pos);
    ws->dd = reinterpret_cast<DSlot *>(b + o_dd);
    ws->list = reinterpret_cast<uint64_t *>(b + o_list);
    ws->trig = reinterpret_cast<uint64_t *>(b + o_trig);
    ws->def = reinterpret_cast<uint64_t *>(b + o_def);
    ws->cand = reinterpret_cast<Cand *>(b + o_cand);
    ws->cand_cnt = reinterpret_cast<uint32_t *>(b + o_cc);
    ws->ctot = reinterpret_cast<uint32_t *>(b + o_ct);
    ws->soff = reinterpret_cast<uint32_t *>(b + o_soff);
    ws->rcnt = reinterpret_cast<uint32_t *>(b + o_rcnt);
    ws->hist2 = reinterpret_cast<uint32_t *>(b + o_h2);
    ws->base2 = reinterpret_cast<uint32_t *>(b + o_b2);
    ws->bstart = reinterpret_cast<uint32_t *>(b + o_bs);
    ws->bdist = reinterpret_cast<uint32_t *>(b + o_bd);
    ws->bcand = reinterpret_cast<Cand *>(b + o_bc);
    ws->np = reinterpret_cast<NewPair *>(b + o_np);
    ws->n_dedupe = nd;
    ws->list_cap = nl;
    ws->seg = seg;
  }
  return off;
}

__device__ __forceinline__ void ws_error(WsHdr *h, int e) { atomicCAS(&h->err, 0, e); }

// Returns the dedupe slot when this call created the entry (first sighting of the
// pair), else -1; the caller lists created slots with one atomic per wavefront.
__device__ int64_t dedupe_pair(const InsWs &ws, uint64_t nd, uint64_t key, uint64_t mine) {
  uint64_t h = mix64(key ^ ((mine >> 32) * 0xC2B2AE3D27D4EB4Full)) & (nd - 1);
  for (uint64_t step = 0; step < nd; ++step, h = (h + 1) & (nd - 1)) {
    DSlot *d = ws.dd + h;
    uint64_t k = __hip_atomic_load(&d->key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (k == KEY_EMPTY) k = atomicCAS(reinterpret_cast<unsigned long long *>(&d->key), KEY_EMPTY, key);
    if (k != KEY_EMPTY && k != key) continue;
    // this slot's key is `key`; its owner instance is decided by the second word
    uint64_t w = __hip_atomic_load(&d->w2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    while (true) {
      if (w == 0) {
        const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long *>(&d->w2), 0ull, mine);
        if (prev == 0) return int64_t(h);
        w = prev;
        continue;
      }
      if ((w >> 32) == (mine >> 32)) {
        if (mine < w) atomicMin(reinterpret_cast<unsigned long long *>(&d->w2), mine);
        return -1;
      }
      break;  // another instance's pair: keep probing
    }
  }
  ws_error(ws.hdr, SMETRIC_EINTERNAL);
  return -1;
}

// Append base + j for every bit j of each lane's mask: one atomicAdd per wavefront.
__device__ __forceinline__ void append_wave_mask(unsigned long long *counter, uint64_t *list, uint64_t cap,
                                                 uint32_t mask, uint64_t base) {
  const uint32_t c = __popc(mask);
  if (!__ballot(c != 0)) return;
  const int lane = threadIdx.x & 63;
  uint32_t x = c;  // inclusive prefix over the wavefront
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  unsigned long long at = 0;
  if (lane == 63) at = atomicAdd(counter, (unsigned long long)x);
  at = __shfl(at, 63, 64) + (x - c);
  while (mask) {
    const int j = __builtin_ctz(mask);
    mask &= mask - 1;
    if (at < cap) list[at] = base + uint64_t(j);  // callers size the list to hold every entry
    ++at;
  }
}

// Append `h` (when >= 0) to the list: one atomicAdd per wavefront for all its lanes.
__device__ __forceinline__ void append_wave(unsigned long long *counter, uint64_t *list, uint64_t cap, int64_t h) {
  const uint64_t want = __ballot(h >= 0);
  if (!want) return;
  const int lane = threadIdx.x & 63;
  const int leader = __builtin_ctzll(want);
  unsigned long long base = 0;
  if (lane == leader) base = atomicAdd(counter, (unsigned long long)__popcll(want));
  base = __shfl(base, leader, 64);
  if (h >= 0) {
    const unsigned long long at = base + __popcll(want & ((uint64_t(1) << lane) - 1));
    if (at < cap) list[at] = uint64_t(h);  // more pairs than blocks: rejected by the check
  }
}

constexpr int IW = 1;  // waves per workgroup in per-request kernels

__device__ __forceinline__ bool range_of(const int64_t *blk_off, int r, int64_t n_blocks, int64_t &b0,
                                         int64_t &nb) {
  b0 = blk_off[r];
  const int64_t b1 = blk_off[r + 1];
  nb = b1 - b0;
  return b0 >= 0 && b0 <= b1 && b1 <= n_blocks;
}

__global__ __launch_bounds__(64 * IW) void ins_probe_kernel(DevIndex ix, InsWs ws, const uint64_t *keys,
                                                            const int64_t *blk_off, int32_t n_req,
                                                            int64_t n_blocks, const int32_t *instance,
                                                            const uint32_t *session, uint32_t epoch) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * IW + wave;
  if (r >= n_req) return;
  int64_t b0, nb;
  if (!range_of(blk_off, r, n_blocks, b0, nb)) {
    if (lane == 0) ws_error(ws.hdr, SMETRIC_EINVAL);
    return;
  }
  if (nb == 0) return;
  if (lane == 0) atomicAdd(&ws.hdr->n_pairs, (unsigned long long)nb);
  const int32_t inst = instance[r];
  const uint32_t sess = session[r];
  if (inst < 0 || inst >= ix.n_inst || sess >= SESSION_LIMIT) {
    if (lane == 0) ws_error(ws.hdr, SMETRIC_EINVAL);
    return;
  }
  for (int64_t j0 = 0; j0 < nb; j0 += 64) {
    const int64_t j = j0 + lane;
    int64_t fresh = -1;
    if (j < nb) {
      const uint64_t key = keys[b0 + j];
      if (key == KEY_EMPTY || key == KEY_TOMB) {
        ws_error(ws.hdr, SMETRIC_EINVAL);
        ws.pos[b0 + j] = 0;
      } else {
        const Found f = find_entry(ix, key, uint32_t(inst));
        if (f.slot >= 0) {
          ws.pos[b0 + j] = val_epoch(f.val) < epoch ? uint64_t(f.slot) + 1 : 0;
        } else {
          ws.pos[b0 + j] = 0;
          fresh = dedupe_pair(ws, ws.n_dedupe, key, ((uint64_t(inst) + 1) << 32) | uint32_t(r));
        }
      }
    }
    append_wave(&ws.hdr->n_new, ws.list, ws.list_cap, fresh);
  }
}

__global__ void ins_check_kernel(DevIndex ix, InsWs ws, int64_t n_blocks) {
  WsHdr *h = ws.hdr;
  int e = h->err;
  if (e == 0 && h->n_pairs > (unsigned long long)n_blocks) e = SMETRIC_EINVAL;
  if (e == 0 && ix.hdr->n_entries + h->n_new > ix.capacity) e = SMETRIC_EFULL;
  if (e != 0) {
    h->abort = 1;
    set_status(ix.hdr, e);
  } else {
    ix.hdr->n_entries += h->n_new;
  }
}

__global__ __launch_bounds__(64 * IW) void ins_refresh_kernel(DevIndex ix, InsWs ws, const int64_t *blk_off,
                                                              int32_t n_req, int64_t n_blocks,
                                                              uint32_t epoch) {
  if (ws.hdr->abort) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * IW + wave;
  if (r >= n_req) return;
  int64_t b0, nb;
  if (!range_of(blk_off, r, n_blocks, b0, nb)) return;
  for (int64_t j = lane; j < nb; j += 64) {
    const uint64_t p = ws.pos[b0 + j];
    if (!p) continue;
    uint64_t *vp = val_ptr(ix, int64_t(p - 1));
    const uint64_t v = *vp;
    if (val_epoch(v) < epoch) *vp = val_raise_epoch(v, epoch);
  }
}

__global__ void ins_place_kernel(DevIndex ix, InsWs ws, const uint32_t *session, uint32_t epoch) {
  if (ws.hdr->abort) return;
  const uint64_t n = ws.hdr->n_new;
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  const uint64_t first = uint64_t(blockIdx.x) * blockDim.x + (threadIdx.x & ~63u);
  for (uint64_t i0 = first; i0 < n; i0 += stride) {  // whole wavefronts iterate together
    const uint64_t i = i0 + (threadIdx.x & 63);
    int64_t tk = -1, df = -1;
    bool rf = false;
    if (i < n) {
      const DSlot d = ws.dd[ws.list[i]];
      bool trig;
      const int pl = place_new(ix, d.key, dd_inst(d.w2), epoch, session[dd_req(d.w2)], trig, true);
      if (pl == FAILED) set_status(ix.hdr, SMETRIC_EINTERNAL);
      else if (pl == DEFERRED) df = int64_t(i);
      else if (pl == REFRESHED) rf = true;
      else if (trig) tk = int64_t(i);
    }
    uncount_refreshed(ix, rf);
    append_wave(&ws.hdr->n_trig, ws.trig, ws.list_cap, tk);  // queue by list index
    append_wave(&ws.hdr->n_def, ws.def, ws.list_cap, df);
  }
}

// Convert the queued keys.  trig holds indexes: key = np[idx].key when `np` is given
// (region-ordered insert: new-pair positions), dd[via[idx]].key when `dd` is (insert:
// positions in the dedupe list), else keys[idx] (rebuild).
__global__ void spill_kernel(DevIndex ix, const uint64_t *trig, const unsigned long long *n_trig,
                             const int *abort_flag, const uint64_t *keys, const DSlot *dd, const uint64_t *via,
                             const NewPair *np) {
  if (abort_flag && *abort_flag) return;
  const uint64_t n = *n_trig;
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t t = trig[i];
    const uint64_t key = np ? np[t].key : (dd ? dd[via[t]].key : keys[t]);
    if (!spill_key(ix, key)) set_status(ix.hdr, SMETRIC_EINTERNAL);
  }
}

// ---------------------------------------------------------------------------------
// Region-ordered insert, from the descriptors of smetric_probe
// ---------------------------------------------------------------------------------
// Pipeline (no sort, no global atomics on the way to the distinct new pairs):
//   classify   per block in region order: refresh position, or candidate appended to the
//              region's part of the workgroup's segment; when no error can abort the
//              insert (checked beforehand: keys, requests, capacity for every block) the
//              refresh is done here and its pass is skipped
//   bins       the candidates partitioned into NREG x nsub bins of home buckets (count,
//              scan, scatter, as the probe's region partition), so all candidates of a
//              pair share a bin
//   dedupe     one workgroup per bin: an LDS pair table keeps each (key, instance) once
//              with its lowest request; bins above BIN_CAP use the global pair table
//   check      all-or-nothing: EINVAL or EFULL leave the index unchanged
//   refresh    epoch = max(old, epoch) at the classified positions (if not done above)
//   place      distinct new pairs in bin (so region) order; spill and deferred as above
// find_member with each bucket read whole (keys and values in one 128-byte request), so
// a chain step is one round trip.
__device__ Found find_member_line(const DevIndex &ix, uint64_t key, uint32_t inst) {
  ChainWalk cw = chain_start(member_bucket(key, inst, ix.n_buckets, ix.nb_inv), member_cls(key, inst));
  bool had_empty;
  do {
    const uint64_t m = cw.b;
    const ulonglong2 *p = reinterpret_cast<const ulonglong2 *>(ix.slots + m * BUCKET_WORDS);
    ulonglong2 kk[SLOTS / 2], vv[SLOTS / 2];
#pragma unroll
    for (int i = 0; i < SLOTS / 2; ++i) kk[i] = p[i];
#pragma unroll
    for (int i = 0; i < SLOTS / 2; ++i) vv[i] = p[SLOTS / 2 + i];
    bool end = false;
#pragma unroll
    for (int s = 0; s < SLOTS; ++s) {
      const uint64_t k = (s & 1) ? kk[s / 2].y : kk[s / 2].x;
      const uint64_t v = (s & 1) ? vv[s / 2].y : vv[s / 2].x;
      end |= k == KEY_EMPTY;
      if (!end && k == key && val_kind(v) == MEMBER && val_inst(v) == inst) return Found{int64_t(m * SLOTS + s), v};
    }
    had_empty = end;
  } while (chain_next(ix, cw, had_empty));
  return Found{-1, 0};
}

// classify: per probed block (region order), is (key, target) already an entry?  The
// descriptor answers it for NONE and ONE; HOT needs the bitmap bit and the member slot
// (inside the key's region), MANY a chain walk.  Existing -> refresh position; absent ->
// candidate, appended to the part of this workgroup's segment that holds its region
// (LDS counters, no global atomics).  The part of region g has room for every position
// of the workgroup in g: with F(x) = the workgroup's positions below x, it starts at
// F(start of g).
// All INS_WG workgroups advance through the region order together.  Each thread takes
// CU positions per round (the same positions as a plain grid-stride loop, so segments
// keep their bound), with every load of the round issued before any result is used.
__device__ __forceinline__ uint32_t positions_below(uint64_t x, uint64_t span, uint32_t w) {
  const uint64_t r = x % span, lo = uint64_t(w) * TB;
  return uint32_t((x / span) * TB + (r <= lo ? 0 : (r - lo < TB ? r - lo : TB)));
}

__global__ __launch_bounds__(TB) void insp_classify_kernel(DevIndex ix, ProbeView pv, InsWs ws,
                                                           const int32_t *instance, const uint32_t *session,
                                                           uint32_t epoch) {
  __shared__ unsigned int lc[NREG];
  __shared__ uint32_t part[NREG];
  __shared__ unsigned long long rb[NREG + 1];  // region boundaries in position order
  const int tid = threadIdx.x;
  const uint64_t span = uint64_t(gridDim.x) * TB;
  if (tid == 0) {
    unsigned long long acc = 0;
    for (int g = 0; g < NREG; ++g) {
      rb[g] = acc;
      acc += pv.hdr->tot[g];
    }
    rb[NREG] = acc;
  }
  __syncthreads();
  if (tid < NREG) {
    lc[tid] = 0;
    part[tid] = positions_below(rb[tid], span, blockIdx.x);
  }
  __syncthreads();
  const uint64_t n = pv.hdr->n;
  if (pv.hdr->err) {
    if (blockIdx.x == 0 && tid == 0) ws_error(ws.hdr, SMETRIC_EINVAL);
    if (tid < NREG) {
      ws.rcnt[uint64_t(blockIdx.x) * NREG + tid] = 0;
      ws.soff[uint64_t(blockIdx.x) * NREG + tid] = 0;
    }
    if (tid == 0) ws.cand_cnt[blockIdx.x] = 0;
    return;
  }
  // No error can abort this insert (valid keys and requests; even if every block were a new
  // entry the index would not overflow): refreshes are done here, in place.
  const bool inl = !pv.hdr->bad_key && !ws.hdr->req_bad && ix.hdr->n_entries + n <= ix.capacity;
  if (blockIdx.x == 0 && tid == 0) ws.hdr->inl = inl;
  Cand *seg = ws.cand + uint64_t(blockIdx.x) * ws.seg;
  constexpr int CU = 2;
  int gcur = 0;  // region of this thread's current position (positions only increase)
  for (uint64_t i0 = uint64_t(blockIdx.x) * TB + tid; i0 < n; i0 += CU * span) {
    // positions past the end read the last position (in bounds) and are dropped below
    uint64_t key[CU], d[CU];
    uint32_t r[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      const uint64_t i = i0 + u * span < n ? i0 + u * span : n - 1;
      key[u] = pv.part_key[i];
      r[u] = pv.part_req[i];
      d[u] = pv.desc_p[i];
    }
    int32_t t[CU];
    uint32_t sess[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      t[u] = instance[r[u]];
      sess[u] = session[r[u]];
    }
    // HOT: the target's bitmap word (a block of another kind reads record 0, always present)
    uint64_t hw[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      const bool hot = desc_kind(d[u]) == D_HOT && t[u] >= 0 && t[u] < ix.n_inst;
      hw[u] = ix.pool[(hot ? desc_x(d[u]) : 0) * uint64_t(ix.words) + (hot ? uint32_t(t[u]) >> 6 : 0u)];
    }
    int64_t slot[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      slot[u] = -1;
      const uint64_t i = i0 + u * span;
      if (i >= n) continue;
      while (gcur < NREG - 1 && rb[gcur + 1] <= i) ++gcur;
      if (t[u] < 0 || t[u] >= ix.n_inst || sess[u] >= SESSION_LIMIT || key[u] == KEY_EMPTY || key[u] == KEY_TOMB) {
        ws_error(ws.hdr, SMETRIC_EINVAL);
      } else {
        const uint32_t kind = desc_kind(d[u]);
        if (kind == D_ONE) {
          if (desc_inst(d[u]) == uint32_t(t[u])) slot[u] = int64_t(desc_x(d[u]));
        } else if (kind == D_HOT) {
          if ((hw[u] >> (t[u] & 63)) & 1) slot[u] = find_member_line(ix, key[u], uint32_t(t[u])).slot;
        } else if (kind == D_MANY) {
          slot[u] = find_entry(ix, key[u], uint32_t(t[u])).slot;
        }
        if (slot[u] < 0)
          seg[part[gcur] + atomicAdd(&lc[gcur], 1u)] = Cand{key[u], ((uint64_t(t[u]) + 1) << 32) | r[u]};
      }
    }
    if (inl) {
      // epoch = max(old, epoch) without a read: the entry is (key, t), a member for a HOT
      // key and a plain slot otherwise
#pragma unroll
      for (int u = 0; u < CU; ++u)
        if (slot[u] >= 0)
          raise_epoch_at(val_ptr(ix, slot[u]), desc_kind(d[u]) == D_HOT ? MEMBER : PLAIN, uint32_t(t[u]), epoch);
    } else {
#pragma unroll
      for (int u = 0; u < CU; ++u)
        if (i0 + u * span < n) ws.pos[i0 + u * span] = slot[u] >= 0 ? uint64_t(slot[u]) + 1 : 0;
    }
  }
  __syncthreads();
  if (tid < NREG) {
    ws.rcnt[uint64_t(blockIdx.x) * NREG + tid] = lc[tid];
    ws.soff[uint64_t(blockIdx.x) * NREG + tid] = part[tid];
  }
  if (tid == 0) {
    unsigned int all = 0;
    for (int g = 0; g < NREG; ++g) all += lc[g];
    ws.cand_cnt[blockIdx.x] = all;
  }
}

// Flags a request whose target or session is out of range (the classify pass then takes
// the path that checks every block before the index changes).
__global__ __launch_bounds__(TB) void insp_valid_kernel(DevIndex ix, InsWs ws, const int32_t *instance,
                                                        const uint32_t *session, int32_t n_req) {
  bool bad = false;
  for (int32_t r = blockIdx.x * TB + threadIdx.x; r < n_req; r += gridDim.x * TB)
    bad |= instance[r] < 0 || instance[r] >= ix.n_inst || session[r] >= SESSION_LIMIT;
  if (bad) atomicOr(&ws.hdr->req_bad, 1);
}

// Sum of n 32-bit counts, by one workgroup of TB threads (eight loads in flight per thread).
__device__ unsigned long long sum_counts(const uint32_t *cnt, uint32_t n) {
  __shared__ unsigned long long part[TB / 64];
  unsigned long long c = 0;
  for (uint32_t w0 = 0; w0 < n; w0 += 8 * TB) {
    uint32_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t w = w0 + u * TB + threadIdx.x;
      v[u] = w < n ? cnt[w] : 0u;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) c += v[u];
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) c += __shfl_xor(c, d, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
  __syncthreads();
  unsigned long long all = 0;
#pragma unroll
  for (int i = 0; i < TB / 64; ++i) all += part[i];
  __syncthreads();
  return all;
}

// total candidates -> bins per region: the least power of two that keeps the mean bin at
// or below BIN_TARGET candidates (at most NSUB_MAX)
__global__ __launch_bounds__(TB) void insp_size_kernel(InsWs ws) {
  const unsigned long long c = sum_counts(ws.cand_cnt, INS_WG);
  if (threadIdx.x != 0) return;
  ws.hdr->n_cand = c;
  uint64_t nsub = 1;
  while (nsub < NSUB_MAX && nsub * NREG * BIN_TARGET < c) nsub <<= 1;
  ws.hdr->nsub = nsub;
}

// Bin of a key among NREG * nsub equal ranges of home buckets; bin / nsub is its region.
__device__ __forceinline__ uint32_t bin_of(uint64_t key, uint64_t n_buckets, uint64_t nb_inv, uint32_t nsub) {
  return uint32_t(scaled_floor(home_bucket(key, n_buckets), uint64_t(NREG) * nsub, n_buckets, nb_inv));
}

// The candidates of chunk (g, c): the region-g parts of classify segments
// [c SEG_PER_CH, (c + 1) SEG_PER_CH), seen as one array through the parts' prefix sums.
struct ChunkParts {
  uint32_t pre[SEG_PER_CH + 1];  // prefix of the parts' counts
  uint64_t at[SEG_PER_CH];       // start of each part in ws.cand
};
__device__ void chunk_parts(const InsWs &ws, int g, int c, ChunkParts &cp) {
  if (threadIdx.x == 0) {
    uint32_t acc = 0;
    for (int p = 0; p < SEG_PER_CH; ++p) {
      const uint64_t w = uint64_t(c) * SEG_PER_CH + p;
      cp.pre[p] = acc;
      cp.at[p] = w * ws.seg + ws.soff[w * NREG + g];
      acc += ws.rcnt[w * NREG + g];
    }
    cp.pre[SEG_PER_CH] = acc;
  }
  __syncthreads();
}
__device__ __forceinline__ const Cand *chunk_item(const InsWs &ws, const ChunkParts &cp, uint32_t v) {
  int lo = 0, hi = SEG_PER_CH;  // the part p with pre[p] <= v < pre[p + 1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cp.pre[mid] <= v) lo = mid;
    else hi = mid;
  }
  return ws.cand + cp.at[lo] + (v - cp.pre[lo]);
}

// Count pass of the bin partition: workgroup (g, c) histograms its chunk over region g's
// bins (eight candidates per thread per round, loads first) and records the chunk's size.
__global__ __launch_bounds__(TB) void insp_bcount_kernel(DevIndex ix, InsWs ws) {
  __shared__ ChunkParts cp;
  __shared__ uint32_t h[NSUB_MAX];
  const int g = blockIdx.x / KCH, c = blockIdx.x % KCH;
  const uint32_t nsub = uint32_t(ws.hdr->nsub);
  for (int s = threadIdx.x; s < NSUB_MAX; s += TB) h[s] = 0;
  chunk_parts(ws, g, c, cp);  // synchronises
  const uint32_t m = cp.pre[SEG_PER_CH];
  constexpr int UC = 8;
  for (uint32_t v0 = 0; v0 < m; v0 += UC * TB) {
    uint64_t k[UC];
#pragma unroll
    for (int u = 0; u < UC; ++u) {
      const uint32_t v = v0 + u * TB + threadIdx.x;
      k[u] = v < m ? chunk_item(ws, cp, v)->key : 0;
    }
#pragma unroll
    for (int u = 0; u < UC; ++u) {
      if (v0 + u * TB + threadIdx.x < m) {
        const uint32_t sub = bin_of(k[u], ix.n_buckets, ix.nb_inv, nsub) - uint32_t(g) * nsub;
        atomicAdd(&h[sub < nsub ? sub : nsub - 1], 1u);
      }
    }
  }
  __syncthreads();
  uint32_t *out = ws.hist2 + (uint64_t(g) * KCH + c) * NSUB_MAX;
  for (uint32_t s = threadIdx.x; s < nsub; s += TB) out[s] = h[s];
  if (threadIdx.x == 0) ws.ctot[g * KCH + c] = m;
}

// Scan pass: workgroup g gives every bin of region g its first position (regions in
// order, bins in order inside a region) and every (chunk, bin) its running offset; bins
// larger than BIN_CAP add their size to n_over.  One thread per bin, its KCH chunk
// counts loaded at once.
constexpr int SCAN_T = NSUB_MAX;
static_assert(NREG * KCH <= SCAN_T, "one chunk total per thread for the region start");
__global__ __launch_bounds__(SCAN_T) void insp_bscan_kernel(InsWs ws) {
  __shared__ uint32_t wt[SCAN_T / 64];
  __shared__ unsigned long long red[SCAN_T / 64];
  const int g = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const uint32_t nsub = uint32_t(ws.hdr->nsub);
  // first position of region g: the chunks of every region before it
  unsigned long long before = t < g * KCH ? ws.ctot[t] : 0u;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) before += __shfl_xor(before, d, 64);
  if (lane == 0) red[wave] = before;
  const uint32_t *hg = ws.hist2 + uint64_t(g) * KCH * NSUB_MAX + t;
  uint32_t hc[KCH];
#pragma unroll
  for (int c = 0; c < KCH; ++c) hc[c] = uint32_t(t) < nsub ? hg[uint64_t(c) * NSUB_MAX] : 0u;
  uint32_t tot = 0;
#pragma unroll
  for (int c = 0; c < KCH; ++c) tot += hc[c];
  uint32_t x = tot;  // inclusive scan of the bin totals over the workgroup
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) wt[wave] = x;
  __syncthreads();
  unsigned long long start = 0;
#pragma unroll
  for (int i = 0; i < SCAN_T / 64; ++i) start += red[i];
  uint32_t pre = x - tot;
  for (int i = 0; i < wave; ++i) pre += wt[i];
  if (uint32_t(t) < nsub) {
    const uint32_t first = uint32_t(start) + pre;
    ws.bstart[uint64_t(g) * nsub + t] = first;
    uint32_t acc = first;
    uint32_t *bg = ws.base2 + uint64_t(g) * KCH * NSUB_MAX + t;
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      bg[uint64_t(c) * NSUB_MAX] = acc;
      acc += hc[c];
    }
    if (tot > uint32_t(BIN_CAP)) atomicAdd(&ws.hdr->n_over, (unsigned long long)tot);
    if (g == NREG - 1 && uint32_t(t) == nsub - 1) ws.bstart[uint64_t(NREG) * nsub] = acc;
  }
}

// fallback pair-table size for the oversized bins: a power of two >= 2 x their candidates;
// every thread sizes it (no separate launch), the first records it, all clear its slots
__global__ void insp_size2_kernel(InsWs ws) {
  const unsigned long long c = ws.hdr->n_over;
  uint64_t nd = 0;
  if (c) {
    nd = 64;
    while (nd < 2 * c && nd < ws.n_dedupe) nd <<= 1;
  }
  const uint64_t t0 = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t0 == 0) ws.hdr->n_dd2 = nd;
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t h = t0; h < nd; h += stride) ws.dd[h] = DSlot{0, 0};
}

__global__ void dd_clear_kernel(DSlot *dd, uint64_t n, const unsigned long long *n_dev) {
  const uint64_t nd = n_dev ? *n_dev : n;
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t h = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; h < nd; h += stride) dd[h] = DSlot{0, 0};
}

// Scatter pass: workgroup (g, c) moves its chunk into bin order one tile at a time (LDS
// ranks per bin, the tile regrouped by bin in LDS, each bin's part written as one run
// after the previous tile's).
constexpr int U2 = 8;
constexpr int TILE2 = U2 * TB;
static_assert(NSUB_MAX % TB == 0, "bins per thread in the scans");
__global__ __launch_bounds__(TB) void insp_bscatter_kernel(DevIndex ix, InsWs ws) {
  __shared__ ChunkParts cp;
  __shared__ uint32_t cnt[NSUB_MAX], tstart[NSUB_MAX], run[NSUB_MAX], wt[TB / 64];
  __shared__ Cand sc[TILE2];
  __shared__ uint16_t ssub[TILE2];
  const int g = blockIdx.x / KCH, c = blockIdx.x % KCH, t = threadIdx.x;
  const uint32_t nsub = uint32_t(ws.hdr->nsub);
  const uint32_t *b2 = ws.base2 + (uint64_t(g) * KCH + c) * NSUB_MAX;
  for (uint32_t s = t; s < NSUB_MAX; s += TB) {
    run[s] = s < nsub ? b2[s] : 0;
    cnt[s] = 0;
  }
  chunk_parts(ws, g, c, cp);  // synchronises
  const uint32_t m = cp.pre[SEG_PER_CH];
  for (uint32_t t0 = 0; t0 < m; t0 += TILE2) {
    Cand e[U2];
    uint32_t sub[U2], rk[U2];
#pragma unroll
    for (int u = 0; u < U2; ++u) {
      const uint32_t v = t0 + u * TB + t;
      e[u] = v < m ? *chunk_item(ws, cp, v) : Cand{0, 0};
    }
#pragma unroll
    for (int u = 0; u < U2; ++u) {
      const uint32_t s = bin_of(e[u].key, ix.n_buckets, ix.nb_inv, nsub) - uint32_t(g) * nsub;
      sub[u] = s < nsub ? s : nsub - 1;
      rk[u] = t0 + u * TB + t < m ? atomicAdd(&cnt[sub[u]], 1u) : 0;
    }
    __syncthreads();
    // exclusive scan of the tile's bin counts
    constexpr int Q = NSUB_MAX / TB;
    uint32_t q[Q], sum = 0;
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      q[j] = cnt[t * Q + j];
      sum += q[j];
    }
    uint32_t x = sum;
    const int lane = t & 63, wave = t >> 6;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane == 63) wt[wave] = x;
    __syncthreads();
    uint32_t pre = x - sum;
    for (int i = 0; i < wave; ++i) pre += wt[i];
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      tstart[t * Q + j] = pre;
      pre += q[j];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U2; ++u) {
      if (t0 + u * TB + t < m) {
        const uint32_t p = tstart[sub[u]] + rk[u];
        sc[p] = e[u];
        ssub[p] = uint16_t(sub[u]);
      }
    }
    __syncthreads();
    const uint32_t in_tile = m - t0 < uint32_t(TILE2) ? m - t0 : uint32_t(TILE2);
#pragma unroll
    for (int u = 0; u < U2; ++u) {
      const uint32_t p = u * TB + t;
      if (p < in_tile) {
        const uint32_t s = ssub[p];
        ws.bcand[run[s] + (p - tstart[s])] = sc[p];
      }
    }
    __syncthreads();
    for (uint32_t s = t; s < nsub; s += TB) {
      run[s] += cnt[s];
      cnt[s] = 0;
    }
    __syncthreads();
  }
}

// Enter candidate (key, mine) in a bin's LDS pair table (the pair table's rule: a slot's
// key is claimed first, then its instance; the same pair keeps the lowest request).
__device__ __forceinline__ void lds_pair(unsigned long long *tk, unsigned long long *tw, uint64_t key,
                                         uint64_t mine) {
  uint32_t h = uint32_t(mix64(key ^ ((mine >> 32) * 0xC2B2AE3D27D4EB4Full))) & (DT - 1);
  for (int step = 0; step < DT; ++step, h = (h + 1) & (DT - 1)) {
    unsigned long long k = tk[h];
    if (k == KEY_EMPTY) k = atomicCAS(&tk[h], 0ull, (unsigned long long)key);
    if (k != KEY_EMPTY && k != key) continue;
    unsigned long long w = tw[h];
    while (true) {
      if (w == 0) {
        const unsigned long long prev = atomicCAS(&tw[h], 0ull, (unsigned long long)mine);
        if (prev == 0) return;
        w = prev;
        continue;
      }
      if ((w >> 32) == (mine >> 32)) {
        if (mine < w) atomicMin(&tw[h], (unsigned long long)mine);
        return;
      }
      break;  // another instance's pair: keep probing
    }
  }
}

// Dedupe pass: each bin of at most BIN_CAP candidates is deduplicated in an LDS pair
// table and its distinct pairs written to the front of its range of np (the rest get
// KEY_EMPTY); a larger bin sends its candidates through the fallback pair table in
// place.  Workgroups take bins in order; a bin's candidates are loaded (all at once)
// before its table is cleared.
constexpr int DD_T = 512;
constexpr int DD_U = BIN_CAP / DD_T;
static_assert(BIN_CAP % DD_T == 0 && DT % DD_T == 0, "whole candidates and slots per thread");
__global__ __launch_bounds__(DD_T) void insp_bdedupe_kernel(InsWs ws) {
  __shared__ unsigned long long tk[DT], tw[DT];
  __shared__ uint32_t wt[DD_T / 64];
  __shared__ unsigned int nfb;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const uint32_t nbin = uint32_t(ws.hdr->nsub) * NREG;
  const uint64_t nd2 = ws.hdr->n_dd2;
  for (uint32_t b = blockIdx.x; b < nbin; b += gridDim.x) {
    const uint32_t lo = ws.bstart[b], hi = ws.bstart[b + 1], m = hi - lo;
    if (m == 0) {
      if (t == 0) ws.bdist[b] = 0;
      continue;
    }
    if (m > uint32_t(BIN_CAP)) {
      if (t == 0) nfb = 0;
      __syncthreads();
      uint32_t mine = 0;
      for (uint32_t k = lo + t; k < hi; k += DD_T) {
        const Cand e = ws.bcand[k];
        const int64_t h = dedupe_pair(ws, nd2, e.key, e.w2);
        ws.np[k] = h >= 0 ? NewPair{e.key, NP_FALLBACK | uint64_t(h)} : NewPair{KEY_EMPTY, 0};
        mine += h >= 0;
      }
      if (mine) atomicAdd(&nfb, mine);
      __syncthreads();
      if (t == 0) ws.bdist[b] = nfb;
      __syncthreads();
      continue;
    }
    Cand e[DD_U];
#pragma unroll
    for (int u = 0; u < DD_U; ++u) {
      const uint32_t k = lo + u * DD_T + t;
      e[u] = k < hi ? ws.bcand[k] : Cand{KEY_EMPTY, 0};
    }
    for (int j = t; j < DT; j += DD_T) {
      tk[j] = 0;
      tw[j] = 0;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < DD_U; ++u)
      if (e[u].key != KEY_EMPTY) lds_pair(tk, tw, e[u].key, e[u].w2);
    __syncthreads();
    // compact the occupied slots: thread t owns slots [t Q, t Q + Q)
    constexpr int Q = DT / DD_T;
    uint32_t occ = 0;
#pragma unroll
    for (int j = 0; j < Q; ++j) occ += tk[t * Q + j] != KEY_EMPTY;
    uint32_t x = occ;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane == 63) wt[wave] = x;
    __syncthreads();
    uint32_t pre = x - occ, total = 0;
#pragma unroll
    for (int i = 0; i < DD_T / 64; ++i) {
      pre += i < wave ? wt[i] : 0;
      total += wt[i];
    }
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      const unsigned long long k = tk[t * Q + j];
      if (k != KEY_EMPTY) ws.np[lo + pre++] = NewPair{uint64_t(k), uint64_t(tw[t * Q + j])};
    }
    for (uint32_t k = lo + total + t; k < hi; k += DD_T) ws.np[k] = NewPair{KEY_EMPTY, 0};
    if (t == 0) ws.bdist[b] = total;
    __syncthreads();
  }
}

__global__ __launch_bounds__(TB) void insp_check_kernel(DevIndex ix, InsWs ws) {
  const unsigned long long c = sum_counts(ws.bdist, uint32_t(ws.hdr->nsub) * NREG);
  if (threadIdx.x != 0) return;
  WsHdr *h = ws.hdr;
  h->n_new = c;
  const int e = h->err != 0 ? h->err : (ix.hdr->n_entries + c > ix.capacity ? SMETRIC_EFULL : 0);
  if (e != 0) {
    h->abort = 1;
    set_status(ix.hdr, e);
  } else {
    ix.hdr->n_entries += c;
  }
}

// The refreshes, when the classify pass could not do them (run by the placement's grid
// after its pairs: placement claims only empty slots, so the two never touch one value
// except an entry that both raise to the same epoch).
__device__ void refresh_pass(const DevIndex &ix, const ProbeView &pv, const InsWs &ws, uint32_t epoch) {
  const uint64_t n = pv.hdr->n;
  const uint64_t span = uint64_t(gridDim.x) * TB;
  for (uint64_t i = uint64_t(blockIdx.x) * TB + threadIdx.x; i < n; i += span) {
    const uint64_t p = ws.pos[i];
    if (!p) continue;
    uint64_t *vp = val_ptr(ix, int64_t(p - 1));
    const uint64_t v = *vp;
    if (val_epoch(v) < epoch) *vp = val_raise_epoch(v, epoch);
  }
}

// place: the distinct new pairs in bin order (so in region order), all FLAT_WG
// workgroups advancing through it together
__global__ __launch_bounds__(TB) void insp_place_kernel(DevIndex ix, ProbeView pv, InsWs ws,
                                                        const uint32_t *session, uint32_t epoch) {
  if (ws.hdr->abort) return;
  const uint64_t n = ws.hdr->n_cand;
  const uint64_t span = uint64_t(gridDim.x) * TB;
  for (uint64_t p0 = uint64_t(blockIdx.x) * TB; p0 < n; p0 += span) {  // whole workgroups iterate together
    const uint64_t p = p0 + threadIdx.x;
    int64_t tk = -1, df = -1;
    bool rf = false;
    if (p < n) {
      const NewPair e = ws.np[p];
      if (e.key != KEY_EMPTY) {
        const uint64_t w2 = np_w2(e, ws.dd);  // a fallback pair's lowest request
        bool trig;
        const int pl = place_new(ix, e.key, dd_inst(w2), epoch, session[dd_req(w2)], trig, true);
        if (pl == FAILED) set_status(ix.hdr, SMETRIC_EINTERNAL);
        else if (pl == DEFERRED) df = int64_t(p);
        else if (pl == REFRESHED) rf = true;  // a block past its probe bound that was an entry
        else if (trig) tk = int64_t(p);
      }
    }
    uncount_refreshed(ix, rf);
    append_wave(&ws.hdr->n_trig, ws.trig, ws.list_cap, tk);  // queue by np position
    append_wave(&ws.hdr->n_def, ws.def, ws.list_cap, df);
  }
  if (!ws.hdr->inl) refresh_pass(ix, pv, ws, epoch);
}

// ---------------------------------------------------------------------------------
// Evict / dump
// ---------------------------------------------------------------------------------
// All live entries (plain and member slots; headers are not entries): each round's tile of
// TB x GB buckets in slot order, the tiles wherever their round's reservation fell.
// Each thread takes GB consecutive buckets per round; a workgroup reserves its round's
// output with one atomic (one per entry made a single counter the bottleneck).  Optional
// outputs: each entry's slot (bit 63 set for a member slot) and the number of tombstones,
// added once per wavefront at the end; with hist1, the eviction's second selection digit
// (the epoch's low 11 bits) is counted over the entries whose first digit is 0, in LDS,
// each thread folding runs of its last EC distinct epochs in registers first.
constexpr int GB = 2;
constexpr int EC = 4;
__global__ __launch_bounds__(TB) void gather_kernel(DevIndex ix, uint64_t *keys, uint64_t *vals, uint64_t *pos,
                                                    unsigned long long *count, unsigned long long *n_tomb,
                                                    unsigned long long *hist1, uint64_t *toff, uint64_t cap) {
  __shared__ uint32_t wt[TB / 64];
  __shared__ unsigned long long wg_base;
  __shared__ uint32_t h1[2048];
  __shared__ uint64_t stage[TB * GB * SLOTS];  // one round's entries, one array at a time
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t per_round = uint64_t(TB) * GB;
  uint32_t tombs = 0, d0_or = 0, d0_and = ~0u;  // the entries' first selection digit (epoch >> 11)
  uint32_t ce[EC], cn[EC];                       // cached epochs (low bits) and their counts
#pragma unroll
  for (int j = 0; j < EC; ++j) cn[j] = ce[j] = 0;
  if (hist1) {
    for (int b = threadIdx.x; b < 2048; b += TB) h1[b] = 0;
    __syncthreads();
  }
  for (uint64_t b0 = uint64_t(blockIdx.x) * per_round; b0 < ix.n_buckets; b0 += uint64_t(gridDim.x) * per_round) {
    uint32_t live = 0;  // bit s + SLOTS * g: slot s of bucket g is an entry
    uint64_t k[GB][SLOTS], v[GB][SLOTS];
#pragma unroll
    for (int g = 0; g < GB; ++g) {
      const uint64_t b = b0 + uint64_t(threadIdx.x) * GB + g;
      const ulonglong2 *p = reinterpret_cast<const ulonglong2 *>(ix.slots + (b < ix.n_buckets ? b : 0) * BUCKET_WORDS);
#pragma unroll
      for (int i = 0; i < SLOTS / 2; ++i) {
        const ulonglong2 kk = p[i], vv = p[SLOTS / 2 + i];
        k[g][2 * i] = kk.x;
        k[g][2 * i + 1] = kk.y;
        v[g][2 * i] = vv.x;
        v[g][2 * i + 1] = vv.y;
      }
#pragma unroll
      for (int s = 0; s < SLOTS; ++s) {
        if (b < ix.n_buckets && k[g][s] != KEY_EMPTY && k[g][s] != KEY_TOMB && val_kind(v[g][s]) != HEADER) {
          live |= 1u << (g * SLOTS + s);
          const uint32_t ep = val_epoch(v[g][s]);
          d0_or |= ep >> 11;
          d0_and &= ep >> 11;
          if (hist1 && (ep >> 11) == 0) {
            bool hit = false;
#pragma unroll
            for (int j = 0; j < EC; ++j)
              if (!hit && (cn[j] == 0 || ce[j] == ep)) {
                ce[j] = ep;
                ++cn[j];
                hit = true;
              }
            if (!hit) atomicAdd(&h1[ep], 1u);
          }
        }
        tombs += b < ix.n_buckets && k[g][s] == KEY_TOMB;
      }
    }
    // exclusive prefix of the live counts over the workgroup
    const uint32_t c = __popc(live);
    uint32_t x = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane == 63) wt[wave] = x;
    __syncthreads();
    uint32_t before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < TB / 64; ++w) {
      before += w < wave ? wt[w] : 0;
      total += wt[w];
    }
    if (threadIdx.x == 0) {
      wg_base = total ? atomicAdd(count, (unsigned long long)total) : 0;
      if (toff) toff[b0 / per_round] = (uint64_t(wg_base) << 16) | total;  // rounds land anywhere
    }
    __syncthreads();
    // the round's entries go out through LDS, one array at a time, so that consecutive
    // lanes write consecutive words (a lane writing its own entries straight out scatters
    // every store instruction over 64 lines)
    const uint32_t lo = before + x - c;  // this thread's first entry in the round
    const unsigned long long base = wg_base;
    const uint32_t n_out = base >= cap ? 0u : (cap - base < total ? uint32_t(cap - base) : total);
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      if (a == 2 && !pos) break;  // uniform
      uint32_t j = lo;
#pragma unroll
      for (int g = 0; g < GB; ++g)
#pragma unroll
        for (int s = 0; s < SLOTS; ++s)
          if ((live >> (g * SLOTS + s)) & 1)
            stage[j++] = a == 0 ? k[g][s]
                                : (a == 1 ? val_dump(v[g][s])
                                          : ((b0 + uint64_t(threadIdx.x) * GB + g) * SLOTS + s) |
                                                (uint64_t(val_kind(v[g][s]) == MEMBER) << 63));
      __syncthreads();
      uint64_t *out = a == 0 ? keys : (a == 1 ? vals : pos);
      for (uint32_t i = threadIdx.x; i < n_out; i += TB) out[base + i] = stage[i];
      __syncthreads();  // stage, wt and wg_base are reused
    }
  }
  if (hist1) {
#pragma unroll
    for (int j = 0; j < EC; ++j)
      if (cn[j]) atomicAdd(&h1[ce[j]], cn[j]);
    __syncthreads();
    for (int b = threadIdx.x; b < 2048; b += TB)
      if (h1[b]) atomicAdd(&hist1[b], (unsigned long long)h1[b]);
  }
  if (n_tomb) {  // n_tomb[1], n_tomb[2]: OR and AND of the first selection digit
    uint32_t t = tombs, o = d0_or, a = d0_and;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
      t += __shfl_xor(t, d, 64);
      o |= __shfl_xor(o, d, 64);
      a &= __shfl_xor(a, d, 64);
    }
    if (lane == 0) {
      if (t) atomicAdd(n_tomb, (unsigned long long)t);
      atomicOr(n_tomb + 1, (unsigned long long)o);
      atomicAnd(n_tomb + 2, (unsigned long long)a);
    }
  }
}

// The header slot of a key with a bitmap record (-1: none); it lies in the key's chain.
__device__ int64_t find_header(const DevIndex &ix, uint64_t key) {
  uint64_t b = home_bucket(key, ix.n_buckets);
  for (uint64_t step = 0; step < ix.n_buckets; ++step, b = next_bucket(b, ix.n_buckets)) {
    const uint64_t *bk = ix.slots + b * BUCKET_WORDS;
    for (int s = 0; s < SLOTS; ++s) {
      const uint64_t k = bk[s];
      if (k == KEY_EMPTY) return -1;
      if (k == key && val_kind(bk[SLOTS + s]) == HEADER) return int64_t(b * SLOTS + s);
    }
  }
  return -1;
}

// Eviction as a selection: the m-th smallest entry under (epoch, key, instance) is found
// digit by digit -- epoch in two 11-bit digits, the key in five 12-bit digits and a last
// 4-bit part joined with the instance's top 6 bits, then the instance's low 10 bits --
// each digit fixed by one histogram pass over the entries that share the digits fixed
// so far.  Entries up to and including that bin under the lexicographic digit order are
// evicted, and the table is rebuilt from the entries above it.  Entries are in
// the dump's value format (instance << 48 | epoch << 24 | session).
constexpr int SEL_LEVELS = 9;
constexpr int SEL_BINS = 4096;
struct SelPrefix {
  int level;  // digits fixed so far
  uint32_t digit[SEL_LEVELS];
};
__device__ __forceinline__ uint32_t sel_digit(uint64_t key, uint64_t v, int l) {
  const uint32_t ep = dump_epoch(v), inst = dump_inst(v);
  switch (l) {
    case 0: return ep >> 11;
    case 1: return ep & 0x7FFu;
    case 2: return uint32_t(key >> 52);
    case 3: return uint32_t(key >> 40) & 0xFFFu;
    case 4: return uint32_t(key >> 28) & 0xFFFu;
    case 5: return uint32_t(key >> 16) & 0xFFFu;
    case 6: return uint32_t(key >> 4) & 0xFFFu;
    case 7: return (uint32_t(key & 15) << 6) | (inst >> 10);
    default: return inst & 0x3FFu;
  }
}
// -1: below the prefix (evicted), 0: on it, 1: above it
__device__ __forceinline__ int sel_cmp(uint64_t key, uint64_t v, const SelPrefix &p) {
  for (int l = 0; l < p.level; ++l) {
    const uint32_t d = sel_digit(key, v, l);
    if (d != p.digit[l]) return d < p.digit[l] ? -1 : 1;
  }
  return 0;
}
// Rebuild, second pass: the entries the tile pass left (tile k's listed by gathered index
// in list[seg, seg + count), toff[k] = seg << 16 | count), one per thread (all survivors:
// the tile pass skips evicted entries).  Claims that trigger a key's conversion or are
// deferred are queued by gathered index for the spill and deferred passes.
__global__ __launch_bounds__(TB) void rebuild_claim_kernel(DevIndex ix, const uint64_t *__restrict__ keys,
                                                           const uint64_t *__restrict__ vals, const uint64_t *list,
                                                           const uint64_t *__restrict__ toff, uint64_t n_tiles,
                                                           uint64_t *trig, unsigned long long *n_trig, uint64_t *def,
                                                           unsigned long long *n_def, uint64_t cap) {
  for (uint64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x)  // whole workgroups iterate together
  for (uint32_t i0 = 0; i0 < uint32_t(toff[tile] & 0xFFFF); i0 += TB) {
    const uint64_t seg = toff[tile] >> 16;
    const uint32_t n = uint32_t(toff[tile] & 0xFFFF);
    const uint32_t i = i0 + threadIdx.x;
    int64_t tk = -1, df = -1;
    if (i < n) {
      const uint64_t t = list[seg + i];
      const uint64_t k = keys[t], v = vals[t];
      bool trg;
      const int pl = place_new(ix, k, dump_inst(v), dump_epoch(v), dump_session(v), trg, true);
      if (pl == FAILED || pl == REFRESHED) set_status(ix.hdr, SMETRIC_EINTERNAL);  // survivors are distinct
      else if (pl == DEFERRED) df = int64_t(t);
      else if (trg) tk = int64_t(t);
    }
    append_wave(n_trig, trig, cap, tk);
    append_wave(n_def, def, cap, df);
  }
}

// Rebuild, first pass: workgroup k writes the whole of the cleared table's tile k (the
// gather's round of TB x GB buckets), assembled in LDS.  The gather wrote each tile's
// entries in slot order, so the entries whose old slot lay in the tile are one
// contiguous run.  The surviving plain entries whose home bucket lies in the tile are
// placed without a walk: with c(b) of them homed at bucket b, home b's entries take the
// consecutive slots from S(b) on, S(b) = max(SLOTS b, S(b - 1) + c(b - 1)), i.e. with P
// the exclusive prefix sum of c, S(b) = P(b) + max over j <= b of (SLOTS j - P(j)).  Every
// slot from an entry's home bucket up to its own is then taken, as linear probing
// requires, and the class bit of each entry past its home bucket goes into that bucket's
// mask.  Everything else -- members (a key's plain slots are capped at T + 1 before its
// conversion, which the claim pass enforces), entries homed in another tile, entries past
// the tile's last slot -- is listed for the claim pass, which enters it from its home
// bucket in the written table: tile k's list takes the gathered indexes of its entries'
// run, left_list[seg, seg + count), and toff[k] becomes seg << 16 | count.
__global__ __launch_bounds__(TB) void rebuild_tile_kernel(DevIndex ix, const uint64_t *__restrict__ keys,
                                                          const uint64_t *__restrict__ vals,
                                                          const uint64_t *__restrict__ pos, uint64_t *toff,
                                                          SelPrefix cut, uint64_t *left_list) {
  constexpr int RT = TB * GB;
  constexpr int PER = RT * SLOTS / TB;  // entries of the run per thread
  static_assert(RT == 2 * TB, "two buckets per thread in the scans");
  __shared__ uint64_t tb[RT * BUCKET_WORDS];  // the tile: keys, then values, per bucket
  __shared__ uint32_t tm[RT];                 // the tile's displacement masks
  __shared__ uint32_t hc[RT];                 // entries homed at each bucket, then S(b)
  __shared__ uint32_t wsum[TB / 64], wmax[TB / 64];
  __shared__ uint16_t lo[RT * SLOTS];         // the entries left, as offsets in the run
  __shared__ uint32_t n_lo;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const uint64_t b_lo = uint64_t(blockIdx.x) * RT;
  const uint64_t nb = ix.n_buckets - b_lo < uint64_t(RT) ? ix.n_buckets - b_lo : uint64_t(RT);
  const uint64_t seg = toff[blockIdx.x] >> 16;
  const uint32_t cnt = uint32_t(toff[blockIdx.x] & 0xFFFF);  // <= RT * SLOTS
  for (int i = t; i < RT * BUCKET_WORDS; i += TB) tb[i] = (i % BUCKET_WORDS) < SLOTS ? KEY_EMPTY : VAL_UNSET;
  for (int i = t; i < RT; i += TB) tm[i] = hc[i] = 0;
  if (t == 0) n_lo = 0;
  __syncthreads();
  // thread t takes entries t + TB u of the run: survivors homed in the tile count
  // themselves at their home (the count is their rank there), the rest are listed
  uint64_t k[PER], v[PER];
  uint32_t home[PER], rank[PER];  // home: offset in the tile, RT when not placed here
  bool member[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {  // every load issued before any is used
    const uint32_t i = uint32_t(u * TB + t), c = i < cnt ? i : 0u;
    k[u] = keys[seg + c];
    v[u] = vals[seg + c];
    member[u] = pos[seg + c] >> 63;
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const uint32_t i = uint32_t(u * TB + t);
    home[u] = RT;
    rank[u] = 0;
    if (i < cnt && sel_cmp(k[u], v[u], cut) > 0) {  // survives
      const uint64_t h = home_bucket(k[u], ix.n_buckets);
      if (!member[u] && h >= b_lo && h < b_lo + nb) {
        home[u] = uint32_t(h - b_lo);
        rank[u] = atomicAdd(&hc[home[u]], 1u);
      } else {
        lo[atomicAdd(&n_lo, 1u)] = uint16_t(i);
      }
    }
  }
  __syncthreads();
  // S(b) over the tile: thread t holds buckets 2t, 2t + 1; exclusive sums P and running
  // maxima of SLOTS j - P(j) across the workgroup (wavefront scans, then the waves' totals)
  const uint32_t c0 = hc[2 * t], c1 = hc[2 * t + 1];
  uint32_t sum = c0 + c1;  // inclusive prefix sum over the threads
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(sum, d, 64);
    if (lane >= d) sum += y;
  }
  if (lane == 63) wsum[wave] = sum;
  __syncthreads();
  uint32_t before = 0;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  const uint32_t p0 = before + sum - c0 - c1, p1 = p0 + c0;  // P(2t), P(2t + 1)
  int32_t m = int32_t(SLOTS * 2 * t) - int32_t(p0);
  const int32_t m1 = int32_t(SLOTS * (2 * t + 1)) - int32_t(p1);
  m = m1 > m ? m1 : m;  // this thread's maximum; then inclusive running maxima
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int32_t y = __shfl_up(m, d, 64);
    if (lane >= d && y > m) m = y;
  }
  if (lane == 63) wmax[wave] = uint32_t(m);
  __syncthreads();
  int32_t mb = INT32_MIN;  // the maximum over the earlier threads
  for (int w = 0; w < wave; ++w) mb = int32_t(wmax[w]) > mb ? int32_t(wmax[w]) : mb;
  {
    const int32_t prev = __shfl_up(m, 1, 64);
    if (lane > 0 && prev > mb) mb = prev;
  }
  const int32_t a0 = int32_t(SLOTS * 2 * t) - int32_t(p0), a1 = int32_t(SLOTS * (2 * t + 1)) - int32_t(p1);
  const int32_t m0 = a0 > mb ? a0 : mb, m01 = a1 > m0 ? a1 : m0;
  __syncthreads();  // every c(b) read before S(b) replaces it
  hc[2 * t] = uint32_t(int32_t(p0) + m0);
  hc[2 * t + 1] = uint32_t(int32_t(p1) + m01);
  __syncthreads();
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    if (home[u] == RT) continue;
    const uint32_t at = hc[home[u]] + rank[u];  // slot index in the tile
    if (at >= uint32_t(nb) * SLOTS) {           // past the tile's last slot
      lo[atomicAdd(&n_lo, 1u)] = uint16_t(u * TB + t);
      continue;
    }
    const uint32_t b = at / SLOTS, s = at % SLOTS;
    tb[b * BUCKET_WORDS + s] = k[u];
    tb[b * BUCKET_WORDS + SLOTS + s] = make_val(dump_inst(v[u]), PLAIN, dump_epoch(v[u]), dump_session(v[u]));
    if (b > home[u]) atomicOr(&tm[home[u]], 1u << (2 * key_cls(k[u]) + (b == home[u] + 1 ? 0 : 1)));
  }
  __syncthreads();
  const uint32_t n_left = n_lo;
  for (uint32_t j = t; j < n_left; j += TB) left_list[seg + j] = seg + lo[j];
  if (t == 0) toff[blockIdx.x] = (seg << 16) | n_left;
  for (uint64_t i = t; i < nb; i += TB) {
    if (MASK_W == 16) reinterpret_cast<uint16_t *>(ix.mask)[b_lo + i] = uint16_t(tm[i]);
    else ix.mask[b_lo + i] = uint8_t(tm[i]);
  }
  ulonglong2 *dst = reinterpret_cast<ulonglong2 *>(ix.slots + b_lo * BUCKET_WORDS);
  const ulonglong2 *src = reinterpret_cast<const ulonglong2 *>(tb);
  for (uint64_t w = t; w < nb * (BUCKET_WORDS / 2); w += TB) dst[w] = src[w];
}

// Enter the deferred pairs once their keys are converted (or, with the pool exhausted,
// as further plain slots).  Items index `keys` (and `vals`) directly, or through
// `via` into the dedupe table `dd` (insert: session of the lowest request).
__global__ void deferred_kernel(DevIndex ix, const uint64_t *items, const unsigned long long *n_items,
                                const int *abort_flag, const uint64_t *via, const DSlot *dd,
                                const uint32_t *session, uint32_t epoch, const uint64_t *keys,
                                const uint64_t *vals, const NewPair *np) {
  if (abort_flag && *abort_flag) return;
  const uint64_t n = *n_items;
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t t = items[i];
    bool trig;
    int pl;
    if (np) {
      const NewPair e = np[t];
      const uint64_t w2 = np_w2(e, dd);
      pl = place_new(ix, e.key, dd_inst(w2), epoch, session[dd_req(w2)], trig, false);
    } else if (via) {
      const DSlot d = dd[via[t]];
      pl = place_new(ix, d.key, dd_inst(d.w2), epoch, session[dd_req(d.w2)], trig, false);
    } else {
      const uint64_t v = vals[t];
      pl = place_new(ix, keys[t], dump_inst(v), dump_epoch(v), dump_session(v), trig, false);
    }
    if (pl == REFRESHED && !np && !via) pl = FAILED;  // rebuild survivors are distinct
    if (pl != PLACED && pl != REFRESHED) set_status(ix.hdr, SMETRIC_EINTERNAL);
    uncount_refreshed(ix, pl == REFRESHED);
  }
}

__global__ void set_counts_kernel(IndexHdr *h, unsigned long long n_entries, int reset_records) {
  h->n_entries = n_entries;
  if (reset_records) h->rec_used = 0;
}

// Eviction in place: the gathered entries at or below the cut become tombstones (a member
// also leaves its key's bitmap); every other entry keeps its slot.  Tombstones are never
// reclaimed by inserts, so the caller rebuilds the table instead once they would pass an
// eighth of the slots.
__device__ void tomb_entry(const DevIndex &ix, uint64_t k, uint64_t v, uint64_t ps) {
  const uint64_t slot = ps & ~(uint64_t(1) << 63);
  ix.slots[(slot / SLOTS) * BUCKET_WORDS + slot % SLOTS] = KEY_TOMB;
  if (ps >> 63) {
    const int64_t h = find_header(ix, k);
    if (h < 0) {
      set_status(ix.hdr, SMETRIC_EINTERNAL);
      return;
    }
    const uint64_t rec = val_rec(*val_ptr(ix, h));
    const uint32_t inst = dump_inst(v);
    atomicAnd(reinterpret_cast<unsigned long long *>(&ix.pool[rec * uint64_t(ix.words) + (inst >> 6)]),
              ~(1ull << (inst & 63)));
  }
}
__global__ __launch_bounds__(TB) void evict_tomb_kernel(DevIndex ix, const uint64_t *__restrict__ keys,
                                                        const uint64_t *__restrict__ vals,
                                                        const uint64_t *__restrict__ pos, uint64_t n, SelPrefix cut) {
  const uint64_t stride = uint64_t(gridDim.x) * TB;
  for (uint64_t i = uint64_t(blockIdx.x) * TB + threadIdx.x; i < n; i += stride) {
    const uint64_t k = keys[i], v = vals[i];
    if (sel_cmp(k, v, cut) <= 0) tomb_entry(ix, k, v, pos[i]);  // at or below the cut
  }
}

// One selection pass: the histogram of the next digit over the entries on the prefix.
// With ck non-null those entries are also copied to (ck, cv) (in no particular order; the
// caller does so only when few are left), so the later passes read them alone.  TOMB
// (eviction in place, on the copying pass, which reads every entry): the entries below
// the prefix, all of them evicted, become tombstones here, and the copied entries' slot
// words go to cpos for the last tombstone pass over the copies alone.
template <bool TOMB>
__global__ __launch_bounds__(TB) void sel_hist_kernel(const uint64_t *keys, const uint64_t *vals, uint64_t n,
                                                      SelPrefix p, unsigned long long *hist, uint64_t *ck,
                                                      uint64_t *cv, unsigned long long *n_c, DevIndex ix,
                                                      const uint64_t *pos, uint64_t *cpos) {
  __shared__ uint32_t h[SEL_BINS];
  for (int b = threadIdx.x; b < SEL_BINS; b += TB) h[b] = 0;
  __syncthreads();
  const uint64_t stride = uint64_t(gridDim.x) * TB;
  for (uint64_t i = uint64_t(blockIdx.x) * TB + threadIdx.x; i < n; i += stride) {
    const uint64_t k = keys[i], v = vals[i];
    const int c = sel_cmp(k, v, p);
    if (c == 0) {
      atomicAdd(&h[sel_digit(k, v, p.level)], 1u);
      if (ck) {
        const unsigned long long at = atomicAdd(n_c, 1ull);
        ck[at] = k;
        cv[at] = v;
        if (TOMB) cpos[at] = pos[i];
      }
    } else if (TOMB && c < 0) {
      tomb_entry(ix, k, v, pos[i]);
    }
  }
  __syncthreads();
  for (int b = threadIdx.x; b < SEL_BINS; b += TB)
    if (h[b]) atomicAdd(&hist[b], (unsigned long long)h[b]);
}
struct EvictWs {
  unsigned long long *count;  // gathered entries, conversion queue, deferred pairs, survivors
  unsigned long long *hist;   // SEL_BINS counts of the eviction's selection passes
  uint64_t *ka, *va, *kb, *vb;  // entries and their sort ping-pong buffers
  uint64_t *ea, *ia;            // eviction's rebuild: conversion queue and deferred pairs
  uint64_t *toff;               // eviction: per gather tile, output offset << 16 | entry count
  void *temp;
  size_t temp_bytes;
};

size_t sort_temp_bytes(uint64_t n) {
  size_t tb = 0;
  rocprim::double_buffer<uint64_t> k(nullptr, nullptr), v(nullptr, nullptr);
  if (rocprim::radix_sort_pairs(nullptr, tb, k, v, size_t(n < 1 ? 1 : n), 0u, 64u, hipStream_t(nullptr)) != hipSuccess)
    return 0;
  return tb;
}

uint64_t evict_ws_layout(uint64_t cap, EvictWs *ws, void *base) {
  const uint64_t n = cap < 1 ? 1 : cap;
  const size_t tb = sort_temp_bytes(n);
  uint64_t off = 0;
  auto take = [&](uint64_t bytes) {
    const uint64_t o = off;
    off = round_up(off + bytes, 256);
    return o;
  };
  const uint64_t o_cnt = take(256), o_hist = take(8 * SEL_BINS), o_ka = take(8 * n), o_va = take(8 * n), o_kb = take(8 * n),
                 o_vb = take(8 * n), o_ea = take(8 * n), o_ia = take(8 * n), o_toff = take(8 * (n / 512 + 64)),
                 o_tmp = take(tb);
  if (ws) {
    char *b = static_cast<char *>(base);
    ws->count = reinterpret_cast<unsigned long long *>(b + o_cnt);
    ws->hist = reinterpret_cast<unsigned long long *>(b + o_hist);
    ws->ka = reinterpret_cast<uint64_t *>(b + o_ka);
    ws->va = reinterpret_cast<uint64_t *>(b + o_va);
    ws->kb = reinterpret_cast<uint64_t *>(b + o_kb);
    ws->vb = reinterpret_cast<uint64_t *>(b + o_vb);
    ws->ea = reinterpret_cast<uint64_t *>(b + o_ea);
    ws->ia = reinterpret_cast<uint64_t *>(b + o_ia);
    ws->toff = reinterpret_cast<uint64_t *>(b + o_toff);
    ws->temp = b + o_tmp;
    ws->temp_bytes = tb;
  }
  return off;
}

int read_hdr(const smetric_index *idx, IndexHdr *out, hipStream_t s) {
  if (hipMemcpyAsync(out, idx->hdr, sizeof(IndexHdr), hipMemcpyDeviceToHost, s) != hipSuccess) return SMETRIC_EHIP;
  return hip_rc(hipStreamSynchronize(s));
}

// Gather all entries and sort them by (key, instance) for the dump.  Stable LSD radix
// passes, each over the full 64-bit sort word (restricting a pass to a bit range gave
// wrong orders for some inputs with the installed rocPRIM):
//   1) by the value word (instance << 48 | epoch << 24 | session);
//   2) stably by key -- (key, instance) is unique, so this is (key, instance) order.
// On return the sorted keys/values are in (*keys_out, *vals_out).
int gather_sorted(const smetric_index *idx, const EvictWs &ws, uint64_t n, uint64_t **keys_out,
                  uint64_t **vals_out, hipStream_t s) {
  const DevIndex ix = dev_view(idx);
  int rc = fill(ws.count, 256, 0, s);
  if (rc) return rc;
  const uint64_t n_slots = ix.n_buckets * SLOTS;
  hipLaunchKernelGGL(gather_kernel, dim3(grid_for(n_slots)), dim3(TB), 0, s, ix, ws.ka, ws.va, nullptr, ws.count,
                     nullptr, nullptr, nullptr, n);
  if ((rc = hip_rc(hipGetLastError()))) return rc;
  unsigned long long got = 0;
  if (hipMemcpyAsync(&got, ws.count, 8, hipMemcpyDeviceToHost, s) != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
    return SMETRIC_EHIP;
  if (got != n) return SMETRIC_EINTERNAL;
  *keys_out = ws.ka;
  *vals_out = ws.va;
  if (n <= 1) return SMETRIC_OK;
  size_t tb = ws.temp_bytes;
  rocprim::double_buffer<uint64_t> vk(ws.va, ws.vb), kv(ws.ka, ws.kb);
  if (rocprim::radix_sort_pairs(ws.temp, tb, vk, kv, size_t(n), 0u, 64u, s) != hipSuccess) return SMETRIC_EHIP;
  rocprim::double_buffer<uint64_t> k2(kv.current(), kv.alternate()), v2(vk.current(), vk.alternate());
  tb = ws.temp_bytes;
  if (rocprim::radix_sort_pairs(ws.temp, tb, k2, v2, size_t(n), 0u, 64u, s) != hipSuccess) return SMETRIC_EHIP;
  *keys_out = k2.current();
  *vals_out = v2.current();
  return SMETRIC_OK;
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_index_bytes(uint64_t capacity, int32_t n_instances, uint64_t n_slots, uint64_t *bytes) {
  Layout L;
  if (!bytes || !layout_for(capacity, n_instances, n_slots, L)) return SMETRIC_EINVAL;
  *bytes = L.bytes;
  return SMETRIC_OK;
}

extern "C" int smetric_index_attach(smetric_index *idx, void *mem, uint64_t mem_bytes, uint64_t capacity,
                                    int32_t n_instances, uint64_t n_slots) {
  return attach(idx, mem, mem_bytes, capacity, n_instances, n_slots);
}

extern "C" int smetric_index_init(smetric_index *idx, void *mem, uint64_t mem_bytes, uint64_t capacity,
                                  int32_t n_instances, uint64_t n_slots, hipStream_t stream) {
  int rc = attach(idx, mem, mem_bytes, capacity, n_instances, n_slots);
  if (rc) return rc;
  Layout L;
  layout_for(capacity, n_instances, n_slots, L);
  if (int rc2 = fill(mem, L.bytes, 0, stream)) return rc2;
  // every slot EMPTY with an unset value
  hipLaunchKernelGGL(unset_values_kernel, dim3(grid_for(L.n_buckets)), dim3(TB), 0, stream, idx->slots, L.n_buckets);
  return hip_rc(hipGetLastError());
}

extern "C" int smetric_index_stats(const smetric_index *idx, uint64_t *n_entries, int32_t *status,
                                   int32_t reset_status, hipStream_t stream) {
  if (!idx || !idx->hdr) return SMETRIC_EINVAL;
  IndexHdr h;
  int rc = read_hdr(idx, &h, stream);
  if (rc) return rc;
  if (n_entries) *n_entries = h.n_entries;
  if (status) *status = h.status;
  if (reset_status) {
    hipLaunchKernelGGL(set_int_kernel, dim3(1), dim3(1), 0, stream, &static_cast<IndexHdr *>(idx->hdr)->status, 0);
    if ((rc = hip_rc(hipGetLastError()))) return rc;
    rc = hip_rc(hipStreamSynchronize(stream));
  }
  return rc;
}

extern "C" int smetric_index_insert_ws_bytes(int64_t n_blocks, uint64_t *ws_bytes) {
  if (n_blocks < 0 || !ws_bytes) return SMETRIC_EINVAL;
  *ws_bytes = insert_ws_layout(n_blocks, nullptr, nullptr);
  return SMETRIC_OK;
}

extern "C" int smetric_index_insert(smetric_index *idx, const uint64_t *keys, const int64_t *blk_off,
                                    int32_t n_req, int64_t n_blocks, const int32_t *instance,
                                    const uint32_t *session, uint32_t epoch, void *workspace,
                                    uint64_t ws_bytes, hipStream_t stream) {
  if (!idx || !idx->slots || n_req < 0 || n_blocks < 0 || epoch >= EPOCH_LIMIT) return SMETRIC_EINVAL;
  if (n_req == 0) return SMETRIC_OK;
  if (!blk_off || !instance || !session || (n_blocks > 0 && !keys)) return SMETRIC_EINVAL;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) ||
      ws_bytes < insert_ws_layout(n_blocks, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  InsWs ws;
  insert_ws_layout(n_blocks, &ws, workspace);
  const DevIndex ix = dev_view(idx);
  int rc;
  if ((rc = fill(ws.hdr, sizeof(WsHdr), 0, stream))) return rc;
  hipLaunchKernelGGL(dd_clear_kernel, dim3(grid_for(ws.n_dedupe)), dim3(TB), 0, stream, ws.dd, ws.n_dedupe,
                     nullptr);
  const dim3 rgrid((n_req + IW - 1) / IW), rblock(64 * IW);
  hipLaunchKernelGGL(ins_probe_kernel, rgrid, rblock, 0, stream, ix, ws, keys, blk_off, n_req, n_blocks, instance,
                     session, epoch);
  hipLaunchKernelGGL(ins_check_kernel, dim3(1), dim3(1), 0, stream, ix, ws, n_blocks);
  hipLaunchKernelGGL(ins_refresh_kernel, rgrid, rblock, 0, stream, ix, ws, blk_off, n_req, n_blocks, epoch);
  hipLaunchKernelGGL(ins_place_kernel, dim3(grid_for(uint64_t(n_blocks))), dim3(TB), 0, stream, ix, ws, session, epoch);
  hipLaunchKernelGGL(spill_kernel, dim3(64), dim3(TB), 0, stream, ix, ws.trig, &ws.hdr->n_trig, &ws.hdr->abort,
                     nullptr, ws.dd, ws.list, nullptr);
  hipLaunchKernelGGL(deferred_kernel, dim3(64), dim3(TB), 0, stream, ix, ws.def, &ws.hdr->n_def, &ws.hdr->abort,
                     ws.list, ws.dd, session, epoch, nullptr, nullptr, nullptr);
  return hip_rc(hipGetLastError());
}

extern "C" int smetric_index_evict_ws_bytes(const smetric_index *idx, uint64_t *ws_bytes) {
  if (!idx || !ws_bytes) return SMETRIC_EINVAL;
  *ws_bytes = evict_ws_layout(idx->capacity, nullptr, nullptr);
  return SMETRIC_OK;
}

extern "C" int smetric_index_evict(smetric_index *idx, uint32_t frac_num, uint32_t frac_den, void *workspace,
                                   uint64_t ws_bytes, hipStream_t stream) {
  if (!idx || !idx->slots || frac_den == 0 || frac_num > frac_den) return SMETRIC_EINVAL;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) ||
      ws_bytes < evict_ws_layout(idx->capacity, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  EvictWs ws;
  evict_ws_layout(idx->capacity, &ws, workspace);
  IndexHdr h;
  int rc = read_hdr(idx, &h, stream);
  if (rc) return rc;
  const uint64_t n = h.n_entries;
  const uint64_t m = uint64_t((static_cast<unsigned __int128>(n) * frac_num + frac_den - 1) / frac_den);
  if (m == 0) return SMETRIC_OK;
  // all entries, tile by tile in slot order
  if ((rc = fill(ws.count, 256, 0, stream)) || (rc = fill(ws.count + 5, 8, ~uint64_t(0), stream)) ||
      (rc = fill(ws.hist, 8 * 2048, 0, stream)))
    return rc;
  const DevIndex ix = dev_view(idx);
  uint64_t *pos = ws.kb;  // free until a dump: each entry's slot
  hipLaunchKernelGGL(gather_kernel, dim3(grid_for(ix.n_buckets * SLOTS)), dim3(TB), 0, stream, ix, ws.ka, ws.va,
                     pos, ws.count, ws.count + 3, ws.hist, ws.toff, n);
  unsigned long long cnt[6] = {0, 0, 0, 0, 0, 0};
  unsigned long long hh[SEL_BINS];
  if (hipMemcpyAsync(cnt, ws.count, sizeof(cnt), hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipMemcpyAsync(hh, ws.hist, 8 * 2048, hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return SMETRIC_EHIP;
  if (cnt[0] != n) return SMETRIC_EINTERNAL;
  const uint64_t n_tomb = cnt[3];
  // select the m-th smallest, one digit per pass; stop once its whole bin is evicted
  SelPrefix p{};
  uint64_t rem = m;          // rank of the m-th smallest among the entries on the prefix (1-based)
  uint64_t on_prefix = n;    // entries on the prefix
  int l0 = 0;
  if (cnt[4] == cnt[5]) {  // every entry has the same first digit (the epochs' top bits): no pass
    p.digit[0] = uint32_t(cnt[4]);
    p.level = l0 = 1;
    if (cnt[4] == 0 && rem < on_prefix) {  // and the gather counted the second digit: no pass either
      uint64_t below = 0;
      int b = 0;
      while (b < 2048 && below + hh[b] < rem) below += hh[b++];
      if (b == 2048) return SMETRIC_EINTERNAL;
      p.digit[1] = uint32_t(b);
      p.level = l0 = 2;
      rem -= below;
      on_prefix = hh[b];
    }
  }
  // few tombstones: evict in place, the survivors keep their slots.  Tombstones may take
  // an eighth of the slots, and at most half of what stays free with the live entries at
  // capacity (the same eighth under the default 3/4 sizing), so every chain keeps
  // reaching an EMPTY slot
  const uint64_t n_slots = ix.n_buckets * SLOTS;
  const uint64_t reserved = idx->capacity + uint64_t(ix.threshold) * ix.n_records;
  const uint64_t tomb_cap_free = n_slots > reserved ? (n_slots - reserved) / 2 : 0;
  const uint64_t tomb_cap = tomb_cap_free < n_slots / 8 ? tomb_cap_free : n_slots / 8;
  const bool in_place = n_tomb + m <= tomb_cap;
  const uint64_t *sk = ws.ka, *sv = ws.va, *sp = pos;  // the entries the passes read, and their slots
  uint64_t sn = n;
  for (int l = l0; l < SEL_LEVELS && rem < on_prefix; ++l) {
    p.level = l;
    // once few entries are left on the prefix, this pass copies them out and the later
    // passes read those alone
    const bool compact = sk == ws.ka && on_prefix <= (uint64_t(1) << 20);
    if ((rc = fill(ws.hist, 8 * SEL_BINS, 0, stream))) return rc;
    if (compact && (rc = fill(ws.count + 6, 8, 0, stream))) return rc;
    const int grid = grid_for(sn) < 1024 ? grid_for(sn) : 1024;
    if (in_place && compact)  // the last pass over every entry also writes the tombstones below the prefix
      hipLaunchKernelGGL(sel_hist_kernel<true>, dim3(grid), dim3(TB), 0, stream, sk, sv, sn, p, ws.hist, ws.ea,
                         ws.ia, ws.count + 6, ix, pos, ws.vb);
    else
      hipLaunchKernelGGL(sel_hist_kernel<false>, dim3(grid), dim3(TB), 0, stream, sk, sv, sn, p, ws.hist,
                         compact ? ws.ea : nullptr, compact ? ws.ia : nullptr, ws.count + 6, ix, nullptr, nullptr);
    unsigned long long n_c = 0;
    if (hipMemcpyAsync(hh, ws.hist, 8 * SEL_BINS, hipMemcpyDeviceToHost, stream) != hipSuccess ||
        (compact && hipMemcpyAsync(&n_c, ws.count + 6, 8, hipMemcpyDeviceToHost, stream) != hipSuccess) ||
        hipStreamSynchronize(stream) != hipSuccess)
      return SMETRIC_EHIP;
    if (compact) {
      if (n_c != on_prefix) return SMETRIC_EINTERNAL;
      sk = ws.ea;
      sv = ws.ia;
      sn = n_c;
      if (in_place) sp = ws.vb;  // and everything below the copies is a tombstone already
    }
    uint64_t below = 0;
    int b = 0;
    while (b < SEL_BINS && below + hh[b] < rem) below += hh[b++];
    if (b == SEL_BINS) return SMETRIC_EINTERNAL;
    p.digit[l] = uint32_t(b);
    p.level = l + 1;
    rem -= below;
    on_prefix = hh[b];  // rem == on_prefix: the whole bin goes, the prefix itself is the cut
    if (rem < on_prefix && l + 1 == SEL_LEVELS) return SMETRIC_EINTERNAL;  // the full tuple is unique
  }
  if (in_place) {  // the entries still to decide: every one, or the copies of the last full pass
    hipLaunchKernelGGL(evict_tomb_kernel, dim3(grid_for(sn)), dim3(TB), 0, stream, ix, sk, sv, sp, sn, p);
    hipLaunchKernelGGL(set_counts_kernel, dim3(1), dim3(1), 0, stream, ix.hdr, (unsigned long long)(n - m), 0);
    if ((rc = hip_rc(hipGetLastError()))) return rc;
    return hip_rc(hipStreamSynchronize(stream));
  }
  // else rebuild from the survivors (the entries above the cut, exactly n - m of them),
  // which also clears every tombstone
  uint64_t *keys = ws.ka, *vals = ws.va;
  if ((rc = fill(ix.pool, ix.n_records * uint64_t(ix.words) * 8, 0, stream))) return rc;
  hipLaunchKernelGGL(set_counts_kernel, dim3(1), dim3(1), 0, stream, ix.hdr, (unsigned long long)(n - m), 1);
  // tile pass (writes every bucket: no clear needed), then the claims for what it left
  const uint64_t n_tiles = (ix.n_buckets + TB * GB - 1) / (TB * GB);
  uint64_t *left_list = ws.vb;  // free: the entries the tile pass leaves, by gathered index
  hipLaunchKernelGGL(rebuild_tile_kernel, dim3(n_tiles), dim3(TB), 0, stream, ix, keys, vals, pos, ws.toff, p,
                     left_list);
  uint64_t *trig = ws.ea;  // free buffers: the conversion queue and the deferred pairs
  unsigned long long *n_trig = ws.count + 1;
  uint64_t *def = ws.ia;
  unsigned long long *n_def = ws.count + 2;
  hipLaunchKernelGGL(rebuild_claim_kernel, dim3(n_tiles < MAX_GRID ? n_tiles : MAX_GRID), dim3(TB), 0, stream, ix,
                     keys, vals, left_list, ws.toff, n_tiles, trig, n_trig, def, n_def, idx->capacity);
  hipLaunchKernelGGL(spill_kernel, dim3(64), dim3(TB), 0, stream, ix, trig, n_trig, nullptr, keys, nullptr, nullptr,
                     nullptr);
  // every member of a key with a bitmap record is deferred here (millions): the full grid
  hipLaunchKernelGGL(deferred_kernel, dim3(MAX_GRID), dim3(TB), 0, stream, ix, def, n_def, nullptr, nullptr, nullptr,
                     nullptr, 0u, keys, vals, nullptr);
  if ((rc = hip_rc(hipGetLastError()))) return rc;
  return hip_rc(hipStreamSynchronize(stream));
}

extern "C" int smetric_index_dump(const smetric_index *idx, uint64_t *keys_out, uint64_t *vals_out, uint64_t cap,
                                  void *workspace, uint64_t ws_bytes, uint64_t *n_out, hipStream_t stream) {
  if (!idx || !idx->slots || !n_out || (cap > 0 && (!keys_out || !vals_out))) return SMETRIC_EINVAL;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) ||
      ws_bytes < evict_ws_layout(idx->capacity, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  EvictWs ws;
  evict_ws_layout(idx->capacity, &ws, workspace);
  IndexHdr h;
  int rc = read_hdr(idx, &h, stream);
  if (rc) return rc;
  const uint64_t n = h.n_entries;
  *n_out = n;
  if (n == 0) return SMETRIC_OK;
  uint64_t *keys, *vals;
  if ((rc = gather_sorted(idx, ws, n, &keys, &vals, stream))) return rc;
  const uint64_t c = n < cap ? n : cap;
  if (c) {
    if (hipMemcpyAsync(keys_out, keys, 8 * c, hipMemcpyDeviceToDevice, stream) != hipSuccess ||
        hipMemcpyAsync(vals_out, vals, 8 * c, hipMemcpyDeviceToDevice, stream) != hipSuccess)
      return SMETRIC_EHIP;
  }
  return hip_rc(hipStreamSynchronize(stream));
}

extern "C" int smetric_index_insert_probed(smetric_index *idx, const void *probe, uint64_t probe_bytes,
                                           int32_t n_req, int64_t n_blocks, const int32_t *instance,
                                           const uint32_t *session, uint32_t epoch, void *workspace,
                                           uint64_t ws_bytes, hipStream_t stream) {
  if (!idx || !idx->slots || n_req < 0 || n_blocks < 0 || n_blocks >= (int64_t(1) << 31) || epoch >= EPOCH_LIMIT)
    return SMETRIC_EINVAL;
  if (n_req == 0) return SMETRIC_OK;
  if (!instance || !session) return SMETRIC_EINVAL;
  if (!probe || (reinterpret_cast<uintptr_t>(probe) & 255) || probe_bytes < probe_layout(n_blocks, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) ||
      ws_bytes < insert_ws_layout(n_blocks, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  ProbeView pv;
  probe_layout(n_blocks, &pv, const_cast<void *>(probe));
  InsWs ws;
  insert_ws_layout(n_blocks, &ws, workspace);
  const DevIndex ix = dev_view(idx);
  int rc;
  if ((rc = fill(ws.hdr, sizeof(WsHdr), 0, stream))) return rc;
  const dim3 flat(FLAT_WG), blk(TB);
  const dim3 chunks(NREG * KCH);
  hipLaunchKernelGGL(insp_valid_kernel, dim3(grid_for(uint64_t(n_req))), blk, 0, stream, ix, ws, instance, session,
                     n_req);
  hipLaunchKernelGGL(insp_classify_kernel, dim3(INS_WG), blk, 0, stream, ix, pv, ws, instance, session, epoch);
  hipLaunchKernelGGL(insp_size_kernel, dim3(1), blk, 0, stream, ws);
  hipLaunchKernelGGL(insp_bcount_kernel, chunks, blk, 0, stream, ix, ws);
  hipLaunchKernelGGL(insp_bscan_kernel, dim3(NREG), dim3(SCAN_T), 0, stream, ws);
  hipLaunchKernelGGL(insp_size2_kernel, dim3(grid_for(ws.n_dedupe)), blk, 0, stream, ws);
  hipLaunchKernelGGL(insp_bscatter_kernel, chunks, blk, 0, stream, ix, ws);
  hipLaunchKernelGGL(insp_bdedupe_kernel, flat, dim3(DD_T), 0, stream, ws);
  hipLaunchKernelGGL(insp_check_kernel, dim3(1), blk, 0, stream, ix, ws);
  hipLaunchKernelGGL(insp_place_kernel, dim3(PLACE_WG), blk, 0, stream, ix, pv, ws, session, epoch);
  hipLaunchKernelGGL(spill_kernel, dim3(64), blk, 0, stream, ix, ws.trig, &ws.hdr->n_trig, &ws.hdr->abort,
                     nullptr, nullptr, nullptr, ws.np);
  hipLaunchKernelGGL(deferred_kernel, dim3(64), blk, 0, stream, ix, ws.def, &ws.hdr->n_def, &ws.hdr->abort,
                     nullptr, ws.dd, session, epoch, nullptr, nullptr, ws.np);
  return hip_rc(hipGetLastError());
}
