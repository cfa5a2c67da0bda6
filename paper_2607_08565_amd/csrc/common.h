// Internal definitions shared by the libsmetric kernels: index layout in HBM, entry
// value packing, bucket hashing, and small wavefront helpers.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smetric.h"

namespace smk {

constexpr uint64_t KEY_EMPTY = 0;
constexpr uint64_t KEY_TOMB = ~uint64_t(0);
constexpr int SLOTS = 8;                 // slots per 128-byte bucket: 8 keys then 8 values
constexpr int BUCKET_WORDS = 2 * SLOTS;  // u64 words per bucket
constexpr uint32_t SESSION_LIMIT = 1u << 24;
constexpr uint32_t EPOCH_LIMIT = 1u << 22;
// Displacement-mask classes (see the masks below): two bits per class and bucket.
constexpr int MASK_CLASSES = 8;
constexpr int MASK_W = 2 * MASK_CLASSES;  // mask bits per bucket: 8 or 16
static_assert(MASK_W == 8 || MASK_W == 16, "a bucket's mask is one byte or one 16-bit word");

// Entry value (64 bits): epoch:22 | kind:2 | instance:16 | session:24.  The high 32-bit
// word is epoch:22 | kind:2 | the instance's high byte, so raising an entry's epoch to
// max(old, e) is one 32-bit atomic maximum on that word, without reading it first: the
// caller knows the entry's kind and instance, which are the same in both operands.
// HEADER values hold a pool record index in the low 40 bits instead (epoch 0).
enum Kind : uint32_t { PLAIN = 0, HEADER = 1, MEMBER = 2 };

__host__ __device__ inline uint64_t make_val(uint32_t inst, uint32_t kind, uint32_t epoch,
                                             uint32_t session) {
  return (uint64_t(epoch) << 42) | (uint64_t(kind) << 40) | (uint64_t(inst) << 24) | uint64_t(session);
}
__host__ __device__ inline uint32_t val_inst(uint64_t v) { return uint32_t(v >> 24) & 0xFFFFu; }
__host__ __device__ inline uint32_t val_kind(uint64_t v) { return uint32_t(v >> 40) & 3u; }
__host__ __device__ inline uint32_t val_epoch(uint64_t v) { return uint32_t(v >> 42); }
__host__ __device__ inline uint32_t val_session(uint64_t v) { return uint32_t(v) & 0xFFFFFFu; }
__host__ __device__ inline uint64_t val_rec(uint64_t v) { return v & ((uint64_t(1) << 40) - 1); }
__host__ __device__ inline uint64_t header_val(uint64_t rec) { return (uint64_t(HEADER) << 40) | rec; }
// v with its epoch replaced by max(its epoch, e)
__host__ __device__ inline uint64_t val_raise_epoch(uint64_t v, uint32_t e) {
  return val_epoch(v) < e ? (v & ((uint64_t(1) << 42) - 1)) | (uint64_t(e) << 42) : v;
}
// The same on the table, for an entry of the given kind and instance: one atomic on the
// value's high word (other fields of that word unchanged, the session word untouched).
__device__ __forceinline__ void raise_epoch_at(uint64_t *vp, uint32_t kind, uint32_t inst, uint32_t e) {
  atomicMax(reinterpret_cast<unsigned int *>(vp) + 1, (e << 10) | (kind << 8) | (inst >> 8));
}
// Value word of an EMPTY slot (kind 3, which no entry has): a slot whose key was just
// claimed still shows it until its claimant writes the value, so another placer walking
// the chain never takes it for an entry.
constexpr uint64_t VAL_UNSET = uint64_t(3) << 40;
// The dump's value layout (instance << 48 | epoch << 24 | session), also the layout of the
// gathered entries that eviction selects on and rebuilds from.
__host__ __device__ inline uint64_t val_dump(uint64_t v) {
  return (uint64_t(val_inst(v)) << 48) | (uint64_t(val_epoch(v)) << 24) | val_session(v);
}
__host__ __device__ inline uint32_t dump_inst(uint64_t d) { return uint32_t(d >> 48); }
__host__ __device__ inline uint32_t dump_epoch(uint64_t d) { return uint32_t(d >> 24) & 0x3FFFFFu; }
__host__ __device__ inline uint32_t dump_session(uint64_t d) { return uint32_t(d) & 0xFFFFFFu; }

// Device-resident counters, first 256 bytes of the index buffer.
struct IndexHdr {
  unsigned long long n_entries;
  int status;
  unsigned int pad0;
  unsigned long long rec_used;  // bitmap records handed out (may exceed n_records: exhausted)
  unsigned long long pad[29];
};
static_assert(sizeof(IndexHdr) == 256, "header size");

// Index view passed by value to kernels.
struct DevIndex {
  uint64_t *slots;
  uint64_t n_buckets;
  uint64_t *pool;
  uint64_t n_records;
  IndexHdr *hdr;
  uint64_t capacity;
  int32_t n_inst;
  int32_t words;      // bitmap words per record
  int32_t threshold;  // spill threshold T
  uint64_t nb_inv;    // floor(2^64 / n_buckets) (any value when n_buckets = 1): see scaled_floor
  uint8_t *mask;      // n_buckets displacement masks (see mask_of)
};

inline DevIndex dev_view(const smetric_index *ix) {
  DevIndex d;
  d.slots = ix->slots;
  d.n_buckets = ix->n_buckets;
  d.pool = ix->pool;
  d.n_records = ix->n_records;
  d.hdr = static_cast<IndexHdr *>(ix->hdr);
  d.capacity = ix->capacity;
  d.n_inst = ix->n_instances;
  d.words = ix->bitmap_words;
  d.threshold = ix->spill_threshold;
  d.nb_inv = d.n_buckets > 1 ? uint64_t((static_cast<unsigned __int128>(1) << 64) / d.n_buckets) : ~uint64_t(0);
  d.mask = reinterpret_cast<uint8_t *>(ix->pool + ix->n_records * uint64_t(ix->bitmap_words));  // after the pool
  return d;
}
// Bytes of the displacement masks (whole 32-bit words: they are set with 32-bit atomics).
inline uint64_t mask_bytes(uint64_t n_buckets) { return (n_buckets * (MASK_W / 8) + 3) / 4 * 4; }

// Bucket of a key: a multiplicative mix of the key mapped onto [0, n_buckets) with a
// 64x64 high product (keys from the hash are already uniform; the mix protects against
// structured caller keys).
__host__ __device__ inline uint64_t mix64(uint64_t k) {
  k ^= k >> 32;
  k *= 0xD6E8FEB86659FD93ull;
  k ^= k >> 32;
  return k;
}
__device__ inline uint64_t home_bucket(uint64_t key, uint64_t n_buckets) {
  return __umul64hi(mix64(key), n_buckets);
}
// floor(h mult / n) for h < n, h mult < 2^64, without a 64-bit division: with inv =
// floor(2^64 / n), q = floor(h mult inv / 2^64) is at most 2 below the quotient.
__device__ __forceinline__ uint64_t scaled_floor(uint64_t h, uint64_t mult, uint64_t n, uint64_t inv) {
  const uint64_t x = h * mult;
  uint64_t q = __umul64hi(x, inv);
  q += (q + 1) * n <= x;
  q += (q + 1) * n <= x;
  return q;
}
// Table regions: the bucket range split into NREG equal parts.  Probes, refreshes and
// claims are issued region by region so the pages live at any moment stay within the
// translation caches' reach (~2 GiB); few regions keep the partition's runs long.
constexpr int NREG = 16;
__device__ __forceinline__ uint32_t region_of(uint64_t key, uint64_t n_buckets, uint64_t nb_inv) {
  return uint32_t(scaled_floor(home_bucket(key, n_buckets), NREG, n_buckets, nb_inv));
}

// Bucket chain for a member entry (key, inst) of a key that uses a bitmap record: a
// pseudo-random bucket inside the region of the key's home bucket, so member lookups
// issued in region order stay inside the same window of the table.
__device__ inline uint64_t member_bucket(uint64_t key, uint32_t inst, uint64_t n_buckets, uint64_t nb_inv) {
  const uint64_t h = mix64(key ^ ((uint64_t(inst) + 1) * 0x9E3779B97F4A7C15ull));
  if (n_buckets < uint64_t(4 * NREG)) return __umul64hi(h, n_buckets);
  const uint64_t g = region_of(key, n_buckets, nb_inv);
  const uint64_t lo = g * n_buckets / NREG, hi = (g + 1) * n_buckets / NREG;
  return lo + __umul64hi(h, hi - lo);
}

__device__ inline void set_status(IndexHdr *h, int err) {
  atomicCAS(&h->status, 0, err);
}

// The 8 keys of bucket b, read as four 16-byte vectors, and the masks of slots equal to
// `key` and of EMPTY slots.  Within a bucket occupied slots form a prefix (claims take
// the first EMPTY slot of a chain and slots never become EMPTY again), so `match`
// is restricted to the slots before the first EMPTY one.
struct BucketScan {
  uint32_t match, empty;
};
__device__ __forceinline__ BucketScan scan_bucket(const uint64_t *bk, uint64_t key) {
  const ulonglong2 *p = reinterpret_cast<const ulonglong2 *>(bk);
  BucketScan r{0, 0};
#pragma unroll
  for (int i = 0; i < SLOTS / 2; ++i) {
    const ulonglong2 v = p[i];
    r.match |= (uint32_t(v.x == key) << (2 * i)) | (uint32_t(v.y == key) << (2 * i + 1));
    r.empty |= (uint32_t(v.x == KEY_EMPTY) << (2 * i)) | (uint32_t(v.y == KEY_EMPTY) << (2 * i + 1));
  }
  if (r.empty) r.match &= (r.empty & (0u - r.empty)) - 1u;
  return r;
}
__device__ __forceinline__ uint64_t next_bucket(uint64_t b, uint64_t n) { return b + 1 == n ? 0 : b + 1; }

// Displacement mask of a chain start h (a key's home bucket, or a member bucket): 16 bits,
// two per class c of 8.  An entry's class is a function of its key (of key and instance
// for a bitmap member) independent of where it lives.  Bit 2c is set once an entry of
// class c was claimed in bucket h + 1 by a walk that started at h, bit 2c + 1 once one was
// claimed at h + 2 or further.  A walk from h claims the first EMPTY slot it meets and
// slots never become EMPTY again, so every entry of class c whose chain starts at h lies
// in bucket h itself, in h + 1 under bit 2c, or -- under bit 2c + 1 -- between h + 2 and
// the first bucket with an EMPTY slot; and none lies past a bucket that holds an EMPTY
// slot.  A lookup therefore reads bucket h, and only when that is full the mask and the
// buckets its class's two bits name, instead of every bucket up to the first EMPTY slot
// (~1.7 buckets on average at 3/4 occupancy, with a long tail).  Keeping classes apart
// halves the further buckets read against one bit per distance 1..7 and a far bit (a
// simulation of the table at 0.745 occupancy: 0.19 against 0.40 per lookup of an entry).
// The mask only grows (tombstones keep their bits); a rebuild recomputes it.
__host__ __device__ inline uint32_t key_cls(uint64_t key) { return uint32_t(key) & (MASK_CLASSES - 1); }
__host__ __device__ inline uint32_t member_cls(uint64_t key, uint32_t inst) {
  return (uint32_t(key >> 3) + inst) & (MASK_CLASSES - 1);
}
__device__ __forceinline__ uint64_t wrap_bucket(uint64_t b, uint64_t n) { return b >= n ? b - n : b; }
__device__ __forceinline__ uint32_t mask_get(const DevIndex &ix, uint64_t h) {
  return MASK_W == 16 ? uint32_t(reinterpret_cast<const uint16_t *>(ix.mask)[h]) : uint32_t(ix.mask[h]);
}
// Records a claim of class cls in bucket b by a walk from h (nothing for h itself): one
// atomic OR.
__device__ __forceinline__ void mask_note(const DevIndex &ix, uint64_t h, uint64_t b, uint32_t cls) {
  const uint64_t d = b >= h ? b - h : b + ix.n_buckets - h;
  if (d == 0) return;
  const uint32_t bit = 1u << (2 * cls + (d == 1 ? 0 : 1));
  constexpr uint64_t PER_WORD = 32 / MASK_W;
  atomicOr(reinterpret_cast<unsigned int *>(ix.mask) + h / PER_WORD, bit << ((h % PER_WORD) * MASK_W));
}

// The buckets that can hold entries of class cls of a chain starting at h, in chain order.
// The walk starts at w.b = h; after each bucket, chain_next(ix, w, the bucket held an
// EMPTY slot) moves w.b to the next one or returns false.  Leaving bucket h it reads h's
// mask (set_mask gives it instead, when the caller has loaded it already).
struct ChainWalk {
  uint64_t h, b;
  uint32_t cls;
  bool at_home;    // w.b == h, the mask not consulted yet
  bool have_mask;  // set_mask was called
  bool near;       // bucket h + 1 may hold entries of the class
  bool far;        // buckets from h + 2 on may
  bool in_far;
  uint64_t steps;
};
__device__ __forceinline__ ChainWalk chain_start(uint64_t h, uint32_t cls) {
  return ChainWalk{h, h, cls, true, false, false, false, false, 0};
}
__device__ __forceinline__ void chain_set_mask(ChainWalk &w, uint32_t m) {
  w.near = (m >> (2 * w.cls)) & 1u;
  w.far = (m >> (2 * w.cls + 1)) & 1u;
  w.have_mask = true;
}
__device__ __forceinline__ bool chain_next(const DevIndex &ix, ChainWalk &w, bool had_empty) {
  const uint64_t n = ix.n_buckets;
  if (had_empty) return false;
  if (w.in_far) {  // h + 2 onwards; h and h + 1 are full, so a bucket with an EMPTY slot comes first
    if (++w.steps + 2 >= n) return false;
    w.b = next_bucket(w.b, n);
    return true;
  }
  if (w.at_home) {
    w.at_home = false;
    if (!w.have_mask) chain_set_mask(w, mask_get(ix, w.h));
    if (w.near) {
      w.b = wrap_bucket(w.h + 1, n);
      return true;
    }
  }
  if (w.far && n > 2) {
    w.in_far = true;
    w.b = wrap_bucket(w.h + 2, n);
    return true;
  }
  return false;
}

// Holder descriptor of one probed block (64 bits): kind:2 | instance:16 | x:46.
//   NONE  no entry holds the key
//   ONE   one plain holder: instance, x = its slot index
//   MANY  two or more plain holders: re-walk the chain when needed
//   HOT   bitmap record: x = record index
enum DescKind : uint32_t { D_NONE = 0, D_ONE = 1, D_MANY = 2, D_HOT = 3 };
constexpr uint64_t DESC_X_MASK = (uint64_t(1) << 46) - 1;
__host__ __device__ inline uint64_t make_desc(uint32_t kind, uint32_t inst, uint64_t x) {
  return (uint64_t(kind) << 62) | (uint64_t(inst & 0xFFFF) << 46) | (x & DESC_X_MASK);
}
__host__ __device__ inline uint32_t desc_kind(uint64_t d) { return uint32_t(d >> 62); }
__host__ __device__ inline uint32_t desc_inst(uint64_t d) { return uint32_t(d >> 46) & 0xFFFFu; }
__host__ __device__ inline uint64_t desc_x(uint64_t d) { return d & DESC_X_MASK; }

// Work split of the region-ordered kernels: a fixed grid of FLAT_WG workgroups whose
// iterations advance through the region-ordered arrays together (iteration t covers
// items [t * FLAT_WG * 256, (t + 1) * FLAT_WG * 256)), so the live window of the table
// slides; PART_WG workgroups partition contiguous chunks of blocks.
constexpr int FLAT_WG = 2048;
constexpr int PART_WG = 1024;
constexpr int WG_THREADS = 256;
inline uint64_t flat_span() { return uint64_t(FLAT_WG) * WG_THREADS; }
// items one workgroup of the fixed grid handles at most (its output segment size)
inline uint64_t flat_segment(uint64_t n) { return (n + flat_span() - 1) / flat_span() * WG_THREADS; }

// Probe state shared by smetric_probe and the calls that consume it.
struct ProbeHdr {
  int err;                          // first input error (EINVAL) found while partitioning
  int bad_key;                      // nonzero if a key is one of the two reserved values
  unsigned long long n;             // number of blocks in the state (0 when invalid)
  unsigned long long tot[NREG];     // blocks per region
  unsigned long long n_skip;        // blocks the lookup did not probe (past their request's bound)
  unsigned long long n_search;      // probes the bound's search made
};
struct ProbeView {
  ProbeHdr *hdr;
  uint32_t *req_of;     // block order: request of each block
  uint32_t *inv;        // block order: position of the block in region order
  uint32_t *hist;       // [PART_WG][NREG] blocks of each region in each partition chunk
  uint64_t *base;       // [PART_WG][NREG] first region-order position of each (chunk, region)
  uint64_t *part_key;   // region order: key
  uint32_t *part_req;   // region order: request of the block
  uint32_t *part_blk;   // region order: the block
  uint64_t *desc_p;     // region order: holder descriptor
  uint32_t *skip;       // block order, one bit per block: past its request's probe bound
  uint64_t cap;         // blocks the buffer holds
};
inline uint64_t skip_words(uint64_t n) { return (n + 31) / 32; }
inline uint64_t probe_layout(int64_t n_blocks, ProbeView *v, void *base) {
  const uint64_t n = uint64_t(n_blocks < 1 ? 1 : n_blocks);
  uint64_t off = 0;
  auto take = [&](uint64_t bytes) {
    const uint64_t o = off;
    off = (off + bytes + 255) / 256 * 256;
    return o;
  };
  const uint64_t o_hdr = take(sizeof(ProbeHdr)), o_req = take(4 * n), o_inv = take(4 * n),
                 o_hist = take(4ull * NREG * PART_WG), o_base = take(8ull * NREG * PART_WG), o_k = take(8 * n),
                 o_rq = take(4 * n), o_bk = take(4 * n), o_dp = take(8 * n), o_sk = take(4 * skip_words(n));
  if (v) {
    char *b = static_cast<char *>(base);
    v->hdr = reinterpret_cast<ProbeHdr *>(b + o_hdr);
    v->req_of = reinterpret_cast<uint32_t *>(b + o_req);
    v->inv = reinterpret_cast<uint32_t *>(b + o_inv);
    v->hist = reinterpret_cast<uint32_t *>(b + o_hist);
    v->base = reinterpret_cast<uint64_t *>(b + o_base);
    v->part_key = reinterpret_cast<uint64_t *>(b + o_k);
    v->part_req = reinterpret_cast<uint32_t *>(b + o_rq);
    v->part_blk = reinterpret_cast<uint32_t *>(b + o_bk);
    v->desc_p = reinterpret_cast<uint64_t *>(b + o_dp);
    v->skip = reinterpret_cast<uint32_t *>(b + o_sk);
    v->cap = n;
  }
  return off;
}

// Region partition of a probe state, shared by smetric_probe_partition and the hash call
// that counts the regions itself (defined with the probe).  partition_head clears the
// state (and the [chunk][region] counts when the hash is to add into them) in one launch;
// partition_tail checks the tiling and maps blocks to requests, counts (unless counted),
// scans and scatters.
int probe_state_args(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                     int64_t n_blocks, void *probe, uint64_t probe_bytes);
void partition_head(ProbeView &pv, bool clear_hist, hipStream_t stream);
int partition_tail(const DevIndex &ix, ProbeView &pv, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                   uint64_t n, bool counted, hipStream_t stream);
inline uint64_t partition_chunk(uint64_t n) { return n ? (n + PART_WG - 1) / PART_WG : 1; }

// Sizing shared by host code.
inline int32_t bitmap_words_for(int32_t n_inst) { return (n_inst + 63) / 64; }
inline int32_t threshold_for(int32_t n_inst) {
  int32_t t = (n_inst + 127) / 128;
  return t < 8 ? 8 : t;
}

inline int hip_rc(hipError_t e) { return e == hipSuccess ? SMETRIC_OK : SMETRIC_EHIP; }

}  // namespace smk
