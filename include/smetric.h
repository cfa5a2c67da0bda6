/*
 * smetric.h -- C ABI of libsmetric.so: batched request -> KV-holder matching and routing
 * for SMetric's balanced session-centric scheduler, on one MI355X (gfx950).
 *
 * Paper: "SMetric: Rethink LLM Scheduling for Serving Agents with Balanced
 * Session-centric Scheduling" (arXiv 2607.08565).  The router scores each instance i by
 * the request's local KV$ prefix hit c_i and its load (Sec. 4.1, the scoring template),
 * and SMetric's rule (Sec. 4.2, pseudocode parts (a)-(c), Eq. (1)) sticks a follow-up
 * request to the instance with the largest hit or balances it by estimated load.  This
 * library computes, for a batch of prompts:
 *   smetric_hash_blocks   block split + chained 64-bit block keys       (Sec. 3.1, App. A)
 *   smetric_match         c[r][i] = longest prefix of request r, in blocks, held by
 *                         instance i in the global block index           (Sec. 4.1)
 *   smetric_route         the stick / balance / migrate decision          (Sec. 4.2, Eq. (1))
 *   smetric_route_seq     the same decision, requests routed one at a time (Sec. 4.2 (a))
 *   smetric_route_coloc   the same decision under PD colocation           (App. B)
 *   smetric_route_seq_coloc  colocation, requests routed one at a time    (App. B, Sec. 4.2 (a))
 *   smetric_sessions      session reconstruction from block hashes        (App. A)
 *   smetric_route_loadaware  the Sec. 5.4 ablation's load-aware filter
 *   smetric_imbalance     per-window max / mean load                      (Sec. 4.1)
 *   smetric_route_score   the comparison scorers of the scoring template  (Sec. 4.1, Sec. 5)
 *   smetric_index_insert  post-route insert of every full block on the target
 *   smetric_index_evict   LRU eviction of a fraction of the entries
 *
 * Conventions (all entry points):
 *  - Pointers are DEVICE pointers owned by the caller unless marked (host).  The library
 *    never allocates device memory: the index lives in one caller-provided buffer and
 *    scratch space in a caller-provided workspace whose size a *_bytes call reports.
 *  - Work is enqueued on `stream` and the call returns before it completes, except where
 *    a call is marked "synchronizes", which waits for `stream` before returning.
 *  - Return value: SMETRIC_OK or a negative code.  Errors visible on the host (null
 *    pointers, out-of-range scalars, short workspace) are returned at once and nothing is
 *    enqueued.  Errors in device-resident inputs are found by the kernels: they never
 *    read or write out of bounds, and they record the first such error in the index's
 *    sticky status word (read it with smetric_index_stats) or in `status` (hash).
 *  - Not thread-safe per index: calls on one index must be ordered on one stream.
 *  - Reserved key values: 0 and 2^64-1 never appear as block keys.
 */
#ifndef SMETRIC_H
#define SMETRIC_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  SMETRIC_OK = 0,
  SMETRIC_EINVAL = -1,     /* bad argument or bad device-resident input           */
  SMETRIC_EFULL = -2,      /* insert would exceed the index capacity (no change)  */
  SMETRIC_EHIP = -3,       /* a HIP runtime call failed                           */
  SMETRIC_EWORKSPACE = -4, /* workspace missing or too small                      */
  SMETRIC_EINTERNAL = -5   /* an internal bound was hit (should not happen)       */
};

/* Library version as (major << 16 | minor). */
int smetric_version(void);

/* ---------------------------------------------------------------------------------
 * Block split (Sec. 3.1: reuse is measured at KV$-block granularity; App. A: a prompt
 * is a sequence of block hashes).  Request r's tokens are tokens[tok_off[r] ..
 * tok_off[r+1]); its blocks are its first floor(len/B) B-token pieces, the trailing
 * partial block is never hashed.
 *
 * smetric_block_offsets (host only, no GPU work): tok_off (host, int64[n_req+1]) ->
 * blk_off (host, int64[n_req+1], blk_off[0] = 0, exclusive prefix sum of floor(len/B)),
 * *n_blocks (host) = blk_off[n_req].  EINVAL if a length is negative or B is not an even
 * number in [2, 256].
 * --------------------------------------------------------------------------------- */
int smetric_block_offsets(const int64_t *tok_off, int32_t n_req, int32_t block_size,
                          int64_t *blk_off, int64_t *n_blocks);

/* Chained 64-bit block keys (the paper fixes only that a prompt is identified by its
 * chained block hashes; the function is the SMH64-v1 reading):
 *   constants from SplitMix64 (Steele, Lea, Flood, OOPSLA 2014) seeded with `seed`:
 *     K_t = low 32 bits of output t for t < B, M = output B with its low bit set,
 *     s_init = output B+1;
 *   d_j   = sum_{k<B/2} (x[2k]+K[2k] mod 2^32) * (x[2k+1]+K[2k+1] mod 2^32) mod 2^64
 *           (the NH digest of UMAC), x = the block's tokens as uint32;
 *   e_j   = F(d_j + j), F = the SplitMix64 finaliser, j = block index in the request;
 *   s_j   = M * s_{j-1} + e_j mod 2^64, s_{-1} = s_init;
 *   key_j = F(s_j), then 0 -> 1 and 2^64-1 -> 2^64-2.
 * key_j depends on exactly the first (j+1)*B tokens, so equal key sequences mean equal
 * prompt prefixes (up to 64-bit collisions).
 *
 *   tokens   int32[n_tokens]          token IDs (any values; used as uint32 bit patterns)
 *   tok_off  int64[n_req+1]           request r = tokens[tok_off[r] .. tok_off[r+1])
 *   blk_off  int64[n_req+1]           output range of request r in keys; must satisfy
 *                                     blk_off[r+1]-blk_off[r] = floor(len_r / B)
 *                                     (smetric_block_offsets computes it)
 *   keys     uint64[n_blocks] (out)   keys[blk_off[r] + j] = key_j of request r
 *   status   int32[1] or NULL         set to SMETRIC_EINVAL (if it is still 0) when a
 *                                     request's offsets are inconsistent or out of range;
 *                                     that request's keys are not written.  The caller
 *                                     clears it.
 * Host errors: EINVAL for n_req < 0, n_tokens < 0, n_blocks < 0, bad block_size, or a
 * null pointer with n_req > 0.
 */
int smetric_hash_blocks(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_off,
                        const int64_t *blk_off, int32_t n_req, int64_t n_blocks,
                        int32_t block_size, uint64_t seed, uint64_t *keys, int32_t *status,
                        hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Global block index: the router's view of every instance's local KV$ (the paper's
 * "kvc", Sec. 4.1, which the router "already knows"; its structure is not described).
 * Semantically a set of entries (key, instance), each with the producing session
 * (24 bits) and the epoch (22 bits) of its last insert.  Physically: an open-addressing
 * table in HBM of 128-byte buckets (8 keys, then 8 values) with linear bucket probing;
 * keys held by more than a threshold of instances keep a holder bitmap in a side pool.
 * --------------------------------------------------------------------------------- */
typedef struct smetric_index {
  /* set by smetric_index_init / smetric_index_attach; treat as read-only */
  void *mem;               /* caller's device buffer holding the whole index        */
  uint64_t mem_bytes;
  uint64_t capacity;       /* maximum number of live entries                        */
  int32_t n_instances;     /* instances are 0 .. n_instances-1, n_instances <= 65536 */
  int32_t bitmap_words;    /* ceil(n_instances / 64)                                */
  int32_t spill_threshold; /* keys with more holders use a bitmap record             */
  int32_t reserved0;
  uint64_t n_buckets;
  uint64_t n_records;      /* bitmap records in the side pool                       */
  uint64_t *slots;         /* n_buckets * 16 words                                  */
  uint64_t *pool;          /* n_records * bitmap_words words                        */
  void *hdr;               /* device counters: entry count, status, pool use        */
} smetric_index;

/* Device bytes needed for an index of `capacity` live entries over `n_instances`
 * instances.  n_slots = 0 sizes the table so that it is at most 3/4 full at capacity
 * (headers and tombstones of keys with holder bitmaps included); otherwise the table has
 * n_slots slots (rounded up to whole 8-slot buckets), which must leave at least 1/16 of
 * them free at capacity.  A fuller table probes longer chains; in-place eviction then
 * allows fewer tombstones (half the slots free at capacity, at most an eighth of all
 * slots) before it rebuilds the table instead.
 * EINVAL if capacity == 0 or > 2^40, n_instances is not in [1, 65536], or n_slots is
 * nonzero and too small (or > 2^41). */
int smetric_index_bytes(uint64_t capacity, int32_t n_instances, uint64_t n_slots, uint64_t *bytes /* host */);

/* Lays the index out in `mem` (>= smetric_index_bytes, 256-byte aligned) and clears it on
 * `stream`.  `idx` (host) is filled in.  EINVAL on bad sizes, EHIP if the clear cannot
 * launch. */
int smetric_index_init(smetric_index *idx, void *mem, uint64_t mem_bytes, uint64_t capacity,
                       int32_t n_instances, uint64_t n_slots, hipStream_t stream);

/* Like init but leaves the buffer's contents alone: attaches `idx` to an index whose
 * bytes were copied from another buffer laid out with the same capacity, n_instances and
 * n_slots (a snapshot / restore of the whole index is a plain device copy of the bytes
 * smetric_index_bytes reports).  No GPU work; EINVAL as for init. */
int smetric_index_attach(smetric_index *idx, void *mem, uint64_t mem_bytes, uint64_t capacity,
                         int32_t n_instances, uint64_t n_slots);

/* Entry count and sticky status (0 or the first device-detected error).  Synchronizes.
 * Pass reset_status != 0 to clear the status afterwards. */
int smetric_index_stats(const smetric_index *idx, uint64_t *n_entries /* host */,
                        int32_t *status /* host */, int32_t reset_status, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Match: c[r][i] = the largest m such that instance i holds the keys of blocks 0..m-1 of
 * request r -- the request's local prefix hit on instance i, in blocks (Sec. 4.1: c_i is
 * the prefix hit length of the prompt in instance i's local KV$; Sec. 3.1: measured at
 * block granularity).  An instance drops out at its first missing block, so a cached
 * block whose ancestors are gone does not count.
 *
 *   keys     uint64[n_blocks]          from smetric_hash_blocks
 *   blk_off  int64[n_req+1]            request r's keys are keys[blk_off[r] .. blk_off[r+1])
 *   matched  int32[n_req * n_instances] (out), row-major: matched[r * n_instances + i]
 * A request whose range is decreasing or leaves [0, n_blocks] gets an all-zero row and
 * sets status EINVAL.  Reads the index; writes only `matched` and the status word.
 */
int smetric_match(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off,
                  int32_t n_req, int64_t n_blocks, int32_t *matched, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Region-ordered probe: the same question as smetric_match (which instances hold each
 * block's key, Sec. 4.1), asked once per block of a batch and answered into a probe
 * state that both smetric_match_probed and smetric_index_insert_probed consume, so the
 * post-route insert needs no second lookup.  Blocks are first partitioned by table
 * region and probed region by region, which keeps the random reads of the index inside
 * a small window of HBM at any moment.
 *
 * smetric_probe_ws_bytes: bytes of the probe state for n_blocks (< 2^32) blocks.
 * smetric_probe: requests must tile the keys: blk_off[0] = 0, non-decreasing,
 *   blk_off[n_req] = n_blocks; otherwise the probe state is marked invalid and the
 *   consumers report EINVAL.  `probe` is caller device memory (256-byte aligned) that the
 *   caller keeps unchanged until the consumers have run; the index must not change in
 *   between (the descriptors describe its state at probe time).
 * smetric_match_probed: exactly smetric_match's output (Sec. 4.1), read from the probe
 *   state; an invalid probe state gives all-zero rows and status EINVAL.
 * smetric_index_insert_probed: exactly smetric_index_insert's effect (same validation,
 *   all-or-nothing, EINVAL/EFULL in the status word) for the probed batch, with
 *   instance/session per request as there; an invalid probe state gives EINVAL.  Its
 *   batch must have n_blocks < 2^31.
 * Host errors: EINVAL (bad scalars, n_blocks >= 2^32; >= 2^31 for the insert), EWORKSPACE
 * (short buffers).
 * --------------------------------------------------------------------------------- */
int smetric_probe_ws_bytes(int64_t n_blocks, uint64_t *bytes /* host */);
int smetric_probe(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                  int64_t n_blocks, void *probe, uint64_t probe_bytes, hipStream_t stream);
/* smetric_probe in two halves, for pipelining consecutive batches:
 *   smetric_probe_partition  validates the tiling and orders the batch's blocks by table
 *                            region; it reads only the index geometry, never its contents, so it
 *                            may run while an earlier batch still inserts into the index;
 *   smetric_probe_lookup     reads the index (the descriptors then describe the index as it is
 *                            when this runs), after smetric_probe_partition on the same state,
 *                            with the same keys, blk_off, n_req and n_blocks.
 * smetric_probe = smetric_probe_partition followed by smetric_probe_lookup on one stream.
 * The lookup first bounds each request's probes: the match never reads past a request's
 * first block that no instance holds, so a search over the request's blocks (about 30
 * probes) finds one such block and the blocks from it on are not probed.  They get the
 * NONE descriptor, which is exact for the bound itself and never read by the match for
 * the others; smetric_index_insert_probed takes them as new pairs and turns any that are
 * entries (a block whose ancestors were evicted) into refreshes.  The bound is applied
 * only while the index cannot overflow whatever those blocks are (entries + n_blocks <=
 * capacity), so the insert's capacity check stays exact; otherwise every block is probed.
 * smetric_probe_stats (synchronizes): blocks the last lookup on the state probed, and the
 * probes its bound's searches made. */
int smetric_probe_partition(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off,
                            int32_t n_req, int64_t n_blocks, void *probe, uint64_t probe_bytes,
                            hipStream_t stream);
int smetric_probe_lookup(const smetric_index *idx, void *probe, uint64_t probe_bytes, const uint64_t *keys,
                         const int64_t *blk_off, int32_t n_req, int64_t n_blocks, hipStream_t stream);
int smetric_probe_stats(const void *probe, uint64_t probe_bytes, int64_t n_blocks, uint64_t *n_probed /* host */,
                        uint64_t *n_search /* host */, hipStream_t stream);

/* smetric_hash_partition: smetric_hash_blocks (the block keys, Sec. 3.1 and App. A)
 * followed by smetric_probe_partition on the keys it writes, in one call; for
 * block_size = 16 the hash kernel takes the partition's region counts itself, so the keys
 * are not read back for counting.  Arguments are those of the two calls (tokens, tok_off,
 * blk_off, keys, status as in smetric_hash_blocks; idx, probe, probe_bytes as in
 * smetric_probe_partition); afterwards `keys` holds the block keys and the probe state is
 * ready for smetric_probe_lookup, exactly as after the two calls.  A request whose token
 * range does not match its block range sets status EINVAL, as in smetric_hash_blocks,
 * and (block_size 16) also marks the probe state invalid, so its consumers report EINVAL.
 * Host errors: those of the two calls. */
int smetric_hash_partition(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_off,
                           const int64_t *blk_off, int32_t n_req, int64_t n_blocks, int32_t block_size,
                           uint64_t seed, uint64_t *keys, int32_t *status, const smetric_index *idx,
                           void *probe, uint64_t probe_bytes, hipStream_t stream);
int smetric_match_probed(const smetric_index *idx, const void *probe, uint64_t probe_bytes,
                         const uint64_t *keys, const int64_t *blk_off, int32_t n_req, int64_t n_blocks,
                         int32_t *matched, hipStream_t stream);
int smetric_index_insert_probed(smetric_index *idx, const void *probe, uint64_t probe_bytes, int32_t n_req,
                                int64_t n_blocks, const int32_t *instance, const uint32_t *session,
                                uint32_t epoch, void *workspace, uint64_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Route (Sec. 4.2 pseudocode (a) routing, (b) SLO checks, (c) load model; Eq. (1)).
 * All requests of the batch see the same load snapshot q.  Exact integer arithmetic in
 * nanoseconds of prefill time (PREFILL_RATE folded into the coefficients):
 *   n_i      = L - B*c[i]                                   new tokens on instance i
 *   est2(i)  = 2*q[i] + 2*c_lin*n_i + c_att*n_i*(2L - n_i)  = 2 * estimate_load
 *   meets(i) : est2(i) * slack_den <= slack_num * 2*(slo_b + slo_a*L)
 *              (always true when slack_den == 0, i.e. SLACK = +inf)
 *   prev     = argmax_i c[i], lowest instance on ties
 *   cached   : B*c[prev] * hit_den > hit_num * hist         (session_cached, strict)
 *   balance  = argmin over (est2(i), (i - start) mod I), start = (rr_base + r) mod I
 *              (the round-robin tie-break of rr_argmin)
 *   turn == 0                    -> balance, branch 0 (first turn)
 *   !cached                      -> balance, branch 1 (session evicted from local tier)
 *   meets(prev)                  -> prev,    branch 2 (stick)
 *   no instance meets            -> prev,    branch 3 (last-resort stick)
 *   otherwise                    -> balance, branch 4 (SLO migration)
 *
 *   matched   int32[n_req * n_instances]   from smetric_match
 *   prompt_len, hist_len, turn  int32[n_req]  L, est_hit in tokens (the previous prompt's
 *                                             length), turn (0 = first)
 *   q         int64[n_instances]           queued prefill per instance, ns
 *   params    (host)                       see smetric_params
 *   target    int32[n_req] (out), branch uint8[n_req] (out)
 * A request with inputs outside the domain (L < 0 or L > 2^24, hist < 0, turn < 0, some
 * c[i] < 0 or > L/B, some q[i] < 0 or >= 2^62) gets target -1, branch 255.
 * Host errors: EINVAL for n_req < 0, n_instances outside [1, 65536], parameters outside
 * their documented ranges.
 * --------------------------------------------------------------------------------- */
typedef struct smetric_params {
  int64_t c_lin;      /* ns per new token,  in [0, 2^32]  (c_linear / PREFILL_RATE) */
  int64_t c_att;      /* ns per token^2,    in [0, 2^32]  (c_attn / PREFILL_RATE)   */
  int64_t slo_b;      /* TTFT budget b, ns, in [0, 2^32]                            */
  int64_t slo_a;      /* TTFT budget a, ns per prompt token, in [0, 2^32]           */
  int32_t slack_num;  /* SLACK = slack_num / slack_den, both >= 0; den 0 = +inf     */
  int32_t slack_den;
  int32_t hit_num;    /* HIT_RATIO = hit_num / hit_den, 0 <= num < den              */
  int32_t hit_den;
  int32_t block_size; /* B, even, in [2, 256]                                       */
} smetric_params;

enum { SMETRIC_FIRST_TURN = 0, SMETRIC_EVICTED = 1, SMETRIC_STICK = 2, SMETRIC_LAST_RESORT = 3,
       SMETRIC_MIGRATE = 4, SMETRIC_MIGRATE_TPOT = 5, SMETRIC_SCORED = 6, SMETRIC_HIT_FILTER = 7,
       SMETRIC_INVALID = 255 };

int smetric_route(const int32_t *matched, int32_t n_req, int32_t n_instances,
                  const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                  const int64_t *q, const smetric_params *params /* host */, uint64_t rr_base,
                  int32_t *target, uint8_t *branch, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * The load-aware filter of the Sec. 5.4 ablation ("overloading migration"): the basic
 * session-centric rule sticks a cached follow-up (turn != 0 and session_cached(prev), as in
 * smetric_route) to prev = argmax c; the filter makes it leave prev when prev's load
 * exceeds the cluster mean by the margin m = margin_num / margin_den:
 *     load[prev] * n_instances * margin_den > (sum of loads) * (margin_den + margin_num)
 * (margin_den == 0: never leaves -- the basic rule).  Leaving, first turns and evicted
 * sessions take smetric_route's balance target.
 *   load  int64[n_instances]  queued prefill plus ongoing decode (any unit), in [0, 2^62)
 * Other arguments, domains and errors as smetric_route (a load outside its range makes
 * every request out of domain).  Branches: FIRST_TURN, EVICTED, STICK, MIGRATE (overloaded).
 * --------------------------------------------------------------------------------- */
int smetric_route_loadaware(const int32_t *matched, int32_t n_req, int32_t n_instances,
                            const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                            const int64_t *q, const int64_t *load, int32_t margin_num, int32_t margin_den,
                            const smetric_params *params /* host */, uint64_t rr_base, int32_t *target,
                            uint8_t *branch, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Load imbalance per time window (the metric of the Sec. 4.1 analysis: an instance's load
 * is its average number of running requests in a window; the imbalance is the maximum load
 * over the mean).  For window w = [w window, (w+1) window) and instance i, the sum over
 * requests r on i of the overlap of [t0[r], t1[r]) with the window (= average running
 * requests x window length, exact in integers):
 *   out_sum[w] = sum over instances, out_max[w] = maximum over instances
 * so the imbalance is out_max[w] * n_instances / out_sum[w].
 *   inst int32[n_req], t0/t1 int64[n_req]  instance and running interval (integer time unit)
 *   n_bad (device int64, out)  requests skipped: instance outside [0, n_instances) or t1 < t0
 *   workspace >= smetric_imbalance_ws_bytes(n_instances, n_windows) bytes, 256-B aligned
 * Host errors: EINVAL (bad scalars, window * (n_windows + 1) >= 2^62), EWORKSPACE.
 * --------------------------------------------------------------------------------- */
int smetric_imbalance_ws_bytes(int32_t n_instances, int32_t n_windows, uint64_t *ws_bytes /* host */);
int smetric_imbalance(const int32_t *inst, const int64_t *t0, const int64_t *t1, int64_t n_req, int32_t n_instances,
                      int64_t window, int32_t n_windows, int64_t *out_sum, int64_t *out_max, int64_t *n_bad,
                      void *workspace, uint64_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Session reconstruction from block hashes (App. A): request r follows an earlier request
 * p of the same user when turn[r] = turn[p] + 1 and r's block-key sequence starts with p's
 * (each turn extends its parent's prompt); chained, such requests form a session.
 * Readings: requests are given in arrival order (index order); when several earlier
 * requests qualify, the most recent is the parent; the empty sequence (a prompt shorter
 * than one block) is a prefix of every sequence; session[r] is the index of the first
 * request of r's chain.  Keys must be chained, as smetric_hash_blocks produces them (key j
 * determines blocks 0..j): "p's sequence is a prefix of r's" is then the single test
 * key_r[nb_p - 1] == key_p[nb_p - 1].
 *   keys, blk_off  block keys, CSR by request (n_req + 1 offsets)
 *   user           uint32[n_req]   opaque user id
 *   turn           int32[n_req]    turn number within its session (>= 0)
 *   parent         int32[n_req] (out)  parent request, or -1
 *   session        int32[n_req] (out)  index of the chain's first request
 *   status         int32 (device, optional: NULL) set to EINVAL if some request has a bad
 *                  key range or a negative turn; such a request gets parent -1, session -1
 *                  and is nobody's parent
 *   workspace      >= smetric_sessions_ws_bytes(n_req) bytes (~32 per request), 256-B aligned
 * Host errors: EINVAL (bad scalars, null pointers), EWORKSPACE.
 * --------------------------------------------------------------------------------- */
int smetric_sessions_ws_bytes(int32_t n_req, uint64_t *ws_bytes /* host */);
int smetric_sessions(const uint64_t *keys, const int64_t *blk_off, int32_t n_req, int64_t n_blocks,
                     const uint32_t *user, const int32_t *turn, int32_t *parent, int32_t *session,
                     int32_t *status, void *workspace, uint64_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Route with the online load update: the rule of smetric_route, but requests are routed
 * one at a time in index order and each routed request's prefill joins its target's
 * queue before the next is routed (Sec. 4.2 (a): q is the prefill queued when the request
 * arrives; prefill_cost is Eq. (1) with the request's hit on the target):
 *   q_r[i] = q[i] + sum over r' < r routed to i of prefill_cost(r', c[r'][i]).
 * A parallel pass first records what does not depend on the loads (domain, prev,
 * session_cached, the prefill cost on prev, the deadline); then one wavefront walks the
 * batch with the running loads kept doubled in 128 bits (exact).
 *   q_out      int64[n_instances] (out, optional: NULL) final loads in ns, rounded down
 *   workspace  >= smetric_route_seq_ws_bytes(n_req) bytes (80 per request), 256-B aligned
 * Other arguments, domains, branches and errors as smetric_route, and n_instances must be
 * <= 4096 (EINVAL otherwise); EWORKSPACE for a short workspace.  Out-of-domain requests
 * (branch 255) add no load.  The running loads must stay representable: EINVAL when
 * (2^63 + (n_req + 1) (2 C_LIN 2^24 + C_ATT 2^48)) max(slack_den, 1) >= 2^126 (the
 * largest load the batch could reach, times SLACK's denominator in the deadline check).
 * --------------------------------------------------------------------------------- */
int smetric_route_seq_ws_bytes(int32_t n_req, uint64_t *ws_bytes /* host */);
int smetric_route_seq(const int32_t *matched, int32_t n_req, int32_t n_instances,
                      const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                      const int64_t *q, const smetric_params *params /* host */, uint64_t rr_base,
                      int32_t *target, uint8_t *branch, int64_t *q_out, void *workspace,
                      uint64_t ws_bytes, hipStream_t stream);

/* smetric_route_seq without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, outputs and errors as smetric_route_seq, with the per-request
 * records kept in a scratch array inside the library -- one per GPU, 80 bytes for each of
 * smetric_route_seq_noalloc_max_req() = 65,536 requests (5 MiB), held until the process
 * ends.  Its device address is looked up on the first call on each device.  Allocates
 * nothing; returns SMETRIC_EWORKSPACE when n_req exceeds the maximum (use smetric_route_seq
 * with a workspace then), SMETRIC_EHIP if the scratch cannot be found.  Every call on a
 * GPU uses that GPU's one array: calls that overlap on one GPU (on different streams, or
 * from different threads) race, and must be ordered by the caller. */
int smetric_route_seq_noalloc_max_req(void);
int smetric_route_seq_noalloc(const int32_t *matched, int32_t n_req, int32_t n_instances,
                              const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                              const int64_t *q, const smetric_params *params /* host */, uint64_t rr_base,
                              int32_t *target, uint8_t *branch, int64_t *q_out, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Route under PD colocation (App. B pseudocode): smetric_route's rule with three changes.
 *   * TPOT filter: a colocated instance also decodes, and the new request's prefill
 *     stalls its live decodes for prefill_cost(req, c[i]) (Eq. (1)); instance i is a
 *     candidate iff that stall fits the smallest slack of its live decodes:
 *     2 C_LIN n + C_ATT n (2L - n) <= 2 tpot_slack[i].  When no instance passes, every
 *     instance is a candidate.
 *   * stick to prev iff turn != 0, prev caches the session, prev meets the TTFT check and
 *     prev is a candidate; there is no last-resort stick.
 *   * balance: argmin over the candidates of LMetric's multiplicative score
 *     est2(i) * n_running[i] (estimated load times the instance's request count), ties to
 *     the rotation order of smetric_route.
 *   tpot_slack  int64[n_instances]  smallest slack of the instance's live decodes, ns of
 *               prefill time; any value >= 2^62 means no live decode (always passes)
 *   n_running   int32[n_instances]  requests at the instance (>= 0)
 * Other arguments, domains and errors as smetric_route; a negative n_running makes every
 * request out of domain.  Branches: FIRST_TURN, EVICTED, STICK, MIGRATE (prev misses the
 * TTFT check), MIGRATE_TPOT (prev fails the TPOT filter while another instance passes).
 * --------------------------------------------------------------------------------- */
int smetric_route_coloc(const int32_t *matched, int32_t n_req, int32_t n_instances,
                        const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                        const int64_t *q, const int64_t *tpot_slack, const int32_t *n_running,
                        const smetric_params *params /* host */, uint64_t rr_base, int32_t *target,
                        uint8_t *branch, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Route under PD colocation with requests taken one at a time (App. B, whose router
 * receives one request at a time): request r is decided by smetric_route_coloc's rule on
 * the state the earlier requests of the batch left -- each routed request's prefill
 * joins its target's queue and it is one more request there:
 *   q_r[i] = q[i] + sum over r' < r routed to i of prefill_cost(r', c[r'][i]),
 *   n_r[i] = n_running[i] + number of r' < r routed to i.
 * The decode slacks stay as given: the request's own decode is not live yet (its length
 * is unknown, App. B).  The LMetric scores est2 x n are compared exactly in 192 bits.
 *   q_out      int64[n_instances] (out, optional: NULL) final loads in ns, rounded down
 *   n_out      int64[n_instances] (out, optional: NULL) final request counts
 *   workspace  >= smetric_route_seq_coloc_ws_bytes(n_req, n_instances) bytes, 256-B
 *              aligned (48 B per request, ~82 KB of candidate lists, 40 B per instance)
 * Other arguments, domains, branches and errors as smetric_route_coloc; n_instances must
 * be <= 4096 and the batch's loads representable as for smetric_route_seq (EINVAL
 * otherwise); EWORKSPACE for a short workspace.  Out-of-domain requests (branch 255)
 * change nothing.  The call enqueues about n_req / 32 + 4 kernel launches: requests are
 * decided in blocks of 32, each from a list of its 64 best candidates ranked on the state
 * before the previous block, which provably contains the exact minimum.
 * --------------------------------------------------------------------------------- */
int smetric_route_seq_coloc_ws_bytes(int32_t n_req, int32_t n_instances, uint64_t *ws_bytes /* host */);
int smetric_route_seq_coloc(const int32_t *matched, int32_t n_req, int32_t n_instances,
                            const int32_t *prompt_len, const int32_t *hist_len, const int32_t *turn,
                            const int64_t *q, const int64_t *tpot_slack, const int32_t *n_running,
                            const smetric_params *params /* host */, uint64_t rr_base, int32_t *target,
                            uint8_t *branch, int64_t *q_out, int64_t *n_out, void *workspace,
                            uint64_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * The scoring template's comparison scorers (Sec. 4.1: a request goes to the instance
 * with the lowest score f of its load and the request's KV$ hit; the scorers of the
 * Sec. 4.1 motivating analysis and the Sec. 5 baselines).  Per request r with prompt
 * length L, hit c[i] (blocks of B tokens), queued prefill q[i] and load l[i]:
 *   SMETRIC_SCORE_LOAD       f = l[i]                         load balance only (JSQ)
 *   SMETRIC_SCORE_TOKENS     f = q[i] + L - B c[i]            fewest tokens left to
 *                                                             prefill (Dynamo)
 *   SMETRIC_SCORE_PRODUCT    f = (q[i] + L - B c[i]) * l[i]   LMetric
 *   SMETRIC_SCORE_LINEAR     f = (1 - lam) l[i] / max_j l[j] + lam (1 - B c[i] / L)
 *                            the production scheduler's weighted sum of normalised load
 *                            and miss ratio, lam = lam_num / lam_den; an idle cluster
 *                            (max load 0) has normalised load 0, an empty prompt hit
 *                            ratio 0; compared exactly (times lam_den * max l * L)
 *   SMETRIC_SCORE_HIT_FILTER Preble: when some instance holds more than half the prompt
 *                            (2 B c[i] > L), the least loaded such instance (argmin l);
 *                            otherwise the weighted sum with the same lam
 * Every argmin breaks ties by smetric_route's rotation order: the first instance met
 * walking start, start + 1, ... (mod n_instances), start = (rr_base + r) mod n_instances.
 *   matched     int32[n_req * n_instances]  from smetric_match
 *   prompt_len  int32[n_req]                L, tokens
 *   q           int64[n_instances]          queued prefill per instance, tokens
 *   load        int32[n_instances]          the instance's load: its batch size (requests
 *                                           running there)
 *   target      int32[n_req] (out); branch uint8[n_req] (out): SMETRIC_SCORED, or
 *               SMETRIC_HIT_FILTER when the hit filter chose
 * A request with L < 0 or > 2^24, some c[i] < 0 or > L / B, some q[i] < 0 or >= 2^62, or
 * some load[i] < 0 gets target -1, branch SMETRIC_INVALID.
 * Host errors: EINVAL for kind outside the five, n_req < 0, n_instances outside
 * [1, 65536], block_size not even in [2, 256], and (LINEAR and HIT_FILTER only)
 * lam_den <= 0 or lam_num outside [0, lam_den].
 * --------------------------------------------------------------------------------- */
enum { SMETRIC_SCORE_LOAD = 0, SMETRIC_SCORE_TOKENS = 1, SMETRIC_SCORE_PRODUCT = 2, SMETRIC_SCORE_LINEAR = 3,
       SMETRIC_SCORE_HIT_FILTER = 4 };
int smetric_route_score(int32_t kind, const int32_t *matched, int32_t n_req, int32_t n_instances,
                        const int32_t *prompt_len, const int64_t *q, const int32_t *load, int32_t block_size,
                        int32_t lam_num, int32_t lam_den, uint64_t rr_base, int32_t *target, uint8_t *branch,
                        hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Post-route insert: every full block of request r goes on instance[r] (the routed
 * target caches the whole prompt it prefills, Sec. 2 and 4.2).  An existing (key,
 * instance) entry keeps its session and takes epoch = max(old, epoch); a new entry
 * records session[r], and a pair repeated within the batch takes the session of the
 * lowest request index.  All-or-nothing: a bad device-resident input (a request range
 * outside [0, n_blocks], total pairs > n_blocks, instance outside [0, n_instances),
 * session >= 2^24, a reserved key) sets status EINVAL, and a batch whose distinct new
 * entries would exceed the capacity sets status EFULL; either way the index is
 * unchanged.
 *
 *   keys, blk_off     as for smetric_match (request ranges must not overlap)
 *   instance          int32[n_req]     target instance per request
 *   session           uint32[n_req]    producing session per request, < 2^24
 *   epoch             host, < 2^22     batch id / recency stamp
 *   workspace         >= smetric_index_insert_ws_bytes(n_blocks) bytes, 256-B aligned
 * Host errors: EINVAL (bad scalars), EWORKSPACE (workspace too small).
 * --------------------------------------------------------------------------------- */
int smetric_index_insert_ws_bytes(int64_t n_blocks, uint64_t *ws_bytes /* host */);
int smetric_index_insert(smetric_index *idx, const uint64_t *keys, const int64_t *blk_off,
                         int32_t n_req, int64_t n_blocks, const int32_t *instance,
                         const uint32_t *session, uint32_t epoch, void *workspace,
                         uint64_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * LRU eviction of a fraction frac_num/frac_den of the entries (the paper's local tier
 * evicts; its policy is not specified): removes exactly ceil(N * num / den) entries, the
 * smallest under the total order (epoch, key, instance).  The removed slots become
 * tombstones while tombstones stay below an eighth of the table's slots; past that the
 * table is rebuilt from the survivors, which clears every tombstone.
 * Synchronizes.  EINVAL if frac_den == 0 or frac_num > frac_den.
 * Dump: all entries sorted by (key, instance) into keys_out / vals_out (device,
 * `cap` each), vals = instance << 48 | epoch << 24 | session; *n_out (host) = entry
 * count (entries beyond cap are not written).  Synchronizes.
 * Both take a workspace of >= smetric_index_evict_ws_bytes(idx) bytes.
 * --------------------------------------------------------------------------------- */
int smetric_index_evict_ws_bytes(const smetric_index *idx, uint64_t *ws_bytes /* host */);
int smetric_index_evict(smetric_index *idx, uint32_t frac_num, uint32_t frac_den,
                        void *workspace, uint64_t ws_bytes, hipStream_t stream);
int smetric_index_dump(const smetric_index *idx, uint64_t *keys_out, uint64_t *vals_out,
                       uint64_t cap, void *workspace, uint64_t ws_bytes,
                       uint64_t *n_out /* host */, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SMETRIC_H */
