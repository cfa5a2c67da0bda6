// SMetric matching/routing oracle: the plain, sequential CPU definition of what the
// request -> KV-holder matching hot path computes.
//
// TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads or calls this
// file; only the test suite, the smoke check and the CPU-baseline leg of the benchmark
// do. It shares no code, header, table or constant generator with the GPU library.
//
// Paper: "SMetric: Rethink LLM Scheduling for Serving Agents with Balanced
// Session-centric Scheduling" (arXiv 2607.08565).
//
// Steps, each written for obviousness rather than speed:
//   hash_blocks  block split + chained 64-bit block keys            (Sec. 3.1, App. A; reading SMH64-v1)
//   index_*      global block index: set of (key, instance) entries  (Sec. 4.1 "kvc"; readings on insert/evict)
//   match        per-request, per-instance longest matched prefix     (Sec. 4.1 score template: c_i)
//   route        stick-or-balance rule with SLO checks and Eq. (1)    (Sec. 4.2 pseudocode, parts (a)-(c))
//   route_seq    the same rule with the queue updated after every decision (Sec. 4.2 (a))
//   sessions     session reconstruction from block hashes              (App. A)
//   route_loadaware  the Sec. 5.4 ablation's load-aware filter        (Sec. 5.4)
//   imbalance    per-window max / mean load                            (Sec. 4.1 analysis)
//   route_coloc  the same rule under PD colocation                    (App. B pseudocode)
//   route_score  the comparison scorers of the scoring template        (Sec. 4.1, Sec. 5)
//
// Where the paper is silent (hash function, tie-breaks, integer units, batch semantics,
// eviction order) the choices are the readings recorded with the design notes; each is
// named at the point of use below.
//
// Parity status: the hash constants are pinned to published SplitMix64 output; the
// hash itself is pinned only by its structural properties (chained prefix identity,
// closed-form == sequential), since the paper specifies no hash.  Match is pinned by a
// hash-free brute-force longest-common-prefix model, route by hand-built decision tables
// and closed forms of Eq. (1), insert/evict by a brute-force dictionary model, the
// comparison scorers by hand-worked tables and the textbook rules they reduce to.

#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstring>
#include <map>
#include <tuple>
#include <unordered_map>
#include <vector>

namespace {

constexpr int ORC_OK = 0;
constexpr int ORC_EINVAL = -1;
constexpr int ORC_EFULL = -2;

constexpr uint64_t KEY_EMPTY = 0;           // reserved: never a key
constexpr uint64_t KEY_TOMB = ~uint64_t(0);  // reserved: never a key
constexpr uint32_t SESSION_LIMIT = 1u << 24;
constexpr uint32_t EPOCH_LIMIT = 1u << 22;

// ---------------------------------------------------------------------------------
// SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number generators",
// OOPSLA 2014): a Weyl-sequence state advanced by the golden-ratio increment, passed
// through a two-multiply xor-shift finaliser.
// ---------------------------------------------------------------------------------
uint64_t splitmix_finalise(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

uint64_t splitmix_next(uint64_t &state) {
  state += 0x9E3779B97F4A7C15ull;
  return splitmix_finalise(state);
}

// Reading SMH64-v1 (the paper fixes only "block granularity" and chained block hashes
// whose sequence identifies a prefix, Sec. 3.1 and App. A):
//   constants from SplitMix64 seeded with `seed`:
//     K_t = low 32 bits of output t (t < B);  M = output B with its low bit set;
//     s_init = output B+1
//   d_j   = sum_{k < B/2} (x[2k] + K[2k] mod 2^32) * (x[2k+1] + K[2k+1] mod 2^32)  mod 2^64
//           (the NH digest of UMAC, Black et al., CRYPTO 1999)
//   e_j   = F(d_j + j)           F = SplitMix64 finaliser, j = block index in the prompt
//   s_j   = M * s_{j-1} + e_j    (s_{-1} = s_init)
//   key_j = F(s_j), with 0 -> 1 and 2^64-1 -> 2^64-2 (both values are reserved markers)
struct HashConsts {
  std::vector<uint32_t> K;
  uint64_t M = 0;
  uint64_t s_init = 0;
};

HashConsts make_consts(uint64_t seed, int B) {
  HashConsts hc;
  uint64_t st = seed;
  for (int t = 0; t < B; ++t) hc.K.push_back(uint32_t(splitmix_next(st)));
  hc.M = splitmix_next(st) | 1ull;
  hc.s_init = splitmix_next(st);
  return hc;
}

uint64_t nh_digest(const int32_t *x, int B, const HashConsts &hc) {
  uint64_t d = 0;
  for (int k = 0; k < B / 2; ++k) {
    uint32_t a = uint32_t(x[2 * k]) + hc.K[2 * k];
    uint32_t b = uint32_t(x[2 * k + 1]) + hc.K[2 * k + 1];
    d += uint64_t(a) * uint64_t(b);
  }
  return d;
}

uint64_t remap_key(uint64_t k) {
  if (k == KEY_EMPTY) return 1;
  if (k == KEY_TOMB) return KEY_TOMB - 1;
  return k;
}

// ---------------------------------------------------------------------------------
// Global block index. The paper's router consults "kvc" for each instance's local
// prefix hit (Sec. 4.1) without describing the structure; here it is the plain set of
// entries (key, instance), each carrying the producing session and the last epoch
// (batch id) that touched it.
// ---------------------------------------------------------------------------------
struct Entry {
  uint32_t session;
  uint32_t epoch;
};

struct Index {
  uint64_t capacity = 0;
  int32_t n_inst = 0;
  uint64_t n = 0;
  int32_t status = ORC_OK;
  std::unordered_map<uint64_t, std::map<int32_t, Entry>> m;

  void set_status(int32_t e) {
    if (status == ORC_OK) status = e;
  }
};

// Request r owns keys[blk_off[r] .. blk_off[r+1]); the range must lie in [0, n_blocks].
bool range_ok(const int64_t *blk_off, int32_t r, int64_t n_blocks) {
  return blk_off[r] >= 0 && blk_off[r] <= blk_off[r + 1] && blk_off[r + 1] <= n_blocks;
}

}  // namespace

extern "C" {

// Parameters of the route step, in integer units (nanoseconds of prefill time).
// Sec. 4.2 (c) load model; Eq. (1); Sec. 4.1 TTFT SLO b + a*L; SLACK and HIT_RATIO as
// rationals (slack_den == 0 means SLACK = +infinity).
typedef struct orc_params {
  int64_t c_lin;   // ns per new token          (c_linear / PREFILL_RATE)
  int64_t c_att;   // ns per new token^2        (c_attn / PREFILL_RATE)
  int64_t slo_b;   // ns                         TTFT budget b
  int64_t slo_a;   // ns per prompt token        TTFT budget a
  int32_t slack_num, slack_den;
  int32_t hit_num, hit_den;
  int32_t block_size;
} orc_params;

// Block split and chained keys (reading SMH64-v1 above). blk_off_out gets R+1 entries:
// request r owns keys[blk_off[r] .. blk_off[r+1]); only full blocks are hashed.
int orc_hash_blocks(const int32_t *tokens, const int64_t *tok_off, int32_t n_req, int32_t B,
                    uint64_t seed, int64_t *blk_off_out, uint64_t *keys_out) {
  if (B < 2 || B > 256 || (B & 1) || n_req < 0) return ORC_EINVAL;
  HashConsts hc = make_consts(seed, B);
  blk_off_out[0] = 0;
  for (int32_t r = 0; r < n_req; ++r) {
    int64_t len = tok_off[r + 1] - tok_off[r];
    if (len < 0) return ORC_EINVAL;
    blk_off_out[r + 1] = blk_off_out[r] + len / B;
  }
  for (int32_t r = 0; r < n_req; ++r) {
    const int32_t *x = tokens + tok_off[r];
    int64_t nb = blk_off_out[r + 1] - blk_off_out[r];
    uint64_t s = hc.s_init;
    for (int64_t j = 0; j < nb; ++j) {
      uint64_t d = nh_digest(x + j * B, B, hc);
      uint64_t e = splitmix_finalise(d + uint64_t(j));
      s = hc.M * s + e;
      keys_out[blk_off_out[r] + j] = remap_key(splitmix_finalise(s));
    }
  }
  return ORC_OK;
}

// Exposes the constants for the SplitMix64 pins.
int orc_hash_consts(uint64_t seed, int32_t B, uint32_t *K_out, uint64_t *M_out,
                    uint64_t *s_init_out) {
  if (B < 2 || B > 256 || (B & 1)) return ORC_EINVAL;
  HashConsts hc = make_consts(seed, B);
  for (int t = 0; t < B; ++t) K_out[t] = hc.K[t];
  *M_out = hc.M;
  *s_init_out = hc.s_init;
  return ORC_OK;
}

uint64_t orc_splitmix_next(uint64_t *state) { return splitmix_next(*state); }

void *orc_index_new(uint64_t capacity, int32_t n_inst) {
  if (n_inst < 1 || n_inst > 65536) return nullptr;
  Index *ix = new Index;
  ix->capacity = capacity;
  ix->n_inst = n_inst;
  return ix;
}

void orc_index_free(void *h) { delete static_cast<Index *>(h); }

uint64_t orc_index_size(void *h) { return static_cast<Index *>(h)->n; }
int32_t orc_index_status(void *h) { return static_cast<Index *>(h)->status; }

// Post-route insert: every full block of request r goes on inst[r] (the routed target).
// Reading: an existing (key, instance) entry keeps its producer session and takes
// epoch = max(old, epoch); a new one records session[r] -- for pairs repeated inside one
// batch that is the session of the lowest request index, because requests are applied
// in order. The call is all-or-nothing: invalid contents (instance out of range,
// session >= 2^24, a reserved key value, inconsistent offsets) give EINVAL, and a batch
// whose distinct new entries would push the entry count past the capacity gives EFULL;
// either way the index is left unchanged and the status word records the first error.
int orc_index_insert(void *h, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                     int64_t n_blocks, const int32_t *inst, const uint32_t *session,
                     uint32_t epoch) {
  Index &ix = *static_cast<Index *>(h);
  if (n_req < 0 || n_blocks < 0 || epoch >= EPOCH_LIMIT) return ORC_EINVAL;
  int64_t n_pairs = 0;
  bool ranges = true;
  for (int32_t r = 0; r < n_req; ++r) {
    if (!range_ok(blk_off, r, n_blocks)) ranges = false;
    else n_pairs += blk_off[r + 1] - blk_off[r];
  }
  if (!ranges || n_pairs > n_blocks) {
    ix.set_status(ORC_EINVAL);
    return ORC_EINVAL;
  }
  for (int32_t r = 0; r < n_req; ++r) {
    bool bad = inst[r] < 0 || inst[r] >= ix.n_inst || session[r] >= SESSION_LIMIT;
    for (int64_t b = blk_off[r]; b < blk_off[r + 1] && !bad; ++b)
      bad = keys[b] == KEY_EMPTY || keys[b] == KEY_TOMB;
    if (bad && blk_off[r + 1] > blk_off[r]) {
      ix.set_status(ORC_EINVAL);
      return ORC_EINVAL;
    }
  }
  // Count distinct (key, instance) pairs that are not yet in the index.
  std::map<std::pair<uint64_t, int32_t>, bool> fresh;
  for (int32_t r = 0; r < n_req; ++r)
    for (int64_t b = blk_off[r]; b < blk_off[r + 1]; ++b) {
      auto it = ix.m.find(keys[b]);
      bool present = it != ix.m.end() && it->second.count(inst[r]);
      if (!present) fresh[{keys[b], inst[r]}] = true;
    }
  if (ix.n + fresh.size() > ix.capacity) {
    ix.set_status(ORC_EFULL);
    return ORC_EFULL;
  }
  for (int32_t r = 0; r < n_req; ++r)
    for (int64_t b = blk_off[r]; b < blk_off[r + 1]; ++b) {
      std::map<int32_t, Entry> &holders = ix.m[keys[b]];
      auto it = holders.find(inst[r]);
      if (it == holders.end()) {
        holders[inst[r]] = Entry{session[r], epoch};
        ix.n += 1;
      } else {
        it->second.epoch = std::max(it->second.epoch, epoch);
      }
    }
  return ORC_OK;
}

// LRU eviction of a fraction f = num/den of the entries. Reading: remove exactly
// ceil(f * N) entries, the smallest under the total order (epoch, key, instance).
int orc_index_evict(void *h, uint32_t num, uint32_t den) {
  Index &ix = *static_cast<Index *>(h);
  if (den == 0 || num > den) return ORC_EINVAL;
  uint64_t m = uint64_t((static_cast<unsigned __int128>(ix.n) * num + den - 1) / den);
  std::vector<std::tuple<uint32_t, uint64_t, int32_t>> all;
  all.reserve(ix.n);
  for (auto &kv : ix.m)
    for (auto &he : kv.second) all.emplace_back(he.second.epoch, kv.first, he.first);
  std::sort(all.begin(), all.end());
  for (uint64_t t = 0; t < m && t < all.size(); ++t) {
    uint64_t key = std::get<1>(all[t]);
    int32_t i = std::get<2>(all[t]);
    auto it = ix.m.find(key);
    it->second.erase(i);
    if (it->second.empty()) ix.m.erase(it);
    ix.n -= 1;
  }
  return ORC_OK;
}

// All entries sorted by (key, instance). vals = instance << 48 | epoch << 24 | session.
uint64_t orc_index_dump(void *h, uint64_t *keys, uint64_t *vals, uint64_t cap) {
  Index &ix = *static_cast<Index *>(h);
  std::vector<std::tuple<uint64_t, int32_t, uint32_t, uint32_t>> all;
  for (auto &kv : ix.m)
    for (auto &he : kv.second)
      all.emplace_back(kv.first, he.first, he.second.epoch, he.second.session);
  std::sort(all.begin(), all.end());
  for (uint64_t t = 0; t < all.size() && t < cap; ++t) {
    keys[t] = std::get<0>(all[t]);
    vals[t] = (uint64_t(std::get<1>(all[t])) << 48) | (uint64_t(std::get<2>(all[t])) << 24) |
              uint64_t(std::get<3>(all[t]));
  }
  return all.size();
}

// c[r][i] = the number of leading blocks of request r whose keys are all held by
// instance i: the local prefix hit of the paper's score template (Sec. 4.1), measured
// at block granularity (Sec. 3.1). The walk follows the prompt block by block and drops
// an instance at its first missing block ("first miss"), so a block cached without its
// ancestors never counts.
int orc_match(void *h, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
              int64_t n_blocks, int32_t *matched) {
  Index &ix = *static_cast<Index *>(h);
  if (n_req < 0 || n_blocks < 0) return ORC_EINVAL;
  const int32_t I = ix.n_inst;
  int rc = ORC_OK;
  for (int32_t r = 0; r < n_req; ++r) {
    int32_t *c = matched + int64_t(r) * I;
    if (!range_ok(blk_off, r, n_blocks)) {  // a request with a bad range matches nothing
      for (int32_t i = 0; i < I; ++i) c[i] = 0;
      ix.set_status(ORC_EINVAL);
      rc = ORC_EINVAL;
      continue;
    }
    int64_t nb = blk_off[r + 1] - blk_off[r];
    std::vector<bool> alive(I, true);
    int32_t n_alive = I;
    for (int32_t i = 0; i < I; ++i) c[i] = int32_t(nb);
    for (int64_t j = 0; j < nb && n_alive > 0; ++j) {
      auto it = ix.m.find(keys[blk_off[r] + j]);
      for (int32_t i = 0; i < I; ++i) {
        if (!alive[i]) continue;
        bool held = it != ix.m.end() && it->second.count(i);
        if (!held) {
          alive[i] = false;
          c[i] = int32_t(j);
          --n_alive;
        }
      }
    }
  }
  return rc;
}

// Route one batch (Sec. 4.2 pseudocode (a)-(c), Eq. (1)). All requests see the same
// load snapshot q (reading: batched routing). Integer form, exact in 128-bit:
//   n_i      = L - B*c[i]                      new tokens on instance i
//   cost2(n) = 2*C_LIN*n + C_ATT*n*(2L - n)    = 2 * Eq. (1)
//   est2(i)  = 2*q[i] + cost2(n_i)              = 2 * estimate_load
//   meets(i) : est2(i)*SLACK_den <= SLACK_num * 2*(b + a*L)   (always true for SLACK = inf)
//   cached   : B*c[prev] * HIT_den > HIT_num * hist            (strict, as in session_cached)
//   prev     = argmax c, lowest instance id on ties
//   balance  = argmin over (est2(i), (i - start) mod I), start = (rr_base + r) mod I
// branch: 0 first turn, 1 session evicted, 2 stick, 3 last-resort stick (no instance
// meets the deadline), 4 migrate; 255 = request with out-of-domain inputs (target -1).
int orc_route(const int32_t *matched, int32_t n_req, int32_t I, const int32_t *prompt_len,
              const int32_t *hist_len, const int32_t *turn, const int64_t *q,
              const orc_params *p, uint64_t rr_base, int32_t *target, uint8_t *branch) {
  typedef __int128 i128;
  const int64_t LIM32 = int64_t(1) << 32;
  if (n_req < 0 || I < 1 || I > 65536) return ORC_EINVAL;
  if (p->c_lin < 0 || p->c_lin > LIM32 || p->c_att < 0 || p->c_att > LIM32 || p->slo_b < 0 ||
      p->slo_b > LIM32 || p->slo_a < 0 || p->slo_a > LIM32 || p->slack_num < 0 ||
      p->slack_den < 0 || p->hit_num < 0 || p->hit_den <= 0 || p->hit_num >= p->hit_den ||
      p->block_size < 2 || p->block_size > 256 || (p->block_size & 1))
    return ORC_EINVAL;
  const int64_t B = p->block_size;
  bool q_ok = true;
  for (int32_t i = 0; i < I; ++i)
    if (q[i] < 0 || q[i] >= (int64_t(1) << 62)) q_ok = false;
  for (int32_t r = 0; r < n_req; ++r) {
    const int32_t *c = matched + int64_t(r) * I;
    const int64_t L = prompt_len[r];
    bool ok = q_ok && L >= 0 && L <= (int64_t(1) << 24) && hist_len[r] >= 0 && turn[r] >= 0;
    for (int32_t i = 0; ok && i < I; ++i) ok = c[i] >= 0 && c[i] <= L / B;
    if (!ok) {
      target[r] = -1;
      branch[r] = 255;
      continue;
    }
    auto est2 = [&](int32_t i) -> i128 {
      i128 n = L - B * c[i];
      return i128(2) * q[i] + i128(2) * p->c_lin * n + i128(p->c_att) * n * (i128(2) * L - n);
    };
    const i128 bound2 = i128(2) * (i128(p->slo_b) + i128(p->slo_a) * L);
    auto meets = [&](int32_t i) -> bool {
      if (p->slack_den == 0) return true;
      return est2(i) * p->slack_den <= i128(p->slack_num) * bound2;
    };
    int32_t prev = 0;
    for (int32_t i = 1; i < I; ++i)
      if (c[i] > c[prev]) prev = i;
    const int32_t start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));
    int32_t best = start;
    for (int32_t k = 1; k < I; ++k) {
      int32_t i = (start + k) % I;
      if (est2(i) < est2(best)) best = i;  // strict: the earlier rotation position wins ties
    }
    const bool none_meets = !meets(best);  // best has the minimum estimated load
    const bool cached =
        i128(B) * c[prev] * p->hit_den > i128(p->hit_num) * hist_len[r];
    if (turn[r] == 0) {
      target[r] = best;
      branch[r] = 0;
    } else if (!cached) {
      target[r] = best;
      branch[r] = 1;
    } else if (meets(prev)) {
      target[r] = prev;
      branch[r] = 2;
    } else if (none_meets) {
      target[r] = prev;
      branch[r] = 3;
    } else {
      target[r] = best;
      branch[r] = 4;
    }
  }
  return ORC_OK;
}

// Load-aware filter (the Sec. 5.4 ablation's "overloading migration"): the basic
// session-centric rule sticks a cached follow-up to prev = argmax c; with the filter it
// leaves prev when prev's load (queued prefill plus ongoing decode, a caller input)
// exceeds the cluster mean by the margin m = m_num / m_den:
//   overloaded  <=>  load[prev] * I * m_den > (sum of loads) * (m_den + m_num).
// Leaving, and the first-turn / evicted cases, balance exactly as orc_route (argmin of
// est2 with the rotation tie-break).  m_den == 0 means an infinite margin (never leave:
// the basic rule).  branch: 0 first turn, 1 evicted, 2 stick, 4 migrate (overloaded);
// 255 out of domain (also: some load[i] < 0 or >= 2^62).
int orc_route_loadaware(const int32_t *matched, int32_t n_req, int32_t I, const int32_t *prompt_len,
                        const int32_t *hist_len, const int32_t *turn, const int64_t *q, const int64_t *load,
                        int32_t m_num, int32_t m_den, const orc_params *p, uint64_t rr_base, int32_t *target,
                        uint8_t *branch) {
  typedef __int128 i128;
  if (m_num < 0 || m_den < 0) return ORC_EINVAL;
  std::vector<uint8_t> br0(n_req > 0 ? n_req : 1);
  std::vector<int32_t> t0(n_req > 0 ? n_req : 1);
  // the balance target of every request is orc_route's (first-turn requests balance)
  std::vector<int32_t> zero_turn(n_req > 0 ? n_req : 1, 0);
  int rc = orc_route(matched, n_req, I, prompt_len, hist_len, n_req ? zero_turn.data() : turn, q, p, rr_base,
                     t0.data(), br0.data());
  if (rc != ORC_OK) return rc;
  bool load_ok = true;
  i128 sum = 0;
  for (int32_t i = 0; i < I; ++i) {
    if (load[i] < 0 || load[i] >= (int64_t(1) << 62)) load_ok = false;
    sum += load[i];
  }
  const int64_t B = p->block_size;
  for (int32_t r = 0; r < n_req; ++r) {
    const int32_t *c = matched + int64_t(r) * I;
    if (br0[r] == 255 || turn[r] < 0 || !load_ok) {
      target[r] = -1;
      branch[r] = 255;
      continue;
    }
    int32_t prev = 0;
    for (int32_t i = 1; i < I; ++i)
      if (c[i] > c[prev]) prev = i;
    const bool cached = i128(B) * c[prev] * p->hit_den > i128(p->hit_num) * hist_len[r];
    const bool overloaded = m_den != 0 && i128(load[prev]) * I * m_den > sum * (i128(m_den) + m_num);
    if (turn[r] == 0) {
      target[r] = t0[r];
      branch[r] = 0;
    } else if (!cached) {
      target[r] = t0[r];
      branch[r] = 1;
    } else if (!overloaded) {
      target[r] = prev;
      branch[r] = 2;
    } else {
      target[r] = t0[r];
      branch[r] = 4;
    }
  }
  return ORC_OK;
}

// Load imbalance, Sec. 4.1 analysis: an instance's load in a window is its average number
// of running requests over the window; the imbalance is the maximum load over the mean.
// Here per window w = [w W, (w+1) W) (times in integer units, e.g. ms): for each request
// with instance i and running interval [t0, t1), its overlap with the window is added to
// instance i's load (so load = average running requests x W, exact in integers); out_sum[w]
// = the sum over instances, out_max[w] = the maximum (imbalance = out_max I / out_sum).
// Requests with i outside [0, I) or t1 < t0 are skipped and counted in *n_bad.
int orc_imbalance(const int32_t *inst, const int64_t *t0, const int64_t *t1, int64_t n_req, int32_t I,
                  int64_t window, int32_t n_windows, int64_t *out_sum, int64_t *out_max, int64_t *n_bad) {
  if (n_req < 0 || I < 1 || window <= 0 || n_windows < 0) return ORC_EINVAL;
  std::vector<int64_t> cell(size_t(n_windows) * I, 0);
  int64_t bad = 0;
  for (int64_t r = 0; r < n_req; ++r) {
    if (inst[r] < 0 || inst[r] >= I || t1[r] < t0[r]) {
      ++bad;
      continue;
    }
    for (int32_t w = 0; w < n_windows; ++w) {
      const int64_t lo = std::max(t0[r], int64_t(w) * window), hi = std::min(t1[r], int64_t(w + 1) * window);
      if (hi > lo) cell[size_t(w) * I + inst[r]] += hi - lo;
    }
  }
  for (int32_t w = 0; w < n_windows; ++w) {
    int64_t s = 0, m = 0;
    for (int32_t i = 0; i < I; ++i) {
      s += cell[size_t(w) * I + i];
      m = std::max(m, cell[size_t(w) * I + i]);
    }
    out_sum[w] = s;
    out_max[w] = m;
  }
  *n_bad = bad;
  return ORC_OK;
}

// Session reconstruction, App. A: a request is the follow-up of an earlier request of
// the same user when (1) its turn is larger by exactly one and (2) its block-hash sequence
// starts with the other's.  Readings: requests are given in arrival order (index order);
// when several earlier requests qualify, the most recent is the parent; the empty
// sequence is a prefix of every sequence; a request's session is the index of the first
// request of its chain (a request without parent starts one).  A request with a bad key
// range gets parent -1, session -1 and is nobody's parent.
int orc_sessions(const uint64_t *keys, const int64_t *blk_off, int32_t n_req, int64_t n_blocks,
                 const uint32_t *user, const int32_t *turn, int32_t *parent, int32_t *session) {
  if (n_req < 0 || n_blocks < 0) return ORC_EINVAL;
  std::vector<bool> ok(n_req);
  for (int32_t r = 0; r < n_req; ++r)
    ok[r] = blk_off[r] >= 0 && blk_off[r] <= blk_off[r + 1] && blk_off[r + 1] <= n_blocks && turn[r] >= 0;
  std::unordered_map<uint32_t, std::vector<int32_t>> by_user;  // earlier requests of each user
  for (int32_t r = 0; r < n_req; ++r) {
    parent[r] = -1;
    session[r] = -1;
    if (!ok[r]) continue;
    std::vector<int32_t> &earlier = by_user[user[r]];
    const int64_t nr = blk_off[r + 1] - blk_off[r];
    for (int32_t k = int32_t(earlier.size()) - 1; k >= 0; --k) {  // most recent first
      const int32_t p = earlier[k];
      if (turn[p] + int64_t(1) != turn[r]) continue;
      const int64_t np = blk_off[p + 1] - blk_off[p];
      if (np > nr) continue;
      bool prefix = true;
      for (int64_t j = 0; prefix && j < np; ++j) prefix = keys[blk_off[p] + j] == keys[blk_off[r] + j];
      if (prefix) {
        parent[r] = p;
        break;
      }
    }
    session[r] = parent[r] >= 0 ? session[parent[r]] : r;
    earlier.push_back(r);
  }
  return ORC_OK;
}

// Route with the paper's online load semantics (Sec. 4.2 (a), where q is the queued
// prefill at the moment each request is routed): requests are routed one at a time in index
// order, and after each decision the request's prefill joins its target's queue,
//   q[target] += prefill_cost(req, c[target])        (Eq. (1)),
// so request r sees q plus the costs of every earlier request of the batch routed to each
// instance.  The decision for each request is orc_route's with that q; loads are kept
// doubled (2q, exact with Eq. (1)'s n/2 term) in 128 bits.  Out-of-domain requests add no
// load.  q_out (optional) gets the final loads in ns, rounded down.
// Requests routed one at a time: the running loads grow with the batch, and the deadline
// check multiplies them by SLACK's denominator.  A batch is in domain only when the largest
// load it can reach -- 2 q < 2^63 plus (n_req + 1) times the largest doubled cost of a
// request in domain, 2 C_LIN 2^24 + C_ATT 2^48 -- times the denominator stays below 2^126.
static bool seq_loads_fit(const orc_params *p, int32_t n_req) {
  typedef __int128 i128;
  const i128 cmax = i128(2) * p->c_lin * (int64_t(1) << 24) + i128(p->c_att) * (i128(1) << 48);
  const i128 worst = (i128(1) << 63) + i128(int64_t(n_req) + 1) * cmax;
  return worst < (i128(1) << 126) / i128(p->slack_den > 0 ? p->slack_den : 1);
}

int orc_route_seq(const int32_t *matched, int32_t n_req, int32_t I, const int32_t *prompt_len,
                  const int32_t *hist_len, const int32_t *turn, const int64_t *q, const orc_params *p,
                  uint64_t rr_base, int32_t *target, uint8_t *branch, int64_t *q_out) {
  typedef __int128 i128;
  const int64_t LIM32 = int64_t(1) << 32;
  if (n_req < 0 || I < 1 || I > 65536) return ORC_EINVAL;
  if (p->c_lin < 0 || p->c_lin > LIM32 || p->c_att < 0 || p->c_att > LIM32 || p->slo_b < 0 ||
      p->slo_b > LIM32 || p->slo_a < 0 || p->slo_a > LIM32 || p->slack_num < 0 ||
      p->slack_den < 0 || p->hit_num < 0 || p->hit_den <= 0 || p->hit_num >= p->hit_den ||
      p->block_size < 2 || p->block_size > 256 || (p->block_size & 1))
    return ORC_EINVAL;
  if (!seq_loads_fit(p, n_req)) return ORC_EINVAL;
  const int64_t B = p->block_size;
  bool q_ok = true;
  std::vector<i128> q2(I);
  for (int32_t i = 0; i < I; ++i) {
    if (q[i] < 0 || q[i] >= (int64_t(1) << 62)) q_ok = false;
    q2[i] = i128(2) * q[i];
  }
  for (int32_t r = 0; r < n_req; ++r) {
    const int32_t *c = matched + int64_t(r) * I;
    const int64_t L = prompt_len[r];
    bool ok = q_ok && L >= 0 && L <= (int64_t(1) << 24) && hist_len[r] >= 0 && turn[r] >= 0;
    for (int32_t i = 0; ok && i < I; ++i) ok = c[i] >= 0 && c[i] <= L / B;
    if (!ok) {
      target[r] = -1;
      branch[r] = 255;
      continue;
    }
    auto cost2 = [&](int32_t i) -> i128 {  // 2 x prefill_cost(req, c[i])
      i128 n = L - B * c[i];
      return i128(2) * p->c_lin * n + i128(p->c_att) * n * (i128(2) * L - n);
    };
    auto est2 = [&](int32_t i) -> i128 { return q2[i] + cost2(i); };
    const i128 bound2 = i128(2) * (i128(p->slo_b) + i128(p->slo_a) * L);
    auto meets = [&](int32_t i) -> bool {
      if (p->slack_den == 0) return true;
      return est2(i) * p->slack_den <= i128(p->slack_num) * bound2;
    };
    int32_t prev = 0;
    for (int32_t i = 1; i < I; ++i)
      if (c[i] > c[prev]) prev = i;
    const int32_t start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));
    int32_t best = start;
    for (int32_t k = 1; k < I; ++k) {
      int32_t i = (start + k) % I;
      if (est2(i) < est2(best)) best = i;
    }
    const bool cached = i128(B) * c[prev] * p->hit_den > i128(p->hit_num) * hist_len[r];
    int32_t t;
    uint8_t br;
    if (turn[r] == 0) {
      t = best;
      br = 0;
    } else if (!cached) {
      t = best;
      br = 1;
    } else if (meets(prev)) {
      t = prev;
      br = 2;
    } else if (!meets(best)) {
      t = prev;
      br = 3;
    } else {
      t = best;
      br = 4;
    }
    target[r] = t;
    branch[r] = br;
    q2[t] += cost2(t);  // the request's prefill joins its target's queue
  }
  if (q_out)
    for (int32_t i = 0; i < I; ++i) {
      const i128 v = q2[i] / 2;
      q_out[i] = v > i128(INT64_MAX) ? INT64_MAX : int64_t(v);
    }
  return ORC_OK;
}

// Route under PD colocation, App. B pseudocode: the Sec. 4.2 rule with two changes.
//   meets_tpot(i): the request's prefill stalls i's live decodes by prefill_cost(c[i]);
//     it must fit the smallest decode slack at i:  cost2(i) <= 2 * slack[i], with cost2
//     as above; slack[i] >= 2^62 means no live decode (always passes).
//   cand = instances meeting it; when none does, every instance.
//   stick to prev iff turn != 0, session_cached(prev), meets_ttft(prev) and prev in cand;
//   otherwise balance: argmin over cand of (est2(i) * n_run[i], (i - start) mod I), the
//   multiplicative score of LMetric (estimate_load times the instance's request count).
//   There is no last-resort clause.
// branch: 0 first turn, 1 session evicted, 2 stick, 4 migrate (prev misses the TTFT check),
// 5 migrate (prev fails the TPOT filter while another instance passes); 255 out of domain
// (additionally some n_run[i] < 0).
int orc_route_coloc(const int32_t *matched, int32_t n_req, int32_t I, const int32_t *prompt_len,
                    const int32_t *hist_len, const int32_t *turn, const int64_t *q,
                    const int64_t *slack, const int32_t *n_run, const orc_params *p, uint64_t rr_base,
                    int32_t *target, uint8_t *branch) {
  typedef __int128 i128;
  const int64_t LIM32 = int64_t(1) << 32;
  if (n_req < 0 || I < 1 || I > 65536) return ORC_EINVAL;
  if (p->c_lin < 0 || p->c_lin > LIM32 || p->c_att < 0 || p->c_att > LIM32 || p->slo_b < 0 ||
      p->slo_b > LIM32 || p->slo_a < 0 || p->slo_a > LIM32 || p->slack_num < 0 ||
      p->slack_den < 0 || p->hit_num < 0 || p->hit_den <= 0 || p->hit_num >= p->hit_den ||
      p->block_size < 2 || p->block_size > 256 || (p->block_size & 1))
    return ORC_EINVAL;
  const int64_t B = p->block_size;
  const int64_t NO_DECODE = int64_t(1) << 62;
  bool inst_ok = true;
  for (int32_t i = 0; i < I; ++i)
    if (q[i] < 0 || q[i] >= (int64_t(1) << 62) || n_run[i] < 0) inst_ok = false;
  for (int32_t r = 0; r < n_req; ++r) {
    const int32_t *c = matched + int64_t(r) * I;
    const int64_t L = prompt_len[r];
    bool ok = inst_ok && L >= 0 && L <= (int64_t(1) << 24) && hist_len[r] >= 0 && turn[r] >= 0;
    for (int32_t i = 0; ok && i < I; ++i) ok = c[i] >= 0 && c[i] <= L / B;
    if (!ok) {
      target[r] = -1;
      branch[r] = 255;
      continue;
    }
    auto cost2 = [&](int32_t i) -> i128 {  // 2 x prefill_cost(req, c[i]), Eq. (1)
      i128 n = L - B * c[i];
      return i128(2) * p->c_lin * n + i128(p->c_att) * n * (i128(2) * L - n);
    };
    auto est2 = [&](int32_t i) -> i128 { return i128(2) * q[i] + cost2(i); };
    auto meets_tpot = [&](int32_t i) -> bool {
      return slack[i] >= NO_DECODE || cost2(i) <= i128(2) * slack[i];
    };
    const i128 bound2 = i128(2) * (i128(p->slo_b) + i128(p->slo_a) * L);
    auto meets_ttft = [&](int32_t i) -> bool {
      if (p->slack_den == 0) return true;
      return est2(i) * p->slack_den <= i128(p->slack_num) * bound2;
    };
    std::vector<bool> in_cand(I);
    bool any = false;
    for (int32_t i = 0; i < I; ++i) {
      in_cand[i] = meets_tpot(i);
      any = any || in_cand[i];
    }
    if (!any)
      for (int32_t i = 0; i < I; ++i) in_cand[i] = true;
    int32_t prev = 0;
    for (int32_t i = 1; i < I; ++i)
      if (c[i] > c[prev]) prev = i;
    const int32_t start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));
    int32_t best = -1;
    for (int32_t k = 0; k < I; ++k) {
      const int32_t i = (start + k) % I;
      if (!in_cand[i]) continue;
      // strict: the earlier rotation position wins ties
      if (best < 0 || est2(i) * n_run[i] < est2(best) * n_run[best]) best = i;
    }
    const bool cached = i128(B) * c[prev] * p->hit_den > i128(p->hit_num) * hist_len[r];
    if (turn[r] == 0) {
      target[r] = best;
      branch[r] = 0;
    } else if (!cached) {
      target[r] = best;
      branch[r] = 1;
    } else if (!meets_ttft(prev)) {
      target[r] = best;
      branch[r] = 4;
    } else if (!in_cand[prev]) {
      target[r] = best;
      branch[r] = 5;
    } else {
      target[r] = prev;
      branch[r] = 2;
    }
  }
  return ORC_OK;
}


// Route under PD colocation with requests taken one at a time (App. B pseudocode, whose
// req = receive() handles one request; Sec. 4.2 (a) for what q means).  Request r is
// decided exactly as orc_route_coloc decides it, on the instance state that the earlier
// requests of the batch left: after each decision the request's prefill joins its target's
// queue (q[t] += prefill_cost(req, c[t])) and the request is one more request at the target
// (n_run[t] += 1).  The TPOT filter's decode slacks are the caller's: the new request has
// no live decode yet (its decode length is unknown, App. B), so they do not change.
// Out-of-domain requests (branch 255) change nothing.  q_out (ns, halved and rounded down
// like orc_route_seq) and n_out receive the final state when non-null.
// a * x < b * y, exactly, for 0 <= a, b < 2^127 and x, y < 2^64: the products (< 2^191) are
// formed as (high 128 bits, low 64 bits).
static bool prod_less(__int128 a, uint64_t x, __int128 b, uint64_t y) {
  typedef unsigned __int128 u128;
  auto mul = [](u128 v, uint64_t m, u128 &hi, uint64_t &lo) {
    const u128 p_lo = (v & ~uint64_t(0)) * u128(m), p_hi = (v >> 64) * u128(m);
    lo = uint64_t(p_lo);
    hi = p_hi + (p_lo >> 64);
  };
  u128 ah, bh;
  uint64_t al, bl;
  mul(u128(a), x, ah, al);
  mul(u128(b), y, bh, bl);
  return ah < bh || (ah == bh && al < bl);
}

// Test hook for the comparison above: a and b as (high, low) 64-bit words.
int orc_test_prod_less(int64_t a_hi, uint64_t a_lo, uint64_t x, int64_t b_hi, uint64_t b_lo, uint64_t y) {
  const __int128 a = (__int128(a_hi) << 64) | a_lo, b = (__int128(b_hi) << 64) | b_lo;
  return prod_less(a, x, b, y) ? 1 : 0;
}

int orc_route_seq_coloc(const int32_t *matched, int32_t n_req, int32_t I, const int32_t *prompt_len,
                        const int32_t *hist_len, const int32_t *turn, const int64_t *q, const int64_t *slack,
                        const int32_t *n_run, const orc_params *p, uint64_t rr_base, int32_t *target,
                        uint8_t *branch, int64_t *q_out, int64_t *n_out) {
  typedef __int128 i128;
  const int64_t LIM32 = int64_t(1) << 32;
  if (n_req < 0 || I < 1 || I > 65536) return ORC_EINVAL;
  if (p->c_lin < 0 || p->c_lin > LIM32 || p->c_att < 0 || p->c_att > LIM32 || p->slo_b < 0 ||
      p->slo_b > LIM32 || p->slo_a < 0 || p->slo_a > LIM32 || p->slack_num < 0 ||
      p->slack_den < 0 || p->hit_num < 0 || p->hit_den <= 0 || p->hit_num >= p->hit_den ||
      p->block_size < 2 || p->block_size > 256 || (p->block_size & 1))
    return ORC_EINVAL;
  if (!seq_loads_fit(p, n_req)) return ORC_EINVAL;
  std::vector<i128> q2(I);         // 2 q, exact
  std::vector<int64_t> n(I);
  bool inst_ok = true;
  for (int32_t i = 0; i < I; ++i) {
    if (q[i] < 0 || q[i] >= (int64_t(1) << 62) || n_run[i] < 0) inst_ok = false;
    q2[i] = i128(2) * q[i];
    n[i] = n_run[i];
  }
  const int64_t B = p->block_size;
  for (int32_t r = 0; r < n_req; ++r) {
    // the batch rule on one request, with the current state (loads kept doubled, so that
    // the half-token costs of Eq. (1) stay exact; the decision compares 2q + cost2)
    const int32_t *c = matched + int64_t(r) * I;
    const int64_t L = prompt_len[r];
    bool ok = inst_ok && L >= 0 && L <= (int64_t(1) << 24) && hist_len[r] >= 0 && turn[r] >= 0;
    for (int32_t i = 0; ok && i < I; ++i) ok = c[i] >= 0 && c[i] <= L / B;
    if (!ok) {
      target[r] = -1;
      branch[r] = 255;
      continue;
    }
    auto cost2 = [&](int32_t i) -> i128 {
      const i128 m = L - B * c[i];
      return i128(2) * p->c_lin * m + i128(p->c_att) * m * (i128(2) * L - m);
    };
    const int64_t NO_DECODE = int64_t(1) << 62;
    std::vector<bool> in_cand(I);
    bool any = false;
    for (int32_t i = 0; i < I; ++i) {
      in_cand[i] = slack[i] >= NO_DECODE || cost2(i) <= i128(2) * slack[i];
      any = any || in_cand[i];
    }
    if (!any)
      for (int32_t i = 0; i < I; ++i) in_cand[i] = true;
    auto est2 = [&](int32_t i) -> i128 { return q2[i] + cost2(i); };
    const i128 bound2 = i128(2) * (i128(p->slo_b) + i128(p->slo_a) * L);
    auto meets_ttft = [&](int32_t i) -> bool {
      if (p->slack_den == 0) return true;
      return est2(i) * p->slack_den <= i128(p->slack_num) * bound2;
    };
    int32_t prev = 0;
    for (int32_t i = 1; i < I; ++i)
      if (c[i] > c[prev]) prev = i;
    const int32_t start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));
    // the loads and counts grow with every request, so the LMetric product is compared in
    // 192 bits (est2 < 2^113, n < 2^33 over any batch)
    int32_t best = -1;
    for (int32_t k = 0; k < I; ++k) {
      const int32_t i = (start + k) % I;
      if (!in_cand[i]) continue;
      if (best < 0 || prod_less(est2(i), uint64_t(n[i]), est2(best), uint64_t(n[best]))) best = i;  // earlier rotation wins ties
    }
    const bool cached = i128(B) * c[prev] * p->hit_den > i128(p->hit_num) * hist_len[r];
    int32_t t;
    uint8_t br;
    if (turn[r] == 0) {
      t = best;
      br = 0;
    } else if (!cached) {
      t = best;
      br = 1;
    } else if (!meets_ttft(prev)) {
      t = best;
      br = 4;
    } else if (!in_cand[prev]) {
      t = best;
      br = 5;
    } else {
      t = prev;
      br = 2;
    }
    target[r] = t;
    branch[r] = br;
    q2[t] += cost2(t);  // the request's prefill joins its target's queue
    n[t] += 1;          // and it is one more request at the target
  }
  if (q_out)
    for (int32_t i = 0; i < I; ++i) {
      const i128 v = q2[i] / 2;
      q_out[i] = v > i128(INT64_MAX) ? INT64_MAX : int64_t(v);
    }
  if (n_out)
    for (int32_t i = 0; i < I; ++i) n_out[i] = n[i];
  return ORC_OK;
}

// The Sec. 4.1 scoring template: each request goes to the instance that minimises a score
// f(req, i) built from the request's KV$ hit c[i] (blocks), its prompt length L, the
// prefill work q[i] already queued at i (tokens) and the instance's load l[i] (its batch
// size, i.e. requests running there).  The scorers are the ones the paper compares against
// (Sec. 4.1 motivating analysis, Sec. 5 baselines); kind selects f:
//   0 load-balance only (join the shortest queue):  f = l[i]
//   1 fewest tokens left to prefill (Dynamo):        f = q[i] + L - B c[i]
//   2 multiplicative (LMetric):                      f = (q[i] + L - B c[i]) * l[i]
//   3 weighted sum (the production scheduler):       f = (1 - lam) lhat[i] + lam (1 - chat[i])
//        lhat[i] = l[i] / max_j l[j]  (reading: normalised by the cluster maximum; an idle
//                                      cluster, max 0, has lhat = 0)
//        chat[i] = B c[i] / L         (the hit ratio; reading: 0 for an empty prompt)
//        lam = lam_num / lam_den
//   4 hit filter, then score (Preble): if some instance caches more than half the prompt
//        (2 B c[i] > L, strict), the least loaded such instance (argmin l[i]); otherwise
//        kind 3's weighted sum with the same lam
// Every argmin breaks ties by the rotation order of orc_route (the earliest of
// start, start+1, ... mod I, start = (rr_base + r) mod I; reading: the paper gives no
// tie-break for these scorers).  Kind 3's fractions are compared exactly: every f[i] of one
// request is multiplied by the same positive constant lam_den * Dl * Dc (Dl = max l or 1,
// Dc = L or 1), leaving integers.
// branch: 6 scored, 7 the hit filter chose (kind 4); 255 out of domain (target -1): L < 0
// or > 2^24, some c[i] < 0 or > L / B, some q[i] < 0 or >= 2^62, some l[i] < 0.
int orc_route_score(int32_t kind, const int32_t *matched, int32_t n_req, int32_t I, const int32_t *prompt_len,
                    const int64_t *q, const int32_t *load, int32_t block_size, int32_t lam_num, int32_t lam_den,
                    uint64_t rr_base, int32_t *target, uint8_t *branch) {
  typedef __int128 i128;
  if (kind < 0 || kind > 4 || n_req < 0 || I < 1 || I > 65536) return ORC_EINVAL;
  if (block_size < 2 || block_size > 256 || (block_size & 1)) return ORC_EINVAL;
  if ((kind == 3 || kind == 4) && (lam_den <= 0 || lam_num < 0 || lam_num > lam_den)) return ORC_EINVAL;
  const int64_t B = block_size;
  bool inst_ok = true;
  int64_t lmax = 0;
  for (int32_t i = 0; i < I; ++i) {
    if (q[i] < 0 || q[i] >= (int64_t(1) << 62) || load[i] < 0) inst_ok = false;
    lmax = std::max<int64_t>(lmax, load[i]);
  }
  for (int32_t r = 0; r < n_req; ++r) {
    const int32_t *c = matched + int64_t(r) * I;
    const int64_t L = prompt_len[r];
    bool ok = inst_ok && L >= 0 && L <= (int64_t(1) << 24);
    for (int32_t i = 0; ok && i < I; ++i) ok = c[i] >= 0 && c[i] <= L / B;
    if (!ok) {
      target[r] = -1;
      branch[r] = 255;
      continue;
    }
    // the weighted sum's terms as fractions over Dl and Dc
    const int64_t Dl = lmax > 0 ? lmax : 1;
    const int64_t Dc = L > 0 ? L : 1;
    auto lhat_num = [&](int32_t i) -> i128 { return lmax > 0 ? load[i] : 0; };
    auto miss_num = [&](int32_t i) -> i128 { return L > 0 ? L - B * c[i] : 1; };  // (1 - chat) Dc
    auto score = [&](int32_t k, int32_t i) -> i128 {
      switch (k) {
        case 0: return load[i];
        case 1: return i128(q[i]) + L - B * c[i];
        case 2: return (i128(q[i]) + L - B * c[i]) * load[i];
        default:  // (1 - lam) lhat + lam (1 - chat), times lam_den Dl Dc
          return i128(lam_den - lam_num) * lhat_num(i) * Dc + i128(lam_num) * miss_num(i) * Dl;
      }
    };
    const int32_t start = int32_t((rr_base % uint64_t(I) + uint64_t(r) % uint64_t(I)) % uint64_t(I));
    // argmin of score kind k over the instances with keep(i), rotation order on ties
    auto argmin = [&](int32_t k, auto keep) -> int32_t {
      int32_t best = -1;
      for (int32_t s = 0; s < I; ++s) {
        const int32_t i = (start + s) % I;
        if (!keep(i)) continue;
        if (best < 0 || score(k, i) < score(k, best)) best = i;  // strict: earlier position wins
      }
      return best;
    };
    auto all = [](int32_t) { return true; };
    if (kind == 4) {
      auto holds_half = [&](int32_t i) { return 2 * B * c[i] > L; };
      const int32_t h = argmin(0, holds_half);
      if (h >= 0) {
        target[r] = h;
        branch[r] = 7;
      } else {
        target[r] = argmin(3, all);
        branch[r] = 6;
      }
    } else {
      target[r] = argmin(kind, all);
      branch[r] = 6;
    }
  }
  return ORC_OK;
}

}  // extern "C"
