// Region-ordered probe of every block of a batch (K3, shared by match and insert).
//
// Paper: c_i is the prefix hit of the prompt in instance i's local KV$ (Sec. 4.1); after
// routing, the target caches every block (Sec. 2, 4.2).  Both steps ask the index the
// same question per block -- which instances hold this key -- so it is asked once.
//
// Mapping to gfx950.  Probes are random 128-byte reads over a table of several GB.  On
// MI355X such reads run ~5x faster when the workgroups in flight stay inside a window of
// a GB or less than when they roam the whole table (the translation caches keep up), so
// the batch's blocks are first partitioned by table region (NREG equal bucket ranges),
// with no global atomics:
//   requests  one wavefront per request checks the tiling and records each block's request
//   count     PART_WG workgroups, one contiguous chunk of blocks each: LDS histogram of
//             regions -> one column of the [region][chunk] matrix
//   scan      per region, running offsets over chunks -> first position of every
//             (region, chunk) pair
//   scatter   each chunk again: LDS ranks per region -> (key, block | request << 32) at
//             its region-order position, and the inverse index block -> position
//   probe     a fixed grid of FLAT_WG workgroups walks the region-ordered keys; all
//             workgroups advance through the regions together, so the live window slides
//             through the table.  One 128-byte bucket read per chain step (keys and values
//             at once) gives a 64-bit holder descriptor, written in region order.
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
}

__global__ __launch_bounds__(TB) void part_count_kernel(DevIndex ix, ProbeView pv, const uint64_t *__restrict__ keys,
                                                        uint64_t n) {
  __shared__ unsigned int h[NREG];
  for (int g = threadIdx.x; g < NREG; g += TB) h[g] = 0;
  __syncthreads();
  uint64_t lo, hi;
  chunk_of(n, lo, hi);
  for (uint64_t b = lo + threadIdx.x; b < hi; b += TB) atomicAdd(&h[region_of(keys[b], ix.n_buckets)], 1u);
  __syncthreads();
  for (int g = threadIdx.x; g < NREG; g += TB) pv.hist[uint64_t(g) * PART_WG + blockIdx.x] = h[g];
}

// one thread per region: region totals, their exclusive scan, then per-chunk offsets
__global__ __launch_bounds__(NREG) void part_scan_kernel(ProbeView pv, uint64_t n) {
  __shared__ unsigned long long tot[NREG];
  const int g = threadIdx.x;
  const uint32_t *row = pv.hist + uint64_t(g) * PART_WG;
  unsigned long long t = 0;
  for (int w = 0; w < PART_WG; ++w) t += row[w];
  tot[g] = t;
  __syncthreads();
  if (g == 0) {
    unsigned long long acc = 0;
    for (int i = 0; i < NREG; ++i) {
      const unsigned long long c = tot[i];
      tot[i] = acc;
      acc += c;
    }
    pv.hdr->n = pv.hdr->err ? 0 : acc;
  }
  __syncthreads();
  unsigned long long acc = tot[g];
  uint64_t *out = pv.base + uint64_t(g) * PART_WG;
  for (int w = 0; w < PART_WG; ++w) {
    out[w] = acc;
    acc += row[w];
  }
}

__global__ __launch_bounds__(TB) void part_scatter_kernel(DevIndex ix, ProbeView pv, const uint64_t *__restrict__ keys,
                                                          uint64_t n) {
  __shared__ unsigned long long base[NREG];
  __shared__ unsigned int rank[NREG];
  if (pv.hdr->err) return;
  for (int g = threadIdx.x; g < NREG; g += TB) {
    base[g] = pv.base[uint64_t(g) * PART_WG + blockIdx.x];
    rank[g] = 0;
  }
  __syncthreads();
  uint64_t lo, hi;
  chunk_of(n, lo, hi);
  for (uint64_t b = lo + threadIdx.x; b < hi; b += TB) {
    const uint64_t key = keys[b];
    const uint32_t g = region_of(key, ix.n_buckets);
    const uint64_t pos = base[g] + atomicAdd(&rank[g], 1u);
    pv.part_key[pos] = key;
    pv.part_br[pos] = b | (uint64_t(pv.req_of[b]) << 32);
    pv.inv[b] = uint32_t(pos);
  }
}

// Holder descriptor of `key`: one chain walk, each step one 128-byte bucket read.
__device__ uint64_t describe(const DevIndex &ix, uint64_t key) {
  uint64_t b = home_bucket(key, ix.n_buckets);
  uint32_t cnt = 0, first_inst = 0;
  uint64_t first_slot = 0;
  for (uint64_t step = 0; step < ix.n_buckets; ++step, b = next_bucket(b, ix.n_buckets)) {
    const ulonglong2 *p = reinterpret_cast<const ulonglong2 *>(ix.slots + b * BUCKET_WORDS);
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
      if (!end && k == key) {
        const uint32_t kind = val_kind(v);
        if (kind == HEADER) return make_desc(D_HOT, 0, val_rec(v));
        if (kind == PLAIN) {
          if (cnt == 0) {
            first_inst = val_inst(v);
            first_slot = b * SLOTS + s;
          }
          ++cnt;
        }
      }
    }
    if (end) break;
  }
  if (cnt == 0) return make_desc(D_NONE, 0, 0);
  if (cnt == 1) return make_desc(D_ONE, first_inst, first_slot);
  return make_desc(D_MANY, 0, 0);
}

__global__ __launch_bounds__(TB) void probe_kernel(DevIndex ix, ProbeView pv) {
  const uint64_t n = pv.hdr->n;
  const uint64_t span = uint64_t(gridDim.x) * TB;
  for (uint64_t i = uint64_t(blockIdx.x) * TB + threadIdx.x; i < n; i += span)
    pv.desc_p[i] = describe(ix, pv.part_key[i]);
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_probe_ws_bytes(int64_t n_blocks, uint64_t *bytes) {
  if (n_blocks < 0 || n_blocks >= (int64_t(1) << 32) || !bytes) return SMETRIC_EINVAL;
  *bytes = probe_layout(n_blocks, nullptr, nullptr);
  return SMETRIC_OK;
}

extern "C" int smetric_probe(const smetric_index *idx, const uint64_t *keys, const int64_t *blk_off, int32_t n_req,
                             int64_t n_blocks, void *probe, uint64_t probe_bytes, hipStream_t stream) {
  if (!idx || !idx->slots || n_req < 0 || n_blocks < 0 || n_blocks >= (int64_t(1) << 32)) return SMETRIC_EINVAL;
  if (!blk_off || (n_blocks > 0 && !keys) || (n_req == 0 && n_blocks != 0)) return SMETRIC_EINVAL;
  if (!probe || (reinterpret_cast<uintptr_t>(probe) & 255) || probe_bytes < probe_layout(n_blocks, nullptr, nullptr))
    return SMETRIC_EWORKSPACE;
  ProbeView pv;
  probe_layout(n_blocks, &pv, probe);
  const DevIndex ix = dev_view(idx);
  const uint64_t n = uint64_t(n_blocks);
  hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(64), 0, stream, reinterpret_cast<uint64_t *>(pv.hdr),
                     uint64_t(sizeof(ProbeHdr) / 8));
  if (n_req > 0)
    hipLaunchKernelGGL(req_of_kernel, dim3(n_req), dim3(64), 0, stream, pv, blk_off, n_req, n_blocks);
  hipLaunchKernelGGL(part_count_kernel, dim3(PART_WG), dim3(TB), 0, stream, ix, pv, keys, n);
  hipLaunchKernelGGL(part_scan_kernel, dim3(1), dim3(NREG), 0, stream, pv, n);
  hipLaunchKernelGGL(part_scatter_kernel, dim3(PART_WG), dim3(TB), 0, stream, ix, pv, keys, n);
  hipLaunchKernelGGL(probe_kernel, dim3(FLAT_WG), dim3(TB), 0, stream, ix, pv);
  return hip_rc(hipGetLastError());
}
