// Load imbalance over time windows (the load-balance metric of the Sec. 4.1 analysis).
//
// Paper: an instance's load is its average number of running requests within a window,
// and the imbalance is the ratio of the maximum load to the mean over the instances.
// Here, exactly in integers: cell (w, i) = sum over requests on instance i of the overlap
// of their running interval [t0, t1) with window w = [w W, (w+1) W), i.e. the average
// running requests x W; per window the sum and the maximum over instances are returned
// (imbalance = max x I / sum).
//
// Mapping to gfx950: one thread per request adds its overlaps to the [window][instance]
// grid with 64-bit atomics (a request touches few windows); one workgroup per window then
// reduces its row.
#include "common.h"

namespace smk {
namespace {

constexpr int TB = 256;

__global__ void grid_clear_kernel(int64_t *g, uint64_t n, unsigned long long *n_bad) {
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  const uint64_t i0 = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  for (uint64_t i = i0; i < n; i += stride) g[i] = 0;
  if (i0 == 0) *n_bad = 0;
}

__global__ __launch_bounds__(TB) void overlap_kernel(const int32_t *__restrict__ inst, const int64_t *__restrict__ t0,
                                                     const int64_t *__restrict__ t1, int64_t n_req, int32_t I,
                                                     int64_t window, int32_t n_windows, int64_t *g,
                                                     unsigned long long *n_bad) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t r = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; r < n_req; r += stride) {
    const int32_t i = inst[r];
    const int64_t a = t0[r], b = t1[r];
    if (i < 0 || i >= I || b < a) {
      atomicAdd(n_bad, 1ull);
      continue;
    }
    if (b <= 0 || n_windows == 0) continue;
    const int64_t end = int64_t(n_windows) * window;
    if (a >= end) continue;
    const int64_t w0 = a > 0 ? a / window : 0;
    const int64_t w1 = ((b < end ? b : end) - 1) / window;  // last window touched
    for (int64_t w = w0; w <= w1; ++w) {
      const int64_t lo = a > w * window ? a : w * window;
      const int64_t hi = b < (w + 1) * window ? b : (w + 1) * window;
      if (hi > lo)
        atomicAdd(reinterpret_cast<unsigned long long *>(&g[w * I + i]), (unsigned long long)(hi - lo));
    }
  }
}

__global__ __launch_bounds__(TB) void window_reduce_kernel(const int64_t *__restrict__ g, int32_t I,
                                                           int64_t *__restrict__ out_sum, int64_t *__restrict__ out_max) {
  __shared__ int64_t ps[TB / 64], pm[TB / 64];
  const int32_t w = blockIdx.x;
  int64_t s = 0, m = 0;
  for (int32_t i = threadIdx.x; i < I; i += TB) {
    const int64_t v = g[int64_t(w) * I + i];
    s += v;
    m = v > m ? v : m;
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    s += __shfl_xor(s, d, 64);
    const int64_t o = __shfl_xor(m, d, 64);
    m = o > m ? o : m;
  }
  if ((threadIdx.x & 63) == 0) {
    ps[threadIdx.x >> 6] = s;
    pm[threadIdx.x >> 6] = m;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t ts = 0, tm = 0;
    for (int k = 0; k < TB / 64; ++k) {
      ts += ps[k];
      tm = pm[k] > tm ? pm[k] : tm;
    }
    out_sum[w] = ts;
    out_max[w] = tm;
  }
}

}  // namespace
}  // namespace smk

using namespace smk;

extern "C" int smetric_imbalance_ws_bytes(int32_t n_instances, int32_t n_windows, uint64_t *ws_bytes) {
  if (n_instances < 1 || n_windows < 0 || !ws_bytes) return SMETRIC_EINVAL;
  *ws_bytes = (uint64_t(n_windows) * uint64_t(n_instances) * 8 + 256 + 255) / 256 * 256;
  return SMETRIC_OK;
}

extern "C" int smetric_imbalance(const int32_t *inst, const int64_t *t0, const int64_t *t1, int64_t n_req,
                                 int32_t n_instances, int64_t window, int32_t n_windows, int64_t *out_sum,
                                 int64_t *out_max, int64_t *n_bad, void *workspace, uint64_t ws_bytes,
                                 hipStream_t stream) {
  if (n_req < 0 || n_instances < 1 || window <= 0 || n_windows < 0 || !n_bad) return SMETRIC_EINVAL;
  if (n_req > 0 && (!inst || !t0 || !t1)) return SMETRIC_EINVAL;
  if (n_windows > 0 && (!out_sum || !out_max)) return SMETRIC_EINVAL;
  if (window > (int64_t(1) << 62) / (int64_t(n_windows) + 1)) return SMETRIC_EINVAL;  // window ends stay in range
  uint64_t need = 0;
  smetric_imbalance_ws_bytes(n_instances, n_windows, &need);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) || ws_bytes < need) return SMETRIC_EWORKSPACE;
  int64_t *g = static_cast<int64_t *>(workspace);
  const uint64_t cells = uint64_t(n_windows) * uint64_t(n_instances);
  auto *bad = reinterpret_cast<unsigned long long *>(n_bad);
  const uint64_t cg = (cells + TB - 1) / TB;
  hipLaunchKernelGGL(grid_clear_kernel, dim3(int(cg < 1 ? 1 : (cg > 4096 ? 4096 : cg))), dim3(TB), 0, stream, g, cells,
                     bad);
  if (n_req > 0) {
    const int64_t rg = (n_req + TB - 1) / TB;
    hipLaunchKernelGGL(overlap_kernel, dim3(int(rg > 8192 ? 8192 : rg)), dim3(TB), 0, stream, inst, t0, t1, n_req,
                       n_instances, window, n_windows, g, bad);
  }
  if (n_windows > 0)
    hipLaunchKernelGGL(window_reduce_kernel, dim3(n_windows), dim3(TB), 0, stream, g, n_instances, out_sum, out_max);
  return hip_rc(hipGetLastError());
}
