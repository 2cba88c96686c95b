// Drafting metrics from per-verification accepted lengths (Sec. 3.1, Metrics):
// counts c_k = #{a_i >= k}, conditional step-wise acceptance rates, MAT and
// the retention ratio, for a batch of verification records that already sits
// in device memory (no copy back, no host synchronisation).
//
// Three launches on the caller's stream: a fill of the K + 1 bins (a kernel,
// so the call can be captured in a graph); a grid-stride histogram -- for up
// to 15 steps over an aligned buffer in packed per-lane registers, otherwise
// in per-workgroup LDS bins -- merged with 64-bit integer
// atomics, so the counts are exact in any order; and a one-wave finish that
// forms c_k, alpha_k, MAT and the retention in float64.
#include "kvshot_metrics.h"

#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kMaxSteps = 255;

__global__ void zero_bins(unsigned long long* bins, int nb) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nb) bins[i] = 0ull;
}

__global__ __launch_bounds__(256) void histogram_kernel(const int32_t* __restrict__ accepted, int64_t n, int K,
                                                        unsigned long long* bins) {
  __shared__ unsigned int local[kMaxSteps + 1];
  for (int i = threadIdx.x; i <= K; i += 256) local[i] = 0u;
  __syncthreads();
  auto add = [&](int32_t a) { atomicAdd(&local[a < 0 ? 0 : (a > K ? K : a)], 1u); };
  const int64_t stride = (int64_t)gridDim.x * 256 * 4;
  const int64_t n4 = n & ~(int64_t)3;
  // four records per thread and step (16-byte loads where the buffer allows)
  const bool vec = ((uintptr_t)accepted & 15u) == 0;
  for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4; i < n4; i += stride) {
    if (vec) {
      const int4 v = *(const int4*)(accepted + i);
      add(v.x);
      add(v.y);
      add(v.z);
      add(v.w);
    } else {
      add(accepted[i]);
      add(accepted[i + 1]);
      add(accepted[i + 2]);
      add(accepted[i + 3]);
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < (int)(n - n4)) add(accepted[n4 + threadIdx.x]);
  __syncthreads();
  for (int i = threadIdx.x; i <= K; i += 256)
    if (local[i]) atomicAdd(&bins[i], (unsigned long long)local[i]);
}

// K <= 15 and a 16-byte aligned buffer: the histogram in registers.  A lane
// counts its records in two 64-bit words of eight 8-bit fields (bin b is
// field b % 8 of word b / 8): one shifted 1 added per record.  After every 16
// records (no field can overflow) the fields are added into 32-bit counters.
// The workgroup then sums its lanes' counters in LDS and merges them with one
// atomic per bin.
constexpr int kPackedBins = 16;

__global__ __launch_bounds__(256) void packed_histogram_kernel(const int32_t* __restrict__ accepted, int64_t n, int K,
                                                               unsigned long long* bins) {
  __shared__ unsigned int part[kPackedBins][257];
  uint32_t cnt[kPackedBins];
#pragma unroll
  for (int b = 0; b < kPackedBins; ++b) cnt[b] = 0u;
  uint64_t w0 = 0, w1 = 0;
  auto add = [&](int32_t a) {
    a = a < 0 ? 0 : (a > K ? K : a);
    const uint64_t inc = 1ull << (8 * (a & 7));
    w0 += a < 8 ? inc : 0ull;
    w1 += a < 8 ? 0ull : inc;
  };
  auto flush = [&]() {
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      cnt[b] += (uint32_t)(w0 >> (8 * b)) & 0xffu;
      cnt[b + 8] += (uint32_t)(w1 >> (8 * b)) & 0xffu;
    }
    w0 = w1 = 0;
  };
  constexpr int kUnroll = 4;                      // 16-byte loads in flight per lane: 16 records between flushes
  const int64_t n4 = n & ~(int64_t)3;
  const int64_t stride = (int64_t)gridDim.x * 256 * 4 * kUnroll;
  for (int64_t i0 = ((int64_t)blockIdx.x * 256 * kUnroll) * 4 + threadIdx.x * 4; i0 < n4; i0 += stride) {
    int4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = i0 + (int64_t)u * 256 * 4;
      v[u] = i < n4 ? *(const int4*)(accepted + i) : make_int4(-1, -1, -1, -1);
    }
    // records past the end were read as -1 and land in bin 0: take them back out below
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      add(v[u].x);
      add(v[u].y);
      add(v[u].z);
      add(v[u].w);
    }
    flush();
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (i0 + (int64_t)u * 256 * 4 >= n4) cnt[0] -= 4u;
  }
  if (blockIdx.x == 0 && threadIdx.x < (int)(n - n4)) {
    add(accepted[n4 + threadIdx.x]);
    flush();
  }
#pragma unroll
  for (int b = 0; b < kPackedBins; ++b) part[b][threadIdx.x] = cnt[b];
  __syncthreads();
  if (threadIdx.x <= K) {
    unsigned long long t = 0ull;
    for (int i = 0; i < 256; ++i) t += part[threadIdx.x][i];
    if (t) atomicAdd(&bins[threadIdx.x], t);
  }
}

// One wave: lane k (k <= K) holds histogram bin k; the suffix sums give c_k.
// The rates and MAT are formed sequentially by lane 0, in the printed order.
__global__ __launch_bounds__(64) void finish_kernel(int K, unsigned long long* bins, double* alpha, double* mat,
                                                    double* retention, int rstep) {
  __shared__ unsigned long long c[kMaxSteps + 2];
  const int lane = threadIdx.x;
  for (int i = lane; i <= K; i += 64) c[i] = bins[i];
  __syncthreads();
  if (lane == 0) {
    unsigned long long run = 0ull;
    for (int k = K; k >= 0; --k) {
      run += c[k];
      c[k] = run;               // c_k = #{a >= k}
    }
    double total = 1.0, prod = 1.0;
    double a0 = 0.0, ar = 0.0;
    for (int k = 0; k < K; ++k) {
      const double a = c[k] ? (double)c[k + 1] / (double)c[k] : 0.0;
      alpha[k] = a;
      prod *= a;
      total += prod;
      if (k == 0) a0 = a;
      if (k == rstep) ar = a;
    }
    *mat = total;
    if (retention) *retention = a0 > 0.0 ? ar / a0 : 0.0;
  }
  __syncthreads();
  for (int i = lane; i <= K; i += 64) bins[i] = c[i];
}

}  // namespace

extern "C" kvshot_status kvshot_acceptance_stats(const int32_t* accepted, int64_t n, int32_t K, int64_t* counts,
                                                 double* alpha, double* mat, double* retention, int32_t retention_step,
                                                 void* stream) {
  if (n < 0 || K < 1 || K > kMaxSteps) return KVSHOT_ERR_INVALID_ARG;
  if ((n > 0 && !accepted) || !counts || !alpha || !mat) return KVSHOT_ERR_INVALID_ARG;
  if (retention && (retention_step < 0 || retention_step >= K)) return KVSHOT_ERR_INVALID_ARG;
  if (((uintptr_t)accepted & 3u) || ((uintptr_t)counts & 7u) || ((uintptr_t)alpha & 7u) || ((uintptr_t)mat & 7u) ||
      ((uintptr_t)retention & 7u))
    return KVSHOT_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  unsigned long long* bins = (unsigned long long*)counts;
  hipLaunchKernelGGL(zero_bins, dim3((K + 1 + 255) / 256), dim3(256), 0, s, bins, K + 1);
  const bool packed = K < kPackedBins && ((uintptr_t)accepted & 15u) == 0;
  if (n > 0) {
    // few workgroups, each covering many records: the merge is one atomic per bin and workgroup
    int64_t wgs = (n + 4095) / 4096;
    if (wgs > 512) wgs = 512;
    if (packed)
      hipLaunchKernelGGL(packed_histogram_kernel, dim3((unsigned)wgs), dim3(256), 0, s, accepted, n, (int)K, bins);
    else
      hipLaunchKernelGGL(histogram_kernel, dim3((unsigned)wgs), dim3(256), 0, s, accepted, n, (int)K, bins);
  }
  hipLaunchKernelGGL(finish_kernel, dim3(1), dim3(64), 0, s, (int)K, bins, alpha, mat, retention,
                     (int)retention_step);
  return hipGetLastError() == hipSuccess ? KVSHOT_OK : KVSHOT_ERR_DEVICE;
}
