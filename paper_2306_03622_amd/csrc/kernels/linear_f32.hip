// fp32 linear layer y = act(x W^T + b) on the vector ALUs (no reduced-precision matrix
// path). One wave per output feature n: lanes stride over k in float4 steps, each lane
// accumulates its own partial sum in order, then a fixed butterfly reduction; rows of x
// are processed one after another by the same wave.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"
#include "swapin.hpp"

namespace tp {
namespace k {
namespace {

__global__ __launch_bounds__(256) void k_linear_f32(const float* __restrict__ x, int M, int K,
                                                    const float* __restrict__ w, int N,
                                                    const float* __restrict__ bias, int act,
                                                    float* __restrict__ y) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const float* wr = w + (size_t)n * K;
  for (int m = 0; m < M; ++m) {
    const float* xr = x + (size_t)m * K;
    float s = 0.f;
    for (int k = lane * 4; k < K; k += 256) {
      const float4 a = *reinterpret_cast<const float4*>(wr + k);
      const float4 b = *reinterpret_cast<const float4*>(xr + k);
      s = fmaf(a.x, b.x, s);
      s = fmaf(a.y, b.y, s);
      s = fmaf(a.z, b.z, s);
      s = fmaf(a.w, b.w, s);
    }
    s = wave_sum(s);
    if (lane == 0) y[(size_t)m * N + n] = act_apply(s + (bias ? bias[n] : 0.f), act);
  }
}

// The first layer of an fp32 model whose weights are still in pinned host memory, fused with
// the model's swap-in. Workgroups [0, cwg) compute y = act(x W^T + b) like k_linear_f32, one
// wave per output feature, reading W from the host copy once (a row is held in registers for
// every row of x, so the result is the same sequence of operations as k_linear_f32's) and
// writing what they read to the device copy; the other workgroups copy every 16-byte vector of
// the image outside W's own [skip0, skip1) host -> device, each thread issuing all its loads
// before its first store. All host reads of the model are thus in flight together.
constexpr int kSwapMaxM = 8, kSwapMaxKV = 4;     // rows of x; float4 per lane and row of W (K <= 1024)
constexpr int kSwapU = 4;                        // 16-byte vectors per gather thread and round

__global__ __launch_bounds__(256) void k_linear_f32_swap(const float* __restrict__ x, int M, int K,
                                                         const float* __restrict__ w_host, int N,
                                                         const float* __restrict__ bias_host, int act,
                                                         float* __restrict__ y, float* __restrict__ w_dev,
                                                         const uint4* __restrict__ img_host,
                                                         uint4* __restrict__ img_dev, uint64_t n16, uint64_t skip0,
                                                         uint64_t skip1, int cwg) {
  if ((int)blockIdx.x < cwg) {
    const int lane = threadIdx.x & 63;
    const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (n >= N) return;
    const float* wr = w_host + (size_t)n * K;
    float4 a[kSwapMaxKV];
#pragma unroll
    for (int i = 0; i < kSwapMaxKV; ++i) {
      const int k = lane * 4 + 256 * i;
      if (k < K) a[i] = *reinterpret_cast<const float4*>(wr + k);
    }
#pragma unroll
    for (int i = 0; i < kSwapMaxKV; ++i) {
      const int k = lane * 4 + 256 * i;
      if (k < K) *reinterpret_cast<float4*>(w_dev + (size_t)n * K + k) = a[i];
    }
    const float b = bias_host ? bias_host[n] : 0.f;
    for (int m = 0; m < M; ++m) {
      const float* xr = x + (size_t)m * K;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < kSwapMaxKV; ++i) {
        const int k = lane * 4 + 256 * i;
        if (k < K) {
          const float4 v = *reinterpret_cast<const float4*>(xr + k);
          s = fmaf(a[i].x, v.x, s);
          s = fmaf(a[i].y, v.y, s);
          s = fmaf(a[i].z, v.z, s);
          s = fmaf(a[i].w, v.w, s);
        }
      }
      s = wave_sum(s);
      if (lane == 0) y[(size_t)m * N + n] = act_apply(s + b, act);
    }
    return;
  }
  // gather: vectors [0, skip0) and [skip1, n16) as one index space of n16 - (skip1 - skip0)
  const uint64_t total = n16 - (skip1 - skip0);
  const uint64_t stride = (uint64_t)(gridDim.x - cwg) * 256;
  for (uint64_t i0 = (uint64_t)(blockIdx.x - cwg) * 256 + threadIdx.x; i0 < total; i0 += kSwapU * stride) {
    uint4 v[kSwapU];
#pragma unroll
    for (int u = 0; u < kSwapU; ++u) {
      const uint64_t i = i0 + u * stride;
      const uint64_t j = i < skip0 ? i : i + (skip1 - skip0);
      if (i < total) v[u] = img_host[j];
    }
#pragma unroll
    for (int u = 0; u < kSwapU; ++u) {
      const uint64_t i = i0 + u * stride;
      const uint64_t j = i < skip0 ? i : i + (skip1 - skip0);
      if (i < total) img_dev[j] = v[u];
    }
  }
}

}  // namespace

hipError_t linear_f32_swap(const float* x, int M, int K, int N, int act, float* y, const void* img_host,
                           void* img_dev, uint64_t img_bytes, uint64_t w_off, uint64_t b_off, hipStream_t s) {
  const uint64_t w_bytes = (uint64_t)N * K * 4;
  if (!x || !y || !img_host || !img_dev || M < 1 || M > kSwapMaxM || N < 1 || K < 4 || (K & 3) ||
      K > 256 * kSwapMaxKV || act < 0 || act > 2 || (img_bytes & 15) || (w_off & 15) ||
      w_off + w_bytes > img_bytes || b_off + (uint64_t)N * 4 > img_bytes || (b_off & 3) ||
      ((uintptr_t)img_host & 15) || ((uintptr_t)img_dev & 15))
    return hipErrorInvalidValue;
  const int cwg = (N + 3) / 4;
  const uint64_t n16 = img_bytes / 16, skip0 = w_off / 16, skip1 = (w_off + w_bytes + 15) / 16;
  const uint64_t rest = n16 - (skip1 - skip0);
  // every gather thread issues kSwapU loads per round: enough workgroups for one round
  const int gwg = (int)std::min<uint64_t>(1024, std::max<uint64_t>(1, (rest + 256 * kSwapU - 1) / (256 * kSwapU)));
  const char* h = static_cast<const char*>(img_host);
  char* d = static_cast<char*>(img_dev);
  (void)launch(k_linear_f32_swap, dim3(cwg + gwg), dim3(256), 0, s, x, M, K,
               reinterpret_cast<const float*>(h + w_off), N, reinterpret_cast<const float*>(h + b_off), act, y,
               reinterpret_cast<float*>(d + w_off), static_cast<const uint4*>(img_host), static_cast<uint4*>(img_dev),
               n16, skip0, skip1, cwg);
  return hipGetLastError();
}

hipError_t linear_f32(const float* x, int M, int K, const float* w, int N, const float* bias, int act, float* y,
                      hipStream_t s) {
  if (!x || !w || !y || M < 1 || N < 1 || K < 4 || (K & 3) || act < 0 || act > 2) return hipErrorInvalidValue;
  (void)launch(k_linear_f32, dim3((N + 3) / 4), dim3(256), 0, s, x, M, K, w, N, bias, act, y);
  return hipGetLastError();
}

}  // namespace k
}  // namespace tp
