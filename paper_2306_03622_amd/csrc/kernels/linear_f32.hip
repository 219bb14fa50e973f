// fp32 linear layer y = act(x W^T + b) on the vector ALUs (no reduced-precision matrix
// path). One wave per output feature n: lanes stride over k in float4 steps, each lane
// accumulates its own partial sum in order, then a fixed butterfly reduction; rows of x
// are processed one after another by the same wave.
#include "common.hpp"
#include "kernels.hpp"

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

}  // namespace

hipError_t linear_f32(const float* x, int M, int K, const float* w, int N, const float* bias, int act, float* y,
                      hipStream_t s) {
  if (!x || !w || !y || M < 1 || N < 1 || K < 4 || (K & 3) || act < 0 || act > 2) return hipErrorInvalidValue;
  (void)launch(k_linear_f32, dim3((N + 3) / 4), dim3(256), 0, s, x, M, K, w, N, bias, act, y);
  return hipGetLastError();
}

}  // namespace k
}  // namespace tp
