// Row LayerNorm and the fused embedding gather + LayerNorm. One wave per row, each lane
// holding D/64 elements in registers; mean and variance (two passes over the registers,
// population variance) use butterfly wave reductions in fp32.
#include "common.hpp"
#include "kernels.hpp"

namespace tp {
namespace k {
namespace {

constexpr int kMaxPer = 16;   // D <= 1024

__device__ __forceinline__ void normalize(float (&v)[kMaxPer], int per, int D, const uint16_t* g,
                                          const uint16_t* b, float eps, int lane, void* out, size_t row_off,
                                          int out_f32) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i)
    if (i < per) s += v[i];
  const float mean = wave_sum(s) / (float)D;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    if (i < per) {
      const float d = v[i] - mean;
      q = fmaf(d, d, q);
    }
  }
  const float var = wave_sum(q) / (float)D;
  const float rstd = 1.f / sqrtf(var + eps);
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    if (i >= per) break;
    const int c = lane + 64 * i;
    const float y = (v[i] - mean) * rstd * bf2f(g[c]) + bf2f(b[c]);
    if (out_f32) static_cast<float*>(out)[row_off + c] = y;
    else static_cast<uint16_t*>(out)[row_off + c] = f2bf(y);
  }
}

__global__ __launch_bounds__(256) void k_layernorm(const float* __restrict__ x, int M, int D,
                                                   const uint16_t* __restrict__ g, const uint16_t* __restrict__ b,
                                                   float eps, void* out, int out_f32) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int per = D >> 6;
  float v[kMaxPer];
  const float* xr = x + (size_t)row * D;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) v[i] = i < per ? xr[lane + 64 * i] : 0.f;
  normalize(v, per, D, g, b, eps, lane, out, (size_t)row * D, out_f32);
}

__global__ __launch_bounds__(256) void k_embed_ln(const int32_t* __restrict__ ids, int M, int S, int D, int vocab,
                                                  const uint16_t* __restrict__ tok, const uint16_t* __restrict__ pos,
                                                  const uint16_t* __restrict__ type, const uint16_t* __restrict__ g,
                                                  const uint16_t* __restrict__ b, float eps, uint16_t* out) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  int id = ids[row];
  id = id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
  const int s = row % S;
  const int per = D >> 6;
  float v[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int c = lane + 64 * i;
    v[i] = i < per ? bf2f(tok[(size_t)id * D + c]) + bf2f(pos[(size_t)s * D + c]) + bf2f(type[c]) : 0.f;
  }
  normalize(v, per, D, g, b, eps, lane, out, (size_t)row * D, 0);
}

}  // namespace

hipError_t layernorm(const float* x, int M, int D, const uint16_t* g, const uint16_t* b, float eps, void* out,
                     int out_f32, hipStream_t s) {
  if (!x || !g || !b || !out || M < 1 || D < 64 || (D & 63) || D > 64 * kMaxPer) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_layernorm, dim3((M + 3) / 4), dim3(256), 0, s, x, M, D, g, b, eps, out, out_f32);
  return hipGetLastError();
}

hipError_t embed_ln(const int32_t* ids, int M, int S, int D, int vocab, const uint16_t* tok, const uint16_t* pos,
                    const uint16_t* type, const uint16_t* g, const uint16_t* b, float eps, uint16_t* out,
                    hipStream_t s) {
  if (!ids || !tok || !pos || !type || !g || !b || !out || M < 1 || S < 1 || vocab < 1 || D < 64 || (D & 63) ||
      D > 64 * kMaxPer)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_embed_ln, dim3((M + 3) / 4), dim3(256), 0, s, ids, M, S, D, vocab, tok, pos, type, g, b, eps,
                     out);
  return hipGetLastError();
}

}  // namespace k
}  // namespace tp
