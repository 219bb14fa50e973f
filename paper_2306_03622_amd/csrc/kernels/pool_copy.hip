// Pooling (NHWC bf16), the host-to-device gather copy, the cache touch and the bounded delay
// kernel.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"
#include "touch.hpp"

namespace tp {
namespace k {
namespace {

// One thread per (sample, output pixel, 8 channels). The nine taps are loaded together (a tap
// in the padding reads the nearest pixel inside the image and is then ignored, so every load
// is in bounds and none waits for another) and reduced in the fixed order dh, dw; padded taps
// never win, as if skipped. (With each tap's load behind its bounds test the loads were issued
// one after another: 7.0 us per launch at ResNet-50 batch 1.)
__global__ __launch_bounds__(256) void k_maxpool3s2(const uint16_t* __restrict__ x, int B, int H, int W, int C,
                                                    int Ho, int Wo, uint16_t* __restrict__ y) {
  const int c8n = C >> 3;
  const long total = (long)B * Ho * Wo * c8n;
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int c8 = (int)(i % c8n);
  long p = i / c8n;
  const int ow = (int)(p % Wo);
  p /= Wo;
  const int oh = (int)(p % Ho);
  const int b = (int)(p / Ho);
  uint4 v[9];
  bool ok[9];
#pragma unroll
  for (int dh = 0; dh < 3; ++dh) {
    const int ih = oh * 2 - 1 + dh;
    const bool hin = ih >= 0 && ih < H;
    const int ihc = ih < 0 ? 0 : (ih >= H ? H - 1 : ih);
#pragma unroll
    for (int dw = 0; dw < 3; ++dw) {
      const int iw = ow * 2 - 1 + dw;
      const int iwc = iw < 0 ? 0 : (iw >= W ? W - 1 : iw);
      ok[dh * 3 + dw] = hin && iw >= 0 && iw < W;
      v[dh * 3 + dw] = *reinterpret_cast<const uint4*>(x + (((size_t)b * H + ihc) * W + iwc) * C + c8 * 8);
    }
  }
  float m[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) m[e] = -INFINITY;
#pragma unroll
  for (int t = 0; t < 9; ++t) {
    if (!ok[t]) continue;
    const uint32_t w[4] = {v[t].x, v[t].y, v[t].z, v[t].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      m[2 * e] = fmaxf(m[2 * e], bf2f(w[e] & 0xffff));
      m[2 * e + 1] = fmaxf(m[2 * e + 1], bf2f(w[e] >> 16));
    }
  }
  uint4 o;
  o.x = (uint32_t)f2bf(m[0]) | ((uint32_t)f2bf(m[1]) << 16);
  o.y = (uint32_t)f2bf(m[2]) | ((uint32_t)f2bf(m[3]) << 16);
  o.z = (uint32_t)f2bf(m[4]) | ((uint32_t)f2bf(m[5]) << 16);
  o.w = (uint32_t)f2bf(m[6]) | ((uint32_t)f2bf(m[7]) << 16);
  *reinterpret_cast<uint4*>(y + (((size_t)b * Ho + oh) * Wo + ow) * C + c8 * 8) = o;
}

// one thread per (sample, channel), positions summed in order in fp32
// One thread per (sample, channel). The HW loads are independent, so they are issued 8 at
// a time into 8 partial sums, which are then added in a fixed order.
__global__ __launch_bounds__(64) void k_avgpool(const uint16_t* __restrict__ x, int B, int HW, int C,
                                                uint16_t* __restrict__ y) {
  const int i = blockIdx.x * 64 + threadIdx.x;
  if (i >= B * C) return;
  const int b = i / C, c = i - b * C;
  const uint16_t* p = x + (size_t)b * HW * C + c;
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  int j = 0;
  for (; j + 8 <= HW; j += 8) {
    uint16_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = p[(size_t)(j + u) * C];
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u] += bf2f(v[u]);
  }
  for (; j < HW; ++j) s[0] += bf2f(p[(size_t)j * C]);
  float t = 0.f;
#pragma unroll
  for (int u = 0; u < 8; ++u) t += s[u];
  y[i] = f2bf(t / (float)HW);
}

// grid-stride copy with U independent 16-byte loads in flight per thread
__global__ __launch_bounds__(256) void k_gather(const uint4* __restrict__ src, uint4* __restrict__ dst, uint64_t n) {
  constexpr int U = 8;
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + (U - 1) * stride < n; i += U * stride) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < U; ++u) dst[i + u * stride] = v[u];
  }
  for (; i < n; i += stride) dst[i] = src[i];
}

// Loads in flight per thread, workgroups per touch (one per CU). Measured on MI355X, warm
// ResNet-50 / BERT-base requests at batch 1 after a cache flush, with every warm request
// touching: 397 / 534 us untouched; 376 / 528 with 32 workgroups, 373 / 508 with 64, 371 / 498
// with 128, 365 / 501 with 256, 377 / 515 with 2048 of 4 loads each. Back to back (the caches
// already warm) a touch costs BERT-base 8-12 us beside its own kernels (none for ResNet-50),
// so by default only a request that follows another model's touches.
constexpr int kTouchLoads = 8, kTouchWGs = 256;

// Reads n 16-byte vectors (grid-stride, U loads in flight per thread) with ordinary,
// cache-allocating loads and discards them: the bytes end up in the Infinity Cache (and the
// L2s), so that kernels reading them shortly after find them there. Nothing is stored unless
// the XOR of everything a thread read equals `magic`, which the caller makes impossible to
// rely on (the store only keeps the compiler from dropping the loads).
__global__ __launch_bounds__(256) void k_touch(const uint4* __restrict__ p, uint64_t n, uint32_t magic,
                                               uint32_t* __restrict__ sink) {
  constexpr int U = kTouchLoads;
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t x = 0;
  for (; i + (U - 1) * stride < n; i += U * stride) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = p[i + u * stride];
#pragma unroll
    for (int u = 0; u < U; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n; i += stride) {
    const uint4 v = p[i];
    x ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (x == magic) sink[blockIdx.x & 63] = x;
}

__global__ void k_delay(int iters) {
  for (int i = 0; i < iters; ++i) __builtin_amdgcn_s_sleep(127);
}

}  // namespace

hipError_t maxpool3s2(const uint16_t* x, int B, int H, int W, int C, uint16_t* y, hipStream_t s) {
  if (!x || !y || B < 1 || H < 1 || W < 1 || C < 8 || (C & 7)) return hipErrorInvalidValue;
  const int Ho = (H + 2 - 3) / 2 + 1, Wo = (W + 2 - 3) / 2 + 1;
  const long total = (long)B * Ho * Wo * (C >> 3);
  (void)launch(k_maxpool3s2, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, x, B, H, W, C, Ho, Wo, y);
  return hipGetLastError();
}

hipError_t avgpool(const uint16_t* x, int B, int HW, int C, uint16_t* y, hipStream_t s) {
  if (!x || !y || B < 1 || HW < 1 || C < 1) return hipErrorInvalidValue;
  (void)launch(k_avgpool, dim3((B * C + 63) / 64), dim3(64), 0, s, x, B, HW, C, y);
  return hipGetLastError();
}

hipError_t gather_copy(const void* src, void* dst, uint64_t bytes, int wgs, hipStream_t s) {
  if (!src || !dst || (bytes & 15) || wgs < 1 || ((uintptr_t)src & 15) || ((uintptr_t)dst & 15))
    return hipErrorInvalidValue;
  if (bytes == 0) return hipSuccess;
  (void)launch(k_gather, dim3(wgs), dim3(256), 0, s, static_cast<const uint4*>(src), static_cast<uint4*>(dst),
                     bytes >> 4);
  return hipGetLastError();
}

hipError_t touch(const void* p, uint64_t bytes, uint32_t* sink, hipStream_t s) {
  if (!p || !sink || (bytes & 15) || ((uintptr_t)p & 15)) return hipErrorInvalidValue;
  if (bytes == 0) return hipSuccess;
  const uint64_t n = bytes >> 4, per_wg = 256 * kTouchLoads;
  const unsigned wgs = (unsigned)std::min<uint64_t>(kTouchWGs, (n + per_wg - 1) / per_wg);
  (void)launch(k_touch, dim3(wgs), dim3(256), 0, s, static_cast<const uint4*>(p), n, 0x9e3779b9u, sink);
  return hipGetLastError();
}

hipError_t delay(int us, hipStream_t s) {
  // s_sleep 127 is about 127 * 64 cycles, ~3.4 us at 2.4 GHz
  const int iters = us <= 3 ? 1 : us / 3;
  (void)launch(k_delay, dim3(1), dim3(64), 0, s, iters);
  return hipGetLastError();
}

}  // namespace k
}  // namespace tp
