// Peak probes (torpor_probe.h): matrix-core throughput, streaming HBM read and kernel-driven
// host-to-device reads on gfx950. Each kernel has a fixed amount of work and bounds-checked
// indexing; results are written so that the compiler cannot drop the work.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "torpor_probe.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;   // independent accumulators per wave: covers the MFMA latency

__global__ __launch_bounds__(256) void k_mfma(int iters, float* out, unsigned long long* clk) {
  const int tid = threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(float)((tid + e) & 7);
    b[e] = (__bf16)(float)((tid * 3 + e) & 7);
  }
  f32x4 acc[kChains];
#pragma unroll
  for (int j = 0; j < kChains; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bool first = blockIdx.x == 0 && tid == 0;
  unsigned long long c0 = 0, r0 = 0;
  if (first) {
    c0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  for (int i = 0; i < iters; ++i)
#pragma unroll
    for (int j = 0; j < kChains; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kChains; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  out[(size_t)blockIdx.x * 256 + tid] = s;
  if (first) {
    clk[0] = __builtin_amdgcn_s_memtime() - c0;
    clk[1] = __builtin_amdgcn_s_memrealtime() - r0;
  }
}

__global__ __launch_bounds__(256) void k_read(const uint4* __restrict__ p, uint64_t n16, uint32_t* out) {
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t x = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p + i + u * stride));
#pragma unroll
    for (int u = 0; u < 4; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p + i));
    x ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = x;
}

__global__ __launch_bounds__(256) void k_gather(const uint4* __restrict__ src, uint4* __restrict__ dst, uint64_t n16) {
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    uint4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u) dst[i + u * stride] = v[u];
  }
  for (; i < n16; i += stride) dst[i] = src[i];
}

struct Events {
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t init() {
    hipError_t e = hipEventCreate(&a);
    return e == hipSuccess ? hipEventCreate(&b) : e;
  }
  ~Events() {
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
  }
};

#define TPP_TRY(x)                     \
  do {                                 \
    hipError_t e_ = (x);               \
    if (e_ != hipSuccess) return e_;   \
  } while (0)

// best time in ms of `reps` launches of `launch`
template <class F>
hipError_t best_ms(int reps, F launch, float* best) {
  Events ev;
  TPP_TRY(ev.init());
  *best = 1e30f;
  for (int r = 0; r < std::max(reps, 1); ++r) {
    TPP_TRY(hipEventRecord(ev.a, nullptr));
    launch();
    TPP_TRY(hipGetLastError());
    TPP_TRY(hipEventRecord(ev.b, nullptr));
    TPP_TRY(hipEventSynchronize(ev.b));
    float ms = 0.f;
    TPP_TRY(hipEventElapsedTime(&ms, ev.a, ev.b));
    *best = std::min(*best, ms);
  }
  return hipSuccess;
}

}  // namespace

extern "C" int tpp_mfma_bf16(int wgs, int iters, int reps, double* tflops, double* clock_ghz) {
  if (wgs < 1 || iters < 1 || !tflops || !clock_ghz) return hipErrorInvalidValue;
  float* out = nullptr;
  unsigned long long* clk = nullptr;
  hipError_t e = hipMalloc(&out, (size_t)wgs * 256 * sizeof(float));
  if (e == hipSuccess) e = hipMalloc(&clk, 2 * sizeof(unsigned long long));
  float ms = 0.f;
  if (e == hipSuccess) e = best_ms(reps, [&] { hipLaunchKernelGGL(k_mfma, dim3(wgs), dim3(256), 0, nullptr, iters, out, clk); }, &ms);
  unsigned long long h[2] = {0, 0};
  if (e == hipSuccess) e = hipMemcpy(h, clk, sizeof(h), hipMemcpyDeviceToHost);
  if (out) (void)hipFree(out);
  if (clk) (void)hipFree(clk);
  if (e != hipSuccess) return e;
  const double flops = (double)wgs * 4 * iters * kChains * 16384.0;
  *tflops = flops / (ms * 1e-3) / 1e12;
  *clock_ghz = h[1] ? (double)h[0] / ((double)h[1] / 100e6) / 1e9 : 0.0;
  return hipSuccess;
}

extern "C" int tpp_hbm_read(uint64_t bytes, int wgs, int reps, double* gbs) {
  if (!bytes || bytes % 16 || wgs < 1 || !gbs) return hipErrorInvalidValue;
  void* buf = nullptr;
  uint32_t* out = nullptr;
  hipError_t e = hipMalloc(&buf, bytes);
  if (e == hipSuccess) e = hipMalloc(&out, (size_t)wgs * 256 * sizeof(uint32_t));
  if (e == hipSuccess) e = hipMemset(buf, 0x5a, bytes);
  float ms = 0.f;
  if (e == hipSuccess)
    e = best_ms(reps, [&] {
      hipLaunchKernelGGL(k_read, dim3(wgs), dim3(256), 0, nullptr, static_cast<const uint4*>(buf), bytes / 16, out);
    }, &ms);
  if (buf) (void)hipFree(buf);
  if (out) (void)hipFree(out);
  if (e != hipSuccess) return e;
  *gbs = (double)bytes / (ms * 1e-3) / 1e9;
  return hipSuccess;
}

extern "C" int tpp_gather_h2d(uint64_t bytes, int wgs, int reps, double* gbs) {
  if (!bytes || bytes % 16 || wgs < 1 || !gbs) return hipErrorInvalidValue;
  void* host = nullptr;
  void* host_dev = nullptr;
  void* dev = nullptr;
  hipError_t e = hipHostMalloc(&host, bytes, hipHostMallocMapped);
  if (e == hipSuccess) e = hipHostGetDevicePointer(&host_dev, host, 0);
  if (e == hipSuccess) e = hipMalloc(&dev, bytes);
  if (e == hipSuccess) e = hipMemset(dev, 0, bytes);
  float ms = 0.f;
  if (e == hipSuccess)
    e = best_ms(reps, [&] {
      hipLaunchKernelGGL(k_gather, dim3(wgs), dim3(256), 0, nullptr, static_cast<const uint4*>(host_dev),
                         static_cast<uint4*>(dev), bytes / 16);
    }, &ms);
  if (dev) (void)hipFree(dev);
  if (host) (void)hipHostFree(host);
  if (e != hipSuccess) return e;
  *gbs = (double)bytes / (ms * 1e-3) / 1e9;
  return hipSuccess;
}
