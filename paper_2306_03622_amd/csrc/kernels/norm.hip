// Row LayerNorm and the fused embedding gather + LayerNorm. One wave per row, each lane
// holding D/64 elements in registers; mean and variance (two passes over the registers,
// population variance) use butterfly wave reductions in fp32.
#include "common.hpp"
#include "kernels.hpp"

namespace tp {
namespace k {
namespace {

constexpr int kMaxPer = 16;   // D <= 1024

// Mean, population variance and affine map of one row held as PER values per lane
// (element c = lane + 64 i); the row is written as bf16 or fp32.
template <int PER>
__device__ __forceinline__ void normalize(float (&v)[PER], int D, const uint16_t* g, const uint16_t* b, float eps,
                                          int lane, void* out, size_t row_off, int out_f32) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) s += v[i];
  const float mean = wave_sum(s) / (float)D;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const float d = v[i] - mean;
    q = fmaf(d, d, q);
  }
  const float var = wave_sum(q) / (float)D;
  const float rstd = 1.f / sqrtf(var + eps);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int c = lane + 64 * i;
    const float y = (v[i] - mean) * rstd * bf2f(g[c]) + bf2f(b[c]);
    if (out_f32) static_cast<float*>(out)[row_off + c] = y;
    else static_cast<uint16_t*>(out)[row_off + c] = f2bf(y);
  }
}

template <int PER>
__global__ __launch_bounds__(256) void k_layernorm(const float* __restrict__ x, int M,
                                                   const uint16_t* __restrict__ g, const uint16_t* __restrict__ b,
                                                   float eps, void* out, int out_f32) {
  constexpr int D = 64 * PER;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  float v[PER];
  const float* xr = x + (size_t)row * D;
#pragma unroll
  for (int i = 0; i < PER; ++i) v[i] = xr[lane + 64 * i];
  normalize<PER>(v, D, g, b, eps, lane, out, (size_t)row * D, out_f32);
}

template <int PER>
__global__ __launch_bounds__(256) void k_embed_ln(const int32_t* __restrict__ ids, int M, int S, int vocab,
                                                  const uint16_t* __restrict__ tok, const uint16_t* __restrict__ pos,
                                                  const uint16_t* __restrict__ type, const uint16_t* __restrict__ g,
                                                  const uint16_t* __restrict__ b, float eps, uint16_t* out) {
  constexpr int D = 64 * PER;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  int id = ids[row];
  id = id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
  const int s = row % S;
  float v[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int c = lane + 64 * i;
    v[i] = bf2f(tok[(size_t)id * D + c]) + bf2f(pos[(size_t)s * D + c]) + bf2f(type[c]);
  }
  normalize<PER>(v, D, g, b, eps, lane, out, (size_t)row * D, 0);
}

template <int PER>
hipError_t launch_ln(const float* x, int M, const uint16_t* g, const uint16_t* b, float eps, void* out, int out_f32,
                     hipStream_t s) {
  hipLaunchKernelGGL((k_layernorm<PER>), dim3((M + 3) / 4), dim3(256), 0, s, x, M, g, b, eps, out, out_f32);
  return hipGetLastError();
}

template <int PER>
hipError_t launch_embed(const int32_t* ids, int M, int S, int vocab, const uint16_t* tok, const uint16_t* pos,
                        const uint16_t* type, const uint16_t* g, const uint16_t* b, float eps, uint16_t* out,
                        hipStream_t s) {
  hipLaunchKernelGGL((k_embed_ln<PER>), dim3((M + 3) / 4), dim3(256), 0, s, ids, M, S, vocab, tok, pos, type, g, b,
                     eps, out);
  return hipGetLastError();
}

}  // namespace

hipError_t layernorm(const float* x, int M, int D, const uint16_t* g, const uint16_t* b, float eps, void* out,
                     int out_f32, hipStream_t s) {
  if (!x || !g || !b || !out || M < 1 || D < 64 || (D & 63) || D > 64 * kMaxPer) return hipErrorInvalidValue;
  switch (D / 64) {
#define TP_LN_CASE(P) \
  case P: return launch_ln<P>(x, M, g, b, eps, out, out_f32, s);
    TP_LN_CASE(1) TP_LN_CASE(2) TP_LN_CASE(3) TP_LN_CASE(4) TP_LN_CASE(5) TP_LN_CASE(6) TP_LN_CASE(7) TP_LN_CASE(8)
    TP_LN_CASE(9) TP_LN_CASE(10) TP_LN_CASE(11) TP_LN_CASE(12) TP_LN_CASE(13) TP_LN_CASE(14) TP_LN_CASE(15)
    TP_LN_CASE(16)
#undef TP_LN_CASE
  }
  return hipErrorInvalidValue;
}

hipError_t embed_ln(const int32_t* ids, int M, int S, int D, int vocab, const uint16_t* tok, const uint16_t* pos,
                    const uint16_t* type, const uint16_t* g, const uint16_t* b, float eps, uint16_t* out,
                    hipStream_t s) {
  if (!ids || !tok || !pos || !type || !g || !b || !out || M < 1 || S < 1 || vocab < 1 || D < 64 || (D & 63) ||
      D > 64 * kMaxPer)
    return hipErrorInvalidValue;
  switch (D / 64) {
#define TP_EMB_CASE(P) \
  case P: return launch_embed<P>(ids, M, S, vocab, tok, pos, type, g, b, eps, out, s);
    TP_EMB_CASE(1) TP_EMB_CASE(2) TP_EMB_CASE(3) TP_EMB_CASE(4) TP_EMB_CASE(5) TP_EMB_CASE(6) TP_EMB_CASE(7)
    TP_EMB_CASE(8) TP_EMB_CASE(9) TP_EMB_CASE(10) TP_EMB_CASE(11) TP_EMB_CASE(12) TP_EMB_CASE(13) TP_EMB_CASE(14)
    TP_EMB_CASE(15) TP_EMB_CASE(16)
#undef TP_EMB_CASE
  }
  return hipErrorInvalidValue;
}

}  // namespace k
}  // namespace tp
