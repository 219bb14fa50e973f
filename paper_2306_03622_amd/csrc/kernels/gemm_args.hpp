// Argument block and row epilogue shared by the bf16 contraction kernels (skinny and
// tiled), and the launcher of the skinny one.
#pragma once
#include "common.hpp"
#include "kernels.hpp"

namespace tp {
namespace k {

// activation loaders: row-major matrix; NHWC im2col with C % 64 == 0 (a 64-deep k-stage
// then lies inside one filter tap); NHWC im2col with C % 8 == 0; element-wise im2col
enum { X_ROWS = 0, X_CONV8 = 1, X_CONV1 = 2, X_CONV64 = 3 };

struct GemmArgs {
  const uint16_t* x;
  const uint16_t* w;
  int M, N, K;
  int H, W, C, KW, stride, pad, Ho, Wo;   // convolution geometry (X_CONV*)
  Epilogue ep;
  int kst, splits;                        // k-stages per split, number of splits
  float* partials;                        // [splits][M][N] fp32 when splits > 1
};

__device__ __forceinline__ void store_row4(const GemmArgs& a, int m, int n0, f32x4 acc) {
  if (m >= a.M || n0 >= a.N) return;
  const Epilogue& ep = a.ep;
  const size_t base = (size_t)m * a.N + n0;
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = acc[e];
  const bool full = (n0 + 3 < a.N) && ((a.N & 3) == 0);
  if (full) {
    if (ep.bias) {
      const uint2 b = *reinterpret_cast<const uint2*>(ep.bias + n0);
      v[0] += bf2f(b.x & 0xffff); v[1] += bf2f(b.x >> 16); v[2] += bf2f(b.y & 0xffff); v[3] += bf2f(b.y >> 16);
    }
    if (ep.res) {
      if (ep.res_f32) {
        const float4 r = *reinterpret_cast<const float4*>(static_cast<const float*>(ep.res) + base);
        v[0] += r.x; v[1] += r.y; v[2] += r.z; v[3] += r.w;
      } else {
        const uint2 r = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(ep.res) + base);
        v[0] += bf2f(r.x & 0xffff); v[1] += bf2f(r.x >> 16); v[2] += bf2f(r.y & 0xffff); v[3] += bf2f(r.y >> 16);
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = act_apply(v[e], ep.act);
    if (ep.out_f32) {
      *reinterpret_cast<float4*>(static_cast<float*>(ep.out) + base) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
      uint2 o;
      o.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
      o.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(ep.out) + base) = o;
    }
    return;
  }
  for (int e = 0; e < 4 && n0 + e < a.N; ++e) {
    float t = v[e];
    if (ep.bias) t += bf2f(ep.bias[n0 + e]);
    if (ep.res) t += ep.res_f32 ? static_cast<const float*>(ep.res)[base + e]
                                : bf2f(static_cast<const uint16_t*>(ep.res)[base + e]);
    t = act_apply(t, ep.act);
    if (ep.out_f32) static_cast<float*>(ep.out)[base + e] = t;
    else static_cast<uint16_t*>(ep.out)[base + e] = f2bf(t);
  }
}

// The reduction of a split contraction fused with the row LayerNorm of its result
// (norm.hip); split_reduce_ln_fits tells whether it applies to width N.
bool split_reduce_ln_fits(int N);
hipError_t split_reduce_ln(const GemmArgs& a, hipStream_t s);

// M <= 32 rows: the skinny kernel (gemv_bf16.hip)
hipError_t launch_skinny(const GemmArgs& a, hipStream_t s);

}  // namespace k
}  // namespace tp
