// Argument block and row epilogue shared by the bf16 contraction kernels (skinny and
// tiled), and the launcher of the skinny one.
#pragma once
#include "common.hpp"
#include "kernels.hpp"

namespace tp {
namespace k {

// activation loaders: row-major matrix; NHWC im2col with C % 64 == 0 (a 64-deep k-stage
// then lies inside one filter tap)
enum { X_ROWS = 0, X_CONV64 = 3 };

struct GemmArgs {
  const uint16_t* x;
  const uint16_t* w;
  int M, N, K;
  int H, W, C, KW, stride, pad, Ho, Wo;   // convolution geometry (X_CONV*)
  Epilogue ep;
  int kst, splits;                        // k-stages per split, number of splits
  float* partials;                        // [splits][M][N] fp32 when splits > 1
};

template <>
struct PtrFields<GemmArgs> {
  static void add(std::vector<uint32_t>& v, uint32_t at) {
    for (size_t o : {offsetof(GemmArgs, x), offsetof(GemmArgs, w), offsetof(GemmArgs, partials),
                     offsetof(GemmArgs, ep) + offsetof(Epilogue, bias), offsetof(GemmArgs, ep) + offsetof(Epilogue, res),
                     offsetof(GemmArgs, ep) + offsetof(Epilogue, out), offsetof(GemmArgs, ep) + offsetof(Epilogue, ln_g),
                     offsetof(GemmArgs, ep) + offsetof(Epilogue, ln_b), offsetof(GemmArgs, ep) + offsetof(Epilogue, ln_out)})
      v.push_back(at + (uint32_t)o);
  }
};

__device__ __forceinline__ int res_kind_dev(const Epilogue& ep) { return !ep.res ? 0 : ep.res_f32 ? 2 : 1; }

// The epilogue's inputs for four consecutive outputs of a row, as raw bits: fetched
// ahead of the values they apply to, so that their loads overlap other loads. `base` is
// m * N + n0; requires n0 % 4 == 0, n0 + 3 < N, N % 4 == 0.
// RES, when not -1, fixes the residual's kind at compile time (0 none, 1 bf16, 2 fp32; see
// res_kind): a kernel that fetches these ahead of other loads then has no branch between
// the loads, which would otherwise make the compiler wait for one before issuing the next.
struct Ep4In {
  uint2 bias;   // bf16 x 4
  uint4 res;    // fp32 x 4, or bf16 x 4 in .x and .y
};

inline int res_kind(const Epilogue& ep) { return !ep.res ? 0 : ep.res_f32 ? 2 : 1; }

template <int RES = -1>
__device__ __forceinline__ Ep4In ep4_fetch(const Epilogue& ep, size_t base, int n0) {
  Ep4In in;   // fields the epilogue does not use stay unset (no copies, no waits)
  if (ep.bias) in.bias = *reinterpret_cast<const uint2*>(ep.bias + n0);
  const int rk = RES >= 0 ? RES : res_kind_dev(ep);
  if (rk == 2) {
    in.res = *reinterpret_cast<const uint4*>(static_cast<const float*>(ep.res) + base);
  } else if (rk == 1) {
    const uint2 r = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(ep.res) + base);
    in.res.x = r.x; in.res.y = r.y;
  }
  return in;
}

// v += bias; v += residual; v = act(v), each step only where the epilogue has it
template <int RES = -1>
__device__ __forceinline__ void ep4_apply(const Epilogue& ep, const Ep4In& in, float (&v)[4]) {
  if (ep.bias) {
    v[0] += bf2f(in.bias.x & 0xffff); v[1] += bf2f(in.bias.x >> 16);
    v[2] += bf2f(in.bias.y & 0xffff); v[3] += bf2f(in.bias.y >> 16);
  }
  const int rk = RES >= 0 ? RES : res_kind_dev(ep);
  if (rk == 2) {
    v[0] += __uint_as_float(in.res.x); v[1] += __uint_as_float(in.res.y);
    v[2] += __uint_as_float(in.res.z); v[3] += __uint_as_float(in.res.w);
  } else if (rk == 1) {
    v[0] += bf2f(in.res.x & 0xffff); v[1] += bf2f(in.res.x >> 16);
    v[2] += bf2f(in.res.y & 0xffff); v[3] += bf2f(in.res.y >> 16);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = act_apply(v[e], ep.act);
}

__device__ __forceinline__ void ep4_store(const Epilogue& ep, size_t base, const float (&v)[4]) {
  if (ep.out_f32) {
    *reinterpret_cast<float4*>(static_cast<float*>(ep.out) + base) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    uint2 o;
    o.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
    o.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(ep.out) + base) = o;
  }
}

__device__ __forceinline__ void store_row4(const GemmArgs& a, int m, int n0, f32x4 acc) {
  if (m >= a.M || n0 >= a.N) return;
  const Epilogue& ep = a.ep;
  const size_t base = (size_t)m * a.N + n0;
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = acc[e];
  const bool full = (n0 + 3 < a.N) && ((a.N & 3) == 0);
  if (full) {
    const Ep4In in = ep4_fetch(ep, base, n0);
    ep4_apply(ep, in, v);
    ep4_store(ep, base, v);
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
// split_group(s): how many split partials a reduction thread loads before it adds any
// (2, 4 or 8: the smallest that covers s, at most 8).
__host__ __device__ constexpr int split_group(int s) { return s <= 2 ? 2 : s <= 4 ? 4 : 8; }
bool split_reduce_ln_fits(int N);
hipError_t split_reduce_ln(const GemmArgs& a, hipStream_t s);

// M <= 32 rows: the skinny kernel (gemv_bf16.hip)
hipError_t launch_skinny(const GemmArgs& a, hipStream_t s);

}  // namespace k
}  // namespace tp
