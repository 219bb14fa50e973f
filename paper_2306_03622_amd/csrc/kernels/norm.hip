// Row LayerNorm and the fused embedding gather + LayerNorm. One wave per row, each lane
// holding D/64 elements in registers; mean and variance (two passes over the registers,
// population variance) use butterfly wave reductions in fp32. When D/64 is a multiple of 4
// a lane holds a contiguous run of the row (16-byte fp32 and 8-byte bf16 accesses);
// otherwise element lane + 64 i.
#include "common.hpp"
#include "gemm_args.hpp"
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

// gamma and beta of a lane's run of PER contiguous elements (c = PER lane + i), raw bf16
// bits, fetched before the row so that their loads overlap the row's
template <int PER>
struct LnAffine {
  uint2 g[PER / 4], b[PER / 4];
  __device__ __forceinline__ void fetch(const uint16_t* gp, const uint16_t* bp, int c0) {
#pragma unroll
    for (int i = 0; i < PER / 4; ++i) {
      g[i] = *reinterpret_cast<const uint2*>(gp + c0 + 4 * i);
      b[i] = *reinterpret_cast<const uint2*>(bp + c0 + 4 * i);
    }
  }
};

// The same for a row held as PER contiguous values per lane (element c = PER lane + i).
template <int PER>
__device__ __forceinline__ void normalize_runs(float (&v)[PER], int D, const LnAffine<PER>& af, float eps, int lane,
                                               void* out, size_t row_off, int out_f32) {
  static_assert(PER % 4 == 0, "runs of 4");
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
  const int c0 = lane * PER;
#pragma unroll
  for (int i = 0; i < PER; i += 4) {
    const uint2 gg = af.g[i / 4], bb = af.b[i / 4];
    float y[4];
    y[0] = (v[i] - mean) * rstd * bf2f(gg.x & 0xffff) + bf2f(bb.x & 0xffff);
    y[1] = (v[i + 1] - mean) * rstd * bf2f(gg.x >> 16) + bf2f(bb.x >> 16);
    y[2] = (v[i + 2] - mean) * rstd * bf2f(gg.y & 0xffff) + bf2f(bb.y & 0xffff);
    y[3] = (v[i + 3] - mean) * rstd * bf2f(gg.y >> 16) + bf2f(bb.y >> 16);
    if (out_f32) {
      *reinterpret_cast<float4*>(static_cast<float*>(out) + row_off + c0 + i) = make_float4(y[0], y[1], y[2], y[3]);
    } else {
      uint2 o;
      o.x = (uint32_t)f2bf(y[0]) | ((uint32_t)f2bf(y[1]) << 16);
      o.y = (uint32_t)f2bf(y[2]) | ((uint32_t)f2bf(y[3]) << 16);
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(out) + row_off + c0 + i) = o;
    }
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
  if constexpr (PER % 4 == 0) {
    LnAffine<PER> af;
    af.fetch(g, b, lane * PER);
#pragma unroll
    for (int i = 0; i < PER; i += 4) {
      const float4 t = *reinterpret_cast<const float4*>(xr + lane * PER + i);
      v[i] = t.x; v[i + 1] = t.y; v[i + 2] = t.z; v[i + 3] = t.w;
    }
    normalize_runs<PER>(v, D, af, eps, lane, out, (size_t)row * D, out_f32);
  } else {
#pragma unroll
    for (int i = 0; i < PER; ++i) v[i] = xr[lane + 64 * i];
    normalize<PER>(v, D, g, b, eps, lane, out, (size_t)row * D, out_f32);
  }
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
  if constexpr (PER % 4 == 0) {
    LnAffine<PER> af;
    af.fetch(g, b, lane * PER);
#pragma unroll
    for (int i = 0; i < PER; i += 4) {
      const int c = lane * PER + i;
      const uint2 t = *reinterpret_cast<const uint2*>(tok + (size_t)id * D + c);
      const uint2 p = *reinterpret_cast<const uint2*>(pos + (size_t)s * D + c);
      const uint2 y = *reinterpret_cast<const uint2*>(type + c);
      v[i] = bf2f(t.x & 0xffff) + bf2f(p.x & 0xffff) + bf2f(y.x & 0xffff);
      v[i + 1] = bf2f(t.x >> 16) + bf2f(p.x >> 16) + bf2f(y.x >> 16);
      v[i + 2] = bf2f(t.y & 0xffff) + bf2f(p.y & 0xffff) + bf2f(y.y & 0xffff);
      v[i + 3] = bf2f(t.y >> 16) + bf2f(p.y >> 16) + bf2f(y.y >> 16);
    }
    normalize_runs<PER>(v, D, af, eps, lane, out, (size_t)row * D, 0);
  } else {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = lane + 64 * i;
      v[i] = bf2f(tok[(size_t)id * D + c]) + bf2f(pos[(size_t)s * D + c]) + bf2f(type[c]);
    }
    normalize<PER>(v, D, g, b, eps, lane, out, (size_t)row * D, 0);
  }
}

// The reduction of a contraction split over k, fused with the row LayerNorm of its result:
// one wave per row sums the fp32 partials in split order, applies the contraction's
// epilogue arithmetic (bias, residual, activation: the same operations in the same order
// as the plain reduction) and normalises the row in registers. Only the LayerNorm output is
// written. The epilogue's inputs, gamma, beta and ZG partials are all fetched before the
// first addition, so the row costs one memory round trip per ZG splits.
template <int PER, int ZG, int RES>
__global__ __launch_bounds__(256) void k_split_reduce_ln(GemmArgs a) {
  constexpr int D = 64 * PER, R = PER / 4;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.M) return;
  const Epilogue& ep = a.ep;
  const int c0 = lane * PER;
  const size_t base = (size_t)row * D + c0, plane = (size_t)a.M * D;
  Ep4In in[R];
#pragma unroll
  for (int i = 0; i < R; ++i) in[i] = ep4_fetch<RES>(ep, base + 4 * i, c0 + 4 * i);
  LnAffine<PER> af;
  af.fetch(ep.ln_g, ep.ln_b, c0);
  float v[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) v[i] = 0.f;
  for (int z0 = 0; z0 < a.splits; z0 += ZG) {
    float4 t[ZG][R];
#pragma unroll
    for (int u = 0; u < ZG; ++u)
#pragma unroll
      for (int i = 0; i < R; ++i)
        if (z0 + u < a.splits) t[u][i] = *reinterpret_cast<const float4*>(a.partials + (z0 + u) * plane + base + 4 * i);
#pragma unroll
    for (int u = 0; u < ZG; ++u)
#pragma unroll
      for (int i = 0; i < R; ++i)
        if (z0 + u < a.splits) {
          v[4 * i] += t[u][i].x; v[4 * i + 1] += t[u][i].y; v[4 * i + 2] += t[u][i].z; v[4 * i + 3] += t[u][i].w;
        }
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    float w[4] = {v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]};
    ep4_apply<RES>(ep, in[i], w);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[4 * i + e] = w[e];
  }
  normalize_runs<PER>(v, D, af, ep.ln_eps, lane, ep.ln_out, (size_t)row * D, ep.ln_out_f32);
}

template <int PER, int RES>
void launch_split_reduce_ln_res(const GemmArgs& a, dim3 grid, dim3 block, hipStream_t s) {
  switch (split_group(a.splits)) {
    case 2: (void)launch((k_split_reduce_ln<PER, 2, RES>), grid, block, 0, s, a); break;
    case 4: (void)launch((k_split_reduce_ln<PER, 4, RES>), grid, block, 0, s, a); break;
    default: (void)launch((k_split_reduce_ln<PER, 8, RES>), grid, block, 0, s, a); break;
  }
}

template <int PER>
void launch_split_reduce_ln(const GemmArgs& a, dim3 grid, dim3 block, hipStream_t s) {
  switch (res_kind(a.ep)) {
    case 0: launch_split_reduce_ln_res<PER, 0>(a, grid, block, s); break;
    case 1: launch_split_reduce_ln_res<PER, 1>(a, grid, block, s); break;
    default: launch_split_reduce_ln_res<PER, 2>(a, grid, block, s); break;
  }
}

template <int PER>
hipError_t launch_ln(const float* x, int M, const uint16_t* g, const uint16_t* b, float eps, void* out, int out_f32,
                     hipStream_t s) {
  (void)launch((k_layernorm<PER>), dim3((M + 3) / 4), dim3(256), 0, s, x, M, g, b, eps, out, out_f32);
  return hipGetLastError();
}

template <int PER>
hipError_t launch_embed(const int32_t* ids, int M, int S, int vocab, const uint16_t* tok, const uint16_t* pos,
                        const uint16_t* type, const uint16_t* g, const uint16_t* b, float eps, uint16_t* out,
                        hipStream_t s) {
  (void)launch((k_embed_ln<PER>), dim3((M + 3) / 4), dim3(256), 0, s, ids, M, S, vocab, tok, pos, type, g, b,
                     eps, out);
  return hipGetLastError();
}

}  // namespace

bool split_reduce_ln_fits(int N) { return N >= 256 && N <= 64 * kMaxPer && N % 256 == 0; }

hipError_t split_reduce_ln(const GemmArgs& a, hipStream_t s) {
  if (!split_reduce_ln_fits(a.N) || !a.ep.ln_g || !a.ep.ln_b || !a.ep.ln_out || a.splits < 1) return hipErrorInvalidValue;
  const dim3 grid((a.M + 3) / 4), block(256);
  switch (a.N / 64) {
    case 4: launch_split_reduce_ln<4>(a, grid, block, s); break;
    case 8: launch_split_reduce_ln<8>(a, grid, block, s); break;
    case 12: launch_split_reduce_ln<12>(a, grid, block, s); break;
    default: launch_split_reduce_ln<16>(a, grid, block, s); break;
  }
  return hipGetLastError();
}

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
