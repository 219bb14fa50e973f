// Multi-head self-attention for head dim 64 and short sequences (S <= 256, S % 32 == 0),
// one workgroup per (sample, head, 16 NW queries); each wave owns 16 queries.
//
// K and V of the head are staged row-major in LDS ([key][d]). Scores are
// computed as S^T = K Q^T on MFMA (A = 16 keys, B = 16 queries), so lane l holds the
// scores of query l % 16 against keys 16 t + 4 (l / 16) + e. The softmax reductions
// over keys therefore stay inside a lane plus two cross-lane exchanges (lanes l ^ 16,
// l ^ 32), in fp32. The normalised probabilities, rounded to bf16, are used directly as
// the A operand of O = P V: a 32-key MFMA k-block takes the lane's own values from two
// consecutive score tiles, and the matching V entries are read with gfx950's transposing LDS
// load (ds_read_b64_tr_b16) in the same key order, so no data moves between lanes.
#include "common.hpp"
#include "kernels.hpp"

namespace tp {
namespace k {
namespace {

// FULL: S == SMAX, so every key tile is valid at compile time (with a run-time tile count
// the conditional MFMA accumulators compiled to hundreds of register copies)
template <int SMAX, bool FULL, int NW>
__global__ __launch_bounds__(64 * NW) void k_attention(const uint16_t* __restrict__ qkv, int S_arg, int H,
                                                       uint16_t* __restrict__ out) {
  constexpr int LDK = 72, LDV = 80, NT = SMAX / 16, NTHR = 64 * NW;
  const int S = FULL ? SMAX : S_arg;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[SMAX * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[SMAX * LDV];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int h = blockIdx.y, b = blockIdx.z;
  const int D = H * 64, ld = 3 * D;
  const uint16_t* base = qkv + (size_t)b * S * ld;

  // this wave's queries first (independent of the staging); a wave past the sequence end
  // loads row 0 and does nothing with it
  const int q0 = blockIdx.x * (16 * NW) + wave * 16;
  const bool active = q0 < S;
  const uint16_t* qrow = base + (size_t)(active ? q0 + r : 0) * ld + h * 64 + (g << 3);
  const uint4 qf0 = *reinterpret_cast<const uint4*>(qrow);
  const uint4 qf1 = *reinterpret_cast<const uint4*>(qrow + 32);

  // K and V of the head: every load of this thread issued before the first LDS store, so
  // the round trips overlap. Both are read as key = 32 i + tid / 8, 8 dims at (tid % 8) * 8,
  // a key's 128 bytes per 8 lanes, so one wave's load covers 8 whole rows; both are stored
  // as whole 16-byte pieces. (V stored transposed 2 bytes at a time, read as 8-byte pieces,
  // took 5.6 / 5.5 us per launch at BERT-base batch 1 / 8 with the best padding of several;
  // other transposes, by lanes holding 64 consecutive keys or by an 8 x 8 exchange among
  // lanes, 6.7-7.4 us; all the same bits.)
  constexpr int NV = SMAX * 8 / NTHR;
  static_assert(SMAX * 8 % NTHR == 0 && SMAX % 64 == 0, "staging map");
  uint4 kv[NV], vv[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int key = (i * NTHR + tid) >> 3, d8 = (tid & 7) << 3;
    const uint16_t* row = base + (size_t)(key < S ? key : 0) * ld + h * 64 + d8;
    kv[i] = *reinterpret_cast<const uint4*>(row + D);
    vv[i] = *reinterpret_cast<const uint4*>(row + 2 * D);
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int key = (i * NTHR + tid) >> 3, d8 = (tid & 7) << 3;
    if (key < S) {
      *reinterpret_cast<uint4*>(&Ks[key * LDK + d8]) = kv[i];
      *reinterpret_cast<uint4*>(&Vs[key * LDV + d8]) = vv[i];
    }
  }
  __syncthreads();

  if (!active) return;
  const int nt = S >> 4;

  f32x4 sc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    sc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (t < nt) {
      const uint16_t* krow = &Ks[(16 * t + r) * LDK + (g << 3)];
      sc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(*reinterpret_cast<const uint4*>(krow)),
                                                      as_bf16x8(qf0), sc[t], 0, 0, 0);
      sc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(*reinterpret_cast<const uint4*>(krow + 32)),
                                                      as_bf16x8(qf1), sc[t], 0, 0, 0);
    }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int t = 0; t < NT; ++t)
    if (t < nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = fmaxf(mx, sc[t][e]);
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  float sum = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
    if (t < nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // exp((s - max) / sqrt(64)) as one hardware base-2 exponential
        const float p = __builtin_amdgcn_exp2f((sc[t][e] - mx) * (0.125f * 1.44269504088896341f));
        sc[t][e] = p;
        sum += p;
      }
  sum += __shfl_xor(sum, 16, 64);
  sum += __shfl_xor(sum, 32, 64);
  const float inv = 1.f / sum;

  f32x4 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < NT / 2; ++u) {
    if (2 * u < nt) {
      const f32x4 p0 = sc[2 * u], p1 = sc[2 * u + 1];
      uint4 pa;
      pa.x = (uint32_t)f2bf(p0[0] * inv) | ((uint32_t)f2bf(p0[1] * inv) << 16);
      pa.y = (uint32_t)f2bf(p0[2] * inv) | ((uint32_t)f2bf(p0[3] * inv) << 16);
      pa.z = (uint32_t)f2bf(p1[0] * inv) | ((uint32_t)f2bf(p1[1] * inv) << 16);
      pa.w = (uint32_t)f2bf(p1[2] * inv) | ((uint32_t)f2bf(p1[3] * inv) << 16);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        // V^T fragment of keys 32 u + 4 g + 0..3 (lo) and 16 further (hi), dim 16 dt + r, read
        // transposed from row-major V: within a 16-lane group, lane l receives element l % 4 of
        // the 8-byte pieces the group's lanes l / 4 + 4 j (j = 0..3) address, so lane s of the
        // group addresses key row (s % 16) / 4 at dims 16 dt + 4 (s % 4)
        const uint16_t* vr = &Vs[(32 * u + 4 * g + (r >> 2)) * LDV + 16 * dt + 4 * (r & 3)];
        typedef short v4s __attribute__((ext_vector_type(4)));
        const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)vr);
        const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(vr + 16 * LDV));
        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(pa), as_bf16x8(make_uint4(l2.x, l2.y, h2.x, h2.y)),
                                                        o[dt], 0, 0, 0);
      }
    }
  }
  // lane holds O[query q0 + 4 g + e][d = 16 dt + r]
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      out[((size_t)b * S + q0 + 4 * g + e) * D + h * 64 + 16 * dt + r] = f2bf(o[dt][e]);
}

}  // namespace

hipError_t attention(const uint16_t* qkv, int B, int S, int H, uint16_t* out, hipStream_t s) {
  if (!qkv || !out || B < 1 || H < 1 || S < 32 || (S & 31) || S > 256) return hipErrorInvalidValue;
  // four waves (64 queries) per workgroup: with one or two, staging K and V once per
  // workgroup costs more than the extra workgroups gain (BERT-base at batch 8: 0.790 ms warm
  // with four, 0.839 with two, 0.915 with one; with the present staging, two waves at batch
  // 1, where four leave 24 workgroups on 256 CUs: 0.462 -> 0.475 ms)
  constexpr int NW = 4;
  dim3 grid((S + 16 * NW - 1) / (16 * NW), H, B), block(64 * NW);
  if (S == 128) (void)launch((k_attention<128, true, NW>), grid, block, 0, s, qkv, S, H, out);
  else if (S < 128) (void)launch((k_attention<128, false, NW>), grid, block, 0, s, qkv, S, H, out);
  else if (S == 256) (void)launch((k_attention<256, true, NW>), grid, block, 0, s, qkv, S, H, out);
  else (void)launch((k_attention<256, false, NW>), grid, block, 0, s, qkv, S, H, out);
  return hipGetLastError();
}

}  // namespace k
}  // namespace tp
