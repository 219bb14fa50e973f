// Skinny bf16 contraction (M <= 32 activation rows) on gfx950 MFMA
// (v_mfma_f32_16x16x32_bf16), fp32 accumulate, fused epilogue. The weights dominate the
// traffic, so the kernel is HBM-bound: each workgroup owns 16 weight rows and each of its
// waves streams one contiguous run of 128-wide k-blocks (measured 3-4% faster than
// interleaving the waves' blocks) with 4 x 16-byte loads per lane per block in flight, then
// the waves reduce through LDS in a fixed order. The operand convention is the one of every
// contraction here: the MFMA "A" operand is 16 weight rows, the "B" operand 16 activation
// rows, so accumulator register e of lane l holds D[n = 4 (l / 16) + e][m = l % 16].
#include "gemm_args.hpp"

#ifndef GEMV_NW
#define GEMV_NW 4
#define GEMV_U 8
#endif

namespace tp {
namespace k {

namespace {

// PK: weights in 16 x 128 blocks (see pack_rows16x128 in the host code), so load j of
// lane (r, q) in k-block kb reads 16 bytes at block offset j*512 + (q*16 + r)*8 and one
// load instruction covers a contiguous 1 KB; otherwise rows are [N][K] and an instruction
// reads 64 contiguous bytes of each of 16 rows. Activation rows beyond M issue no load.
template <int MT, int NW, int U, bool PK>
__global__ __launch_bounds__(NW * 64) void k_gemv(GemmArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int n0 = blockIdx.x * 16;
  const bool nvalid = n0 + r < a.N;
  const int nkb = (a.K + 127) >> 7;
  const uint16_t* wrow = PK ? a.w + (size_t)blockIdx.x * nkb * 2048 + lane * 8
                            : a.w + (size_t)(nvalid ? n0 + r : 0) * a.K;
  const uint16_t* xrow[MT];
  bool mvalid[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int m = (t << 4) + r;
    mvalid[t] = m < a.M;
    xrow[t] = a.x + (size_t)(mvalid[t] ? m : 0) * a.K;
  }
  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  // the epilogue's bias, fetched now (raw bits, converted at the end) so that its latency
  // hides behind the weight stream
  const int nst = n0 + (q << 2);
  const bool bias_pre = wave < MT && a.ep.bias && nst + 3 < a.N && (a.N & 3) == 0;
  uint2 braw = make_uint2(0, 0);
  if (bias_pre) braw = *reinterpret_cast<const uint2*>(a.ep.bias + nst);
  // k-block of 128: load j of lane (r, q) covers k = kb*128 + 32 j + 8 q .. +8
  const int per = (nkb + NW - 1) / NW, kb_end = min(nkb, (wave + 1) * per);
  for (int kb0 = wave * per; kb0 < kb_end; kb0 += U) {
    uint4 av[U][4], bv[U][MT][4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + u;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kk = (kb << 7) + (j << 5) + (q << 3);
        const bool kin = kb < kb_end && kk < a.K;
        const int ks = kin ? kk : 0;
        // weights are streamed once per forward pass: non-temporal loads
        if (PK)
          av[u][j] = mask_u4(load_nt16(wrow + (size_t)(kin ? kb : 0) * 2048 + j * 512), kin);
        else
          av[u][j] = mask_u4(load_nt16(wrow + ks), nvalid && kin);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          uint4 v = make_uint4(0, 0, 0, 0);
          if (mvalid[t] && kin) v = *reinterpret_cast<const uint4*>(xrow[t] + ks);
          bv[u][t][j] = v;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int t = 0; t < MT; ++t)
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av[u][j]), as_bf16x8(bv[u][t][j]), acc[t], 0, 0,
                                                           0);
  }
  __shared__ f32x4 red[NW][MT][64];
#pragma unroll
  for (int t = 0; t < MT; ++t) red[wave][t][lane] = acc[t];
  __syncthreads();
  if (wave < MT) {
    f32x4 s = red[0][wave][lane];
    for (int w = 1; w < NW; ++w) s += red[w][wave][lane];
    if (bias_pre) {
      // the same arithmetic as store_row4 with the bias it would load
      GemmArgs b = a;
      b.ep.bias = nullptr;
      s[0] += bf2f(braw.x & 0xffff); s[1] += bf2f(braw.x >> 16); s[2] += bf2f(braw.y & 0xffff); s[3] += bf2f(braw.y >> 16);
      store_row4(b, (wave << 4) + r, nst, s);
    } else {
      store_row4(a, (wave << 4) + r, nst, s);
    }
  }
}

}  // namespace

hipError_t launch_skinny(const GemmArgs& a, hipStream_t s) {
  const dim3 grid((a.N + 15) / 16), block(GEMV_NW * 64);
  if (a.M <= 16) {
    if (a.ep.w_packed) (void)launch((k_gemv<1, GEMV_NW, GEMV_U, true>), grid, block, 0, s, a);
    else (void)launch((k_gemv<1, GEMV_NW, GEMV_U, false>), grid, block, 0, s, a);
  } else {
    if (a.ep.w_packed) (void)launch((k_gemv<2, GEMV_NW, GEMV_U, true>), grid, block, 0, s, a);
    else (void)launch((k_gemv<2, GEMV_NW, GEMV_U, false>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace k
}  // namespace tp
