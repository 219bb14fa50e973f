// bf16 contractions on gfx950 MFMA (v_mfma_f32_16x16x32_bf16), fp32 accumulate, with a
// fused epilogue (bias, optional residual, ReLU/GELU, bf16 or fp32 store).
//
// Convention for every kernel here: the MFMA "A" operand is a 16-row block of the weight
// matrix W[N][K] (rows = output features n) and the "B" operand a 16-row block of the
// activations X[M][K] (rows = tokens / output pixels m). Both are read as 8 consecutive
// k per lane, lane l covering row (l % 16) and k-slot (l / 16), so one accumulator
// register e of lane l holds D[n = 4 (l / 16) + e][m = l % 16]: four consecutive output
// features of one row, which the epilogue stores as one vector.
//
// Kernels here (the skinny M <= 32 case is in gemv_bf16.hip):
//   * k_gemm: LDS-tiled BN x BM x BK tiles, 4 waves in a 2 x 2 arrangement, global loads
//     issued several k-stages ahead into a register ring, double-buffered LDS, and a
//     deterministic split over k when the tile grid alone cannot fill the chip. The
//     activation loader is either a plain row-major matrix or an NHWC implicit-GEMM
//     (im2col) gather for convolutions, k = (kh * KW + kw) * C + c, matching OHWI weight
//     rows.
//   * k_conv_smallc: convolutions with fewer than 8 input channels (the ResNet stem),
//     whose input window rows are staged in LDS.
#include "gemm_args.hpp"

namespace tp {
namespace k {

namespace {

// Epilogue of 16 consecutive outputs n0 .. n0+15 of row m (contiguous loads and stores)
__device__ __forceinline__ void store_row16(const GemmArgs& a, int m, int n0, const float (&v_in)[16]) {
  const Epilogue& ep = a.ep;
  const size_t base = (size_t)m * a.N + n0;
  if (n0 + 15 < a.N && (a.N & 7) == 0) {
    float v[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) v[e] = v_in[e];
    if (ep.bias) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4 b = *reinterpret_cast<const uint4*>(ep.bias + n0 + 8 * h);
        const uint32_t w[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[8 * h + 2 * e] += bf2f(w[e] & 0xffff);
          v[8 * h + 2 * e + 1] += bf2f(w[e] >> 16);
        }
      }
    }
    if (ep.res) {
      if (ep.res_f32) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const float4 r = *reinterpret_cast<const float4*>(static_cast<const float*>(ep.res) + base + 4 * h);
          v[4 * h] += r.x; v[4 * h + 1] += r.y; v[4 * h + 2] += r.z; v[4 * h + 3] += r.w;
        }
      } else {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint4 r = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(ep.res) + base + 8 * h);
          const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[8 * h + 2 * e] += bf2f(w[e] & 0xffff);
            v[8 * h + 2 * e + 1] += bf2f(w[e] >> 16);
          }
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) v[e] = act_apply(v[e], ep.act);
    if (ep.out_f32) {
#pragma unroll
      for (int h = 0; h < 4; ++h)
        *reinterpret_cast<float4*>(static_cast<float*>(ep.out) + base + 4 * h) =
            make_float4(v[4 * h], v[4 * h + 1], v[4 * h + 2], v[4 * h + 3]);
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint4 o;
        o.x = (uint32_t)f2bf(v[8 * h]) | ((uint32_t)f2bf(v[8 * h + 1]) << 16);
        o.y = (uint32_t)f2bf(v[8 * h + 2]) | ((uint32_t)f2bf(v[8 * h + 3]) << 16);
        o.z = (uint32_t)f2bf(v[8 * h + 4]) | ((uint32_t)f2bf(v[8 * h + 5]) << 16);
        o.w = (uint32_t)f2bf(v[8 * h + 6]) | ((uint32_t)f2bf(v[8 * h + 7]) << 16);
        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(ep.out) + base + 8 * h) = o;
      }
    }
    return;
  }
  for (int e = 0; e < 16 && n0 + e < a.N; ++e) {
    float t = v_in[e];
    if (ep.bias) t += bf2f(ep.bias[n0 + e]);
    if (ep.res) t += ep.res_f32 ? static_cast<const float*>(ep.res)[base + e]
                                : bf2f(static_cast<const uint16_t*>(ep.res)[base + e]);
    t = act_apply(t, ep.act);
    if (ep.out_f32) static_cast<float*>(ep.out)[base + e] = t;
    else static_cast<uint16_t*>(ep.out)[base + e] = f2bf(t);
  }
}

// store_row16 with the bias and a bf16 residual already loaded (raw bits of 16 values each);
// requires n0 + 15 < N and N % 8 == 0. The same operations in the same order, so the same bits.
__device__ __forceinline__ void store_row16_pre(const GemmArgs& a, int m, int n0, const float (&v_in)[16],
                                                const uint4 (&bias)[2], const uint4 (&res)[2]) {
  const Epilogue& ep = a.ep;
  const size_t base = (size_t)m * a.N + n0;
  float v[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) v[e] = v_in[e];
  if (ep.bias) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t w[4] = {bias[h].x, bias[h].y, bias[h].z, bias[h].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[8 * h + 2 * e] += bf2f(w[e] & 0xffff);
        v[8 * h + 2 * e + 1] += bf2f(w[e] >> 16);
      }
    }
  }
  if (ep.res) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t w[4] = {res[h].x, res[h].y, res[h].z, res[h].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[8 * h + 2 * e] += bf2f(w[e] & 0xffff);
        v[8 * h + 2 * e + 1] += bf2f(w[e] >> 16);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 16; ++e) v[e] = act_apply(v[e], ep.act);
  if (ep.out_f32) {
#pragma unroll
    for (int h = 0; h < 4; ++h)
      *reinterpret_cast<float4*>(static_cast<float*>(ep.out) + base + 4 * h) =
          make_float4(v[4 * h], v[4 * h + 1], v[4 * h + 2], v[4 * h + 3]);
  } else {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint4 o;
      o.x = (uint32_t)f2bf(v[8 * h]) | ((uint32_t)f2bf(v[8 * h + 1]) << 16);
      o.y = (uint32_t)f2bf(v[8 * h + 2]) | ((uint32_t)f2bf(v[8 * h + 3]) << 16);
      o.z = (uint32_t)f2bf(v[8 * h + 4]) | ((uint32_t)f2bf(v[8 * h + 5]) << 16);
      o.w = (uint32_t)f2bf(v[8 * h + 6]) | ((uint32_t)f2bf(v[8 * h + 7]) << 16);
      *reinterpret_cast<uint4*>(static_cast<uint16_t*>(ep.out) + base + 8 * h) = o;
    }
  }
}

// ------------------------------------------------------------------ tiled

struct RowInfo {
  int b, ih0, iw0;   // conv: sample and top-left input corner; rows: b = m
  bool valid;
  size_t base;       // X_CONV64: element offset of (b, ih0, iw0, 0)
};

template <int MODE>
__device__ __forceinline__ RowInfo row_info(const GemmArgs& a, int m) {
  RowInfo ri;
  ri.valid = m < a.M;
  if (MODE == X_ROWS) {
    ri.b = m; ri.ih0 = 0; ri.iw0 = 0;
  } else {
    const int mm = ri.valid ? m : 0;
    const int hw = a.Ho * a.Wo;
    ri.b = mm / hw;
    const int rem = mm - ri.b * hw;
    const int oh = rem / a.Wo, ow = rem - (rem / a.Wo) * a.Wo;
    ri.ih0 = oh * a.stride - a.pad;
    ri.iw0 = ow * a.stride - a.pad;
    ri.base = (((size_t)ri.b * a.H + ri.ih0) * a.W + ri.iw0) * (size_t)a.C;
  }
  return ri;
}

// k-stage position of an X_CONV64 contraction: filter tap (kh, kw) and channel offset c0,
// identical for every thread of the workgroup
struct TapPos {
  int kh, kw, c0;
  __device__ void init(const GemmArgs& a, int k0) {
    const int tap = k0 / a.C;
    c0 = k0 - tap * a.C;
    kh = tap / a.KW;
    kw = tap - kh * a.KW;
  }
};

// 16 zero bytes in device memory: the blocked-weight loader (not read through buffer loads)
// reads them for an operand outside the matrix, so invalid data is zero as loaded. (Zeroing it after the load
// instead, when stored to LDS, made the compiler compute every ring slot's masks at the
// top of the main loop, and so wait there for every load in flight, including those just
// issued for later stages: a ring of any depth then hid one stage of latency.)
__device__ uint4 g_zero16[1];

__device__ __forceinline__ uint4 load_or_zero(const uint16_t* p, bool ok) {
  return *(ok ? reinterpret_cast<const uint4*>(p) : static_cast<const uint4*>(g_zero16));
}

// Buffer loads of a row-major operand: one buffer resource per matrix (base, size in bytes
// < 2^31), a 32-bit byte offset per load; an offset at or beyond the size reads zero, so an
// invalid operand costs an offset select and no address arithmetic in 64 bits.
constexpr uint32_t kOffNone = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// weights in 16 x 128 blocks (N % 16 == 0, K % 128 == 0): element (n, k) of an 8-run
__device__ __forceinline__ uint4 load_w8_packed(const GemmArgs& a, int n, int k) {
  const bool ok = n < a.N && k < a.K;
  const int nn = ok ? n : 0, kk = ok ? k : 0;
  const size_t off = ((((size_t)(nn >> 4) * (a.K >> 7) + (kk >> 7)) * 4 + ((kk >> 5) & 3)) * 512) +
                     ((((kk >> 3) & 3) << 4) + (nn & 15)) * 8;
  return load_or_zero(a.w + off, ok);
}

// One BN x BM output tile over the k-stages [s0, s0 + n) of this split (blockIdx.z). The
// global loads of a stage are issued D stages before its multiplications, into a ring of D
// register sets, so D memory round trips overlap (the tiles are small and the contractions
// short, so latency, not bandwidth, bounds these kernels); LDS is double-buffered, one
// barrier per stage. Invalid operand data (outside the matrix or the image) is loaded from a
// zero block, so a stage's LDS store waits only for that stage's loads. With a.splits > 1
// every split stores its fp32 partial to a.partials and k_split_reduce (the next launch on
// the stream) sums the partials in split order, which is fixed, so results are
// bit-reproducible.
// WGN x WGM waves (64 WGN WGM threads) share a tile, each owning a (BN / WGN) x (BM / WGM)
// block of it. 64 x 64 tiles of 2 x 2 waves are capped at 128 VGPRs, so four workgroups (16
// waves) fit a CU as the LDS allows, instead of two at the uncapped register count (the
// element-gather loader would spill under the cap and keeps it off); 8-wave tiles are capped
// the same way for two workgroups per CU.
template <int BN, int BM, int MODE>
constexpr int gemm_min_waves_per_simd(int nt) {
  return (nt == 256 && BN == 64 && BM == 64) ? 4 : nt == 512 ? 4 : 1;
}

// EPF (no k split, a bf16 or no residual, N a multiple of BN): each thread's epilogue inputs
// (16 bias values and 16 residuals of its output row run) are loaded with the first stages'
// operands instead of after the main loop, so that their memory round trip overlaps the
// operands' rather than following the multiplications.
template <int BN, int BM, int BK, int MODE, bool WVEC, bool PK, int D, int WGN = 2, int WGM = 2, bool EPF = false>
__global__ __launch_bounds__(64 * WGN * WGM, (gemm_min_waves_per_simd<BN, BM, MODE>(64 * WGN * WGM)))
void k_gemm(GemmArgs a) {
  constexpr int NT = 64 * WGN * WGM;            // threads
  // LDS row stride of the operand tiles: 80 bf16 (160 B). With 72 (144 B) the 16-byte
  // fragment reads and stores conflicted on banks (rocprofv3 SQ_LDS_BANK_CONFLICT: 1.18 M
  // cycles per BERT-base FFN1 launch at batch 8, 2.5 per LDS instruction); 80 measured zero
  // conflicts (88 and 104 did not help), 4.5% off BERT-base's warm forward
  constexpr int LDK = BK + 16;
  constexpr int KV = BK / 8;                    // 16-byte vectors per row and stage
  constexpr int RSTEP = NT / KV;                // rows covered by one pass of all threads
  constexpr int VA = BN / RSTEP, VB = BM / RSTEP;
  constexpr int NB = BN / WGN / 16, MB = BM / WGM / 16;   // 16 x 16 blocks per wave
  static_assert(VA >= 1 && VB >= 1 && BN % RSTEP == 0 && BM % RSTEP == 0 && NB >= 1 && MB >= 1 &&
                    BK % 32 == 0 && D >= 2 && D % 2 == 0, "tile shape");
  static_assert(MODE != X_CONV64 || BK == 64, "X_CONV64 steps one 64-deep stage per tap position");
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * (BN + BM) * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave % WGN, wm = wave / WGN;
  const int n_base = blockIdx.x * BN, m_base = blockIdx.y * BM;
  const int row0 = tid / KV, kq = (tid % KV) * 8;

  RowInfo ri[VB];
#pragma unroll
  for (int p = 0; p < VB; ++p) ri[p] = row_info<MODE>(a, m_base + row0 + RSTEP * p);

  f32x4 acc[NB][MB];
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < MB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nst = (a.K + BK - 1) / BK;
  const int s0 = blockIdx.z * a.kst;
  const int n = min(s0 + a.kst, nst) - s0;      // stages of this split (>= 1: no empty split)
  uint4 ra[D][VA], rb[D][VB];
  // row-major operands through buffer loads: per-thread byte offsets of k = 0
  // (X_CONV64: the input image, offsets of each row's top-left tap, wrapping modulo 2^32 where
  // the window starts in the padding; a valid tap brings them back inside the image)
  constexpr bool BUFW = WVEC && !PK, BUFX = MODE == X_ROWS, BUFC = MODE == X_CONV64;
  const __amdgpu_buffer_rsrc_t rw = buffer_of(a.w, BUFW ? (uint32_t)((size_t)a.N * a.K * 2) : 0u);
  const uint32_t xbytes = BUFX ? (uint32_t)((size_t)a.M * a.K * 2)
                          : BUFC ? (uint32_t)((size_t)(a.M / (a.Ho * a.Wo)) * a.H * a.W * a.C * 2) : 0u;
  const __amdgpu_buffer_rsrc_t rx = buffer_of(a.x, xbytes);
  uint32_t offw[VA], offx[VB];
  if constexpr (BUFW) {
#pragma unroll
    for (int p = 0; p < VA; ++p) {
      const int nn = n_base + row0 + RSTEP * p;
      offw[p] = nn < a.N ? (uint32_t)(((size_t)nn * a.K + kq) * 2) : kOffNone;
    }
  }
  if constexpr (BUFX) {
#pragma unroll
    for (int p = 0; p < VB; ++p) offx[p] = ri[p].valid ? (uint32_t)(((size_t)ri[p].b * a.K + kq) * 2) : kOffNone;
  }
  if constexpr (BUFC) {
#pragma unroll
    for (int p = 0; p < VB; ++p) offx[p] = (uint32_t)((ri[p].base + kq) * 2);
  }
  auto load = [&](int s, uint4 (&A)[VA], uint4 (&Bv)[VB]) {
    const int k = s * BK + kq;
    const bool kin = k < a.K;
    if constexpr (BUFW) {
#pragma unroll
      for (int p = 0; p < VA; ++p) A[p] = buffer_load16(rw, kin ? offw[p] + (uint32_t)(s * BK * 2) : kOffNone);
    } else {
      static_assert(PK && WVEC, "weights: row-major (buffer loads) or blocked");
#pragma unroll
      for (int p = 0; p < VA; ++p) A[p] = load_w8_packed(a, n_base + row0 + RSTEP * p, k);
    }
    if constexpr (BUFX) {
#pragma unroll
      for (int p = 0; p < VB; ++p) Bv[p] = buffer_load16(rx, kin ? offx[p] + (uint32_t)(s * BK * 2) : kOffNone);
    } else {
      static_assert(BUFC, "activation modes: rows or 64-channel convolution taps");
      TapPos tap;
      tap.init(a, s * BK);
      const uint32_t toff = (uint32_t)(((tap.kh * a.W + tap.kw) * a.C + tap.c0) * 2);
#pragma unroll
      for (int p = 0; p < VB; ++p) {
        const int ih = ri[p].ih0 + tap.kh, iw = ri[p].iw0 + tap.kw;
        const bool ok = ri[p].valid && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
        Bv[p] = buffer_load16(rx, ok ? offx[p] + toff : kOffNone);
      }
    }
  };
  auto store = [&](int buf, const uint4 (&A)[VA], const uint4 (&Bv)[VB]) {
    uint16_t* As = lds + buf * (BN + BM) * LDK;
    uint16_t* Bs = As + BN * LDK;
#pragma unroll
    for (int p = 0; p < VA; ++p) *reinterpret_cast<uint4*>(&As[(row0 + RSTEP * p) * LDK + kq]) = A[p];
#pragma unroll
    for (int p = 0; p < VB; ++p) *reinterpret_cast<uint4*>(&Bs[(row0 + RSTEP * p) * LDK + kq]) = Bv[p];
  };
  auto compute = [&](int buf) {
    const uint16_t* As = lds + buf * (BN + BM) * LDK;
    const uint16_t* Bs = As + BN * LDK;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      uint4 fa[NB], fb[MB];
#pragma unroll
      for (int i = 0; i < NB; ++i)
        fa[i] = *reinterpret_cast<const uint4*>(&As[(wn * (BN / WGN) + i * 16 + (lane & 15)) * LDK + kk + ((lane >> 4) << 3)]);
#pragma unroll
      for (int j = 0; j < MB; ++j)
        fb[j] = *reinterpret_cast<const uint4*>(&Bs[(wm * (BM / WGM) + j * 16 + (lane & 15)) * LDK + kk + ((lane >> 4) << 3)]);
#pragma unroll
      for (int i = 0; i < NB; ++i)
#pragma unroll
        for (int j = 0; j < MB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(fa[i]), as_bf16x8(fb[j]), acc[i][j], 0, 0, 0);
    }
  };

  // prologue: stages 0 .. D-1 (relative) into ring slots 0 .. D-1, stage 0 into LDS buffer 0,
  // then stage D into the freed slot 0
#pragma unroll
  for (int i = 0; i < D; ++i)
    if (i < n) load(s0 + i, ra[i], rb[i]);
  // the epilogue's inputs of this thread's output run (EPF); an absent bias or residual is a
  // buffer of no bytes, which reads zero, so no branch separates these loads
  constexpr int TPR = BN / 16, RPI = NT / TPR;
  static_assert(!EPF || (BM <= RPI && MODE == X_ROWS), "EPF: one output row per thread, row-major operands");
  uint4 pre_b[2], pre_r[2];
  if constexpr (EPF) {
    const int ml = tid / TPR, m = m_base + ml, n0 = n_base + (tid % TPR) * 16;
    const __amdgpu_buffer_rsrc_t rbias = buffer_of(a.ep.bias, a.ep.bias ? (uint32_t)(a.N * 2) : 0u);
    const __amdgpu_buffer_rsrc_t rres =
        buffer_of(a.ep.res, a.ep.res ? (uint32_t)((size_t)a.M * a.N * 2) : 0u);
    const uint32_t ro = (ml < BM && m < a.M) ? (uint32_t)(((size_t)m * a.N + n0) * 2) : kOffNone;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      pre_b[h] = buffer_load16(rbias, (uint32_t)(n0 * 2 + 16 * h));
      pre_r[h] = buffer_load16(rres, ro + (uint32_t)(16 * h));
    }
  }
  store(0, ra[0], rb[0]);
  if (D < n) load(s0 + D, ra[0], rb[0]);
  __syncthreads();
  // Stage j sits in ring slot j % D and LDS buffer j % 2; the loops are unrolled by D (even),
  // so every slot and buffer index is a constant. Steady state: trips whose loads are all
  // needed, with no branch around any load, so the compiler waits for exactly the stage it
  // stores. Drain: the last trips, where loads and stores beyond the split are skipped.
  int j0 = 0;
  for (; j0 + 2 * D < n; j0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int nx = (u + 1) % D;
      compute(u & 1);
      store((u + 1) & 1, ra[nx], rb[nx]);        // stage j0+u+1
      load(s0 + j0 + u + 1 + D, ra[nx], rb[nx]);  // stage j0+u+1+D
      __syncthreads();
    }
  }
  for (; j0 < n; j0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int j = j0 + u, nx = (u + 1) % D;
      if (j < n) {
        compute(u & 1);
        if (j + 1 < n) store((u + 1) & 1, ra[nx], rb[nx]);
        if (j + 1 + D < n) load(s0 + j + 1 + D, ra[nx], rb[nx]);
        __syncthreads();
      }
    }
  }

  // Output: the fp32 tile is staged in LDS (row-major [m][n], padded) so that each thread then
  // handles a 16-wide run of one row with contiguous loads and stores (the accumulator layout
  // would otherwise give 16 rows x 8 bytes per store instruction). The main loop ended with a
  // barrier, so the LDS is free.
  constexpr int TS = BN + 4;
  static_assert((size_t)BM * TS * 4 <= sizeof(lds), "output tile must fit the operand buffers");
  float* T = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      const int ml = wm * (BM / WGM) + j * 16 + (lane & 15);
      const int nl = wn * (BN / WGN) + i * 16 + ((lane >> 4) << 2);
      const f32x4 v = acc[i][j];
      *reinterpret_cast<float4*>(&T[ml * TS + nl]) = make_float4(v[0], v[1], v[2], v[3]);
    }
  __syncthreads();
  const int nl = (tid % TPR) * 16;
  const int n0 = n_base + nl;
  const bool vec = n0 + 15 < a.N && (a.N & 3) == 0;
  for (int ml = tid / TPR; ml < BM; ml += RPI) {
    const int m = m_base + ml;
    if (m >= a.M || n0 >= a.N) continue;
    float v[16];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const float4 t = *reinterpret_cast<const float4*>(&T[ml * TS + nl + 4 * h]);
      v[4 * h] = t.x; v[4 * h + 1] = t.y; v[4 * h + 2] = t.z; v[4 * h + 3] = t.w;
    }
    if (a.splits > 1) {
      // fp32 partial of this split: P[split][m][n]
      float* p = a.partials + (size_t)blockIdx.z * a.M * a.N + (size_t)m * a.N + n0;
      if (vec) {
#pragma unroll
        for (int h = 0; h < 4; ++h)
          *reinterpret_cast<float4*>(p + 4 * h) = make_float4(v[4 * h], v[4 * h + 1], v[4 * h + 2], v[4 * h + 3]);
      } else {
        for (int e = 0; e < 16 && n0 + e < a.N; ++e) p[e] = v[e];
      }
    } else if constexpr (EPF) {
      store_row16_pre(a, m, n0, v, pre_b, pre_r);
    } else {
      store_row16(a, m, n0, v);
    }
  }
}

// ------------------------------------------------------------------ few input channels

// Convolutions whose input has at most 4 channels (the ResNet stem: 7 x 7, stride 2,
// 3 channels), where an im2col row is not made of 16-byte runs. A workgroup owns all
// (<= 64) output channels and SC_W consecutive output pixels of `rows` consecutive output
// rows of one sample. Its loads are issued together before any LDS store, so it waits for
// memory once: the weights as 16-byte loads of the flat [N][K] array (re-laid out in LDS
// with rows zero-padded to a multiple of 32), and every input row the windows of its output
// rows touch (zero outside the image). Wave w multiplies the 16 pixels 16w .. 16w+15 of each
// output row against every output channel: the activation operand is gathered element by
// element from the staged rows (k = (kh * KW + kw) * C + c, so a k-run inside one filter row
// is a run of a staged input row), the weight operand read as 16-byte vectors.
constexpr int SC_W = 64, SC_MAXC = 4, SC_MAXK = 7, SC_MAXS = 2, SC_MAXR = 8;
constexpr int SC_KP = ((SC_MAXK * SC_MAXK * SC_MAXC + 31) / 32) * 32;   // 224
constexpr int SC_KS = SC_KP + 8;                                        // weight row stride in LDS
constexpr int SC_RL = ((SC_W - 1) * SC_MAXS + SC_MAXK) * SC_MAXC;       // longest staged input row
constexpr int SC_MAXIN = (SC_MAXR - 1) * SC_MAXS + SC_MAXK;             // input rows of SC_MAXR output rows
constexpr int SC_PER = (SC_RL + 255) / 256;                             // staged elements per thread and row
constexpr int SC_WV = (64 * SC_MAXK * SC_MAXK * SC_MAXC * 2 / 16 + 255) / 256;  // 16-byte weight loads per thread
// the staged input rows, or the flat weights (with the tail of their last 16-byte vector) on their way to wl
constexpr int SC_RLV = (SC_MAXC * 2 + SC_RL + 7) / 8 * 8;   // staged row stride of the vector path (below)
constexpr int SC_XL = SC_MAXIN * SC_RLV > 64 * SC_MAXK * SC_MAXK * SC_MAXC + 8 ? SC_MAXIN * SC_RLV
                                                                             : 64 * SC_MAXK * SC_MAXK * SC_MAXC + 8;

// IN: input rows staged at most (SC_MAXK for one output row per workgroup, SC_MAXIN for up to
// SC_MAXR), so that a workgroup of one output row computes no addresses for rows it never loads.
// VX: image rows of a multiple of 8 elements from a 16-byte aligned image are staged as whole
// 16-byte vectors (the window's first element then sits `sh` elements into the staged row;
// vectors outside the image read as zero, and the image's edges fall on vector boundaries), so
// that staging costs a few vector loads per thread instead of element loads with their
// addressing; otherwise element by element.
template <int C, int IN, bool VX>
__global__ __launch_bounds__(256) void k_conv_smallc(GemmArgs a, int rows) {
  __shared__ __align__(16) uint16_t wl[64 * SC_KS];
  __shared__ __align__(16) uint16_t xl[SC_XL];
  __shared__ __align__(16) int koff[SC_KP];   // staged-row offset of window element k, -1 beyond K
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int KW = a.KW, K = a.K, KWC = KW * C, KH = K / KWC;
  const int KP = (K + 31) & ~31;
  const int ow0 = blockIdx.x * SC_W, b = blockIdx.z;
  const int rl = ((SC_W - 1) * a.stride + KW) * C;
  const int oh_first = blockIdx.y * rows;
  const int nrows = min(rows, a.Ho - oh_first);          // >= 1: the grid covers Ho exactly
  const int nin = (nrows - 1) * a.stride + KH;            // input rows staged
  const int ih_first = oh_first * a.stride - a.pad, iw0 = ow0 * a.stride - a.pad;
  // vector path: staged row r holds image-row elements from vector vfirst on, so the window's
  // element j sits at sh + j; element path: at j
  const int vfirst = (iw0 * C) >> 3;                      // floor division (iw0 may be negative)
  const int sh = VX ? iw0 * C - vfirst * 8 : 0;
  const int rs = VX ? (sh + rl + 7) & ~7 : rl;            // staged row stride
  const int nvec = rs >> 3;
  for (int k = tid; k < KP; k += 256) {
    const int kh = k / KWC;
    koff[k] = k < K ? kh * rs + (k - kh * KWC) : -1;
  }
  // every global load first: the flat weights, then the staged input rows
  const int nw = a.N * K;                         // weight elements; the array starts 16-byte aligned
  const int nv = (nw * 2 + 15) / 16;
  uint4 wv[SC_WV];
#pragma unroll
  for (int u = 0; u < SC_WV; ++u) {
    const int i = u * 256 + tid;
    // the last vector may extend past the array end; it stays inside the 256-byte
    // aligned allocation unit of the weight tensor
    wv[u] = i < nv ? reinterpret_cast<const uint4*>(a.w)[i] : make_uint4(0, 0, 0, 0);
  }
  static_assert(IN <= SC_MAXIN, "staged rows");
  static_assert(SC_RLV / 8 <= 128, "two vectors per lane cover a staged row");
  constexpr int XE = VX ? 1 : IN, XU = VX ? 1 : SC_PER;       // element path: rows x elements per thread
  constexpr int XR = VX ? (IN + 3) / 4 : 1;                   // vector path: rows per wave (row r = wave + 4 i)
  uint16_t xv[XE][XU];
  uint4 xq[XR][2];
  if constexpr (VX) {
    const int rowv = (a.W * C) >> 3;                        // vectors per image row
#pragma unroll
    for (int i = 0; i < XR; ++i) {
      const int r = wave + 4 * i, ih = ih_first + r;
      const bool hin = r < nin && ih >= 0 && ih < a.H;
      const uint4* xrow = reinterpret_cast<const uint4*>(a.x + ((size_t)b * a.H + (hin ? ih : 0)) * a.W * C);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int vi = lane + 64 * h, gv = vfirst + vi;
        xq[i][h] = (hin && vi < nvec && gv >= 0 && gv < rowv) ? xrow[gv] : make_uint4(0, 0, 0, 0);
      }
    }
  } else {
#pragma unroll
    for (int r = 0; r < IN; ++r) {
      const int ih = ih_first + r;
      const bool hin = r < nin && ih >= 0 && ih < a.H;
      const uint16_t* xrow = a.x + ((size_t)b * a.H + (hin ? ih : 0)) * a.W * C;
#pragma unroll
      for (int u = 0; u < SC_PER; ++u) {
        const int j = u * 256 + tid;
        const int col = j / C, iw = iw0 + col;
        xv[r][u] = (hin && j < rl && iw >= 0 && iw < a.W) ? xrow[(size_t)iw * C + (j - col * C)] : (uint16_t)0;
      }
    }
  }
  // the flat weights through xl, then padded rows into wl (four threads per row, every fourth
  // k: no division by the run-time row length), then the input rows into xl
#pragma unroll
  for (int u = 0; u < SC_WV; ++u) {
    const int i = u * 256 + tid;
    if (i < nv) reinterpret_cast<uint4*>(xl)[i] = wv[u];
  }
  __syncthreads();
  const int wn = tid >> 2;
  for (int k = tid & 3; k < KP; k += 4)
    wl[wn * SC_KS + k] = (wn < a.N && k < K) ? xl[wn * K + k] : (uint16_t)0;
  __syncthreads();
  if constexpr (VX) {
#pragma unroll
    for (int i = 0; i < XR; ++i) {
      const int r = wave + 4 * i;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int vi = lane + 64 * h;
        if (r < nin && vi < nvec) *reinterpret_cast<uint4*>(&xl[r * rs + vi * 8]) = xq[i][h];
      }
    }
  } else {
#pragma unroll
    for (int r = 0; r < IN; ++r)
#pragma unroll
      for (int u = 0; u < SC_PER; ++u) {
        const int j = u * 256 + tid;
        if (r < nin && j < rl) xl[r * rs + j] = xv[r][u];
      }
  }
  __syncthreads();

  const int p = wave * 16 + (lane & 15), q = lane >> 4;
  const int pofs = p * a.stride * C;
  for (int r = 0; r < nrows; ++r) {
    const int oh = oh_first + r, rbase = r * a.stride * rs + pofs + sh;
    f32x4 acc[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the same number of k-steps in every lane; element reads are unconditional (offset
    // clamped to 0) and masked afterwards
    for (int ks = 0; ks < KP / 32; ++ks) {
      const int k0 = ks * 32 + q * 8;
      const int4 o0 = *reinterpret_cast<const int4*>(&koff[k0]);
      const int4 o1 = *reinterpret_cast<const int4*>(&koff[k0 + 4]);
      const int o[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
      uint32_t bw[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t v = xl[(o[e] < 0 ? 0 : o[e]) + rbase];
        bw[e >> 1] |= (o[e] < 0 ? 0u : v) << (16 * (e & 1));
      }
      const uint4 bv = make_uint4(bw[0], bw[1], bw[2], bw[3]);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const uint4 av = *reinterpret_cast<const uint4*>(&wl[(16 * g + (lane & 15)) * SC_KS + k0]);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av), as_bf16x8(bv), acc[g], 0, 0, 0);
      }
    }
    if (ow0 + p < a.Wo) {
      const int m = ((b * a.Ho) + oh) * a.Wo + ow0 + p;
#pragma unroll
      for (int g = 0; g < 4; ++g)
        if (16 * g < a.N) store_row4(a, m, 16 * g + 4 * q, acc[g]);
    }
  }
}

// y = epilogue(sum over splits z = 0, 1, ... of P[z]) for four consecutive outputs per thread.
// A thread fetches the epilogue's inputs and ZG partials before it adds any (a launch that
// waited for each partial in turn spent ~5 us on a few MB: one memory round trip per split);
// the additions keep split order, so results are the same as summing one split at a time.
template <int ZG, int RES>
__global__ __launch_bounds__(256) void k_split_reduce(GemmArgs a) {
  const long q = (long)blockIdx.x * 256 + threadIdx.x;       // index of a group of 4 outputs
  const int groups_per_row = (a.N + 3) >> 2;
  const long total = (long)a.M * groups_per_row;
  if (q >= total) return;
  const int m = (int)(q / groups_per_row), n0 = (int)(q - (long)m * groups_per_row) * 4;
  const size_t plane = (size_t)a.M * a.N, base = (size_t)m * a.N + n0;
  f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
  if (n0 + 3 < a.N && (a.N & 3) == 0) {
    const Ep4In in = ep4_fetch<RES>(a.ep, base, n0);
    for (int z0 = 0; z0 < a.splits; z0 += ZG) {
      float4 t[ZG];
#pragma unroll
      for (int u = 0; u < ZG; ++u)
        if (z0 + u < a.splits) t[u] = *reinterpret_cast<const float4*>(a.partials + (z0 + u) * plane + base);
#pragma unroll
      for (int u = 0; u < ZG; ++u)
        if (z0 + u < a.splits) sum += f32x4{t[u].x, t[u].y, t[u].z, t[u].w};
    }
    float v[4] = {sum[0], sum[1], sum[2], sum[3]};
    ep4_apply<RES>(a.ep, in, v);
    ep4_store(a.ep, base, v);
    return;
  }
  for (int z = 0; z < a.splits; ++z) {
    const float* p = a.partials + z * plane + base;
    for (int e = 0; e < 4 && n0 + e < a.N; ++e) sum[e] += p[e];
  }
  store_row4(a, m, n0, sum);
}

template <int RES>
void launch_split_reduce_res(const GemmArgs& a, dim3 grid, dim3 block, hipStream_t s) {
  switch (split_group(a.splits)) {
    case 2: (void)launch((k_split_reduce<2, RES>), grid, block, 0, s, a); break;
    case 4: (void)launch((k_split_reduce<4, RES>), grid, block, 0, s, a); break;
    default: (void)launch((k_split_reduce<8, RES>), grid, block, 0, s, a); break;
  }
}

void launch_split_reduce(const GemmArgs& a, dim3 grid, dim3 block, hipStream_t s) {
  switch (res_kind(a.ep)) {
    case 0: launch_split_reduce_res<0>(a, grid, block, s); break;
    case 1: launch_split_reduce_res<1>(a, grid, block, s); break;
    default: launch_split_reduce_res<2>(a, grid, block, s); break;
  }
}

// After the contraction: the reduction of a k split (fused with the epilogue's row
// LayerNorm when the width allows), then the LayerNorm of an fp32 result if one is asked for
// and not yet done.
hipError_t finish(const GemmArgs& a, hipStream_t s) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.splits > 1) {
    if (a.ep.ln_g && split_reduce_ln_fits(a.N)) return split_reduce_ln(a, s);
    const long groups = (long)a.M * ((a.N + 3) / 4);
    const dim3 grid((unsigned)((groups + 255) / 256)), block(256);
    launch_split_reduce(a, grid, block, s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.ep.ln_g)
    return layernorm(static_cast<const float*>(a.ep.out), a.M, a.N, a.ep.ln_g, a.ep.ln_b, a.ep.ln_eps, a.ep.ln_out,
                     a.ep.ln_out_f32, s);
  return hipSuccess;
}

template <int BN, int BM, int BK, int MODE, bool WVEC, int D, int WGN = 2, int WGM = 2>
hipError_t launch_tiled(GemmArgs a, int splits, const Split& sp, hipStream_t s) {
  const int tn = (a.N + BN - 1) / BN, tm = (a.M + BM - 1) / BM;
  const int nst = (a.K + BK - 1) / BK;
  a.kst = (nst + splits - 1) / splits;
  a.splits = (nst + a.kst - 1) / a.kst;        // no empty split
  a.partials = sp.partials;
  dim3 grid(tn, tm, a.splits);
  if constexpr (MODE == X_ROWS) {
    if (a.ep.w_packed) {
      (void)launch((k_gemm<BN, BM, BK, MODE, WVEC, true, D, WGN, WGM>), grid, dim3(64 * WGN * WGM), 0, s, a);
      return finish(a, s);
    }
  }
  // an unsplit row-major contraction fetches its epilogue inputs with its first operands
  // (EPF). Against fetching them after the main loop, whole warm forwards (A/B on one machine):
  // ResNet-50 -3 to -4% at batch 1 and 8, BERT-base -3% at batch 1, -1% at batch 8; for
  // the convolution taps as well, no further change (-0.5% to +0.3%), so those do not.
  constexpr bool kEpfTile = MODE == X_ROWS && BM <= 64 * WGN * WGM / (BN / 16);
  if constexpr (kEpfTile) {
    if (a.splits == 1 && !(a.ep.res && a.ep.res_f32) && a.N % BN == 0 && a.N % 16 == 0 &&
        (size_t)a.M * a.N * 2 < (1u << 31)) {
      (void)launch((k_gemm<BN, BM, BK, MODE, WVEC, false, D, WGN, WGM, true>), grid, dim3(64 * WGN * WGM), 0, s, a);
      return finish(a, s);
    }
  }
  (void)launch((k_gemm<BN, BM, BK, MODE, WVEC, false, D, WGN, WGM>), grid, dim3(64 * WGN * WGM), 0, s, a);
  return finish(a, s);
}

// Tile shape and k split of a tiled contraction. Measured on MI355X over every contraction of
// ResNet-50 and BERT-base at batch 1 and 8 (each shape timed under graph replay with 20 tile
// shapes and 6 split counts): the fastest launches fill the 256 CUs with about one to three
// workgroups each rather than many small ones or a few large ones; a k split pays only for
// contractions deeper than about 12 stages whose tiles alone leave CUs idle, since its
// reduction is a launch of its own (about 2-3 us); tiles larger than 64 x 64 and 128-deep
// stages were never faster at these sizes (in whole forward passes, 128-deep stages for the
// smaller tiles: -1% at batch 1, +3% at batch 8; a ring of four stages: +3-6%). So: the largest of 64 x 64, 64 x 32, 32 x 64 and
// 32 x 32 (output features x rows) whose grid has at least 256 tiles (else 32 x 32); then
// splits while a split keeps more than 12 stages, the grid stays within 768 workgroups, each
// split keeps at least 4 stages and the fp32 partials fit the scratch. A row LayerNorm then
// rides on the split reduction, or takes a launch of its own. 128 x 128 tiles for grids of
// well over a few such tiles per CU.
struct TilePlan {
  int bn, bm, splits;
};

TilePlan plan_tiles(const GemmArgs& a, const Split& sp) {
  auto tiles = [&](int bn, int bm) { return (long)((a.N + bn - 1) / bn) * ((a.M + bm - 1) / bm); };
  if (tiles(128, 128) >= 1024) return {128, 128, 1};
  static constexpr int kShapes[4][2] = {{64, 64}, {64, 32}, {32, 64}, {32, 32}};
  TilePlan p{32, 32, 1};
  for (const auto& t : kShapes)
    if (tiles(t[0], t[1]) >= 256) {
      p.bn = t[0];
      p.bm = t[1];
      break;
    }
  const long nt = tiles(p.bn, p.bm);
  const int nst = (a.K + 63) / 64;
  const size_t per_split = (size_t)a.M * a.N * 4;
  if (sp.partials)
    while (nst > 12 * p.splits && nt * (p.splits + 1) <= 768 && nst >= 4 * (p.splits + 1) &&
           per_split * (p.splits + 1) <= sp.partial_bytes)
      ++p.splits;
  return p;
}

template <int MODE, bool WVEC>
hipError_t pick_tiled(const GemmArgs& a, const Split& sp, hipStream_t s) {
  const TilePlan p = plan_tiles(a, sp);
  if (p.bn == 128) return launch_tiled<128, 128, 64, MODE, WVEC, 2>(a, p.splits, sp, s);
  if (p.bn == 64 && p.bm == 64) return launch_tiled<64, 64, 64, MODE, WVEC, 2>(a, p.splits, sp, s);
  if (p.bn == 64) return launch_tiled<64, 32, 64, MODE, WVEC, 2>(a, p.splits, sp, s);
  if (p.bm == 64) return launch_tiled<32, 64, 64, MODE, WVEC, 2>(a, p.splits, sp, s);
  return launch_tiled<32, 32, 64, MODE, WVEC, 2>(a, p.splits, sp, s);
}

bool ep_ok(const Epilogue& ep) {
  if (ep.ln_g && (!ep.ln_b || !ep.ln_out || !ep.out_f32)) return false;
  return ep.out != nullptr && ep.act >= 0 && ep.act <= 2;
}

}  // namespace

hipError_t linear_bf16(const uint16_t* x, int M, int K, const uint16_t* w, int N, const Epilogue& ep,
                       const Split& sp, hipStream_t s) {
  if (!x || !w || M < 1 || N < 1 || K < 8 || (K & 7) || !ep_ok(ep)) return hipErrorInvalidValue;
  if (ep.w_packed && ((N & 15) || (K & 127))) return hipErrorInvalidValue;
  GemmArgs a{};
  a.x = x; a.w = w; a.M = M; a.N = N; a.K = K; a.ep = ep;
  if (M <= 32) {
    a.splits = 1;
    hipError_t e = launch_skinny(a, s);
    return e == hipSuccess ? finish(a, s) : e;
  }
  // the tiled kernel addresses x and w through 32-bit buffer offsets
  if ((size_t)M * K * 2 >= (1u << 31) || (size_t)N * K * 2 >= (1u << 31)) return hipErrorInvalidValue;
  return pick_tiled<X_ROWS, true>(a, sp, s);
}

hipError_t conv_bf16(const uint16_t* x, int B, int H, int W, int C, const uint16_t* w, int O, int KH, int KW,
                     int stride, int pad, const Epilogue& ep, const Split& sp, hipStream_t s) {
  if (!x || !w || B < 1 || H < 1 || W < 1 || C < 1 || O < 1 || KH < 1 || KW < 1 || stride < 1 || pad < 0 ||
      !ep_ok(ep) || ep.ln_g)
    return hipErrorInvalidValue;
  const int Ho = (H + 2 * pad - KH) / stride + 1, Wo = (W + 2 * pad - KW) / stride + 1;
  if (Ho < 1 || Wo < 1) return hipErrorInvalidValue;
  if (KH == 1 && KW == 1 && stride == 1 && pad == 0 && (C & 7) == 0)
    return linear_bf16(x, B * H * W, C, w, O, ep, sp, s);
  GemmArgs a{};
  a.x = x; a.w = w; a.M = B * Ho * Wo; a.N = O; a.K = KH * KW * C;
  a.H = H; a.W = W; a.C = C; a.KW = KW; a.stride = stride; a.pad = pad; a.Ho = Ho; a.Wo = Wo;
  a.ep = ep;
  a.ep.w_packed = 0;
  if ((size_t)B * H * W * C * 2 >= (1u << 31) || (size_t)O * KH * KW * C * 2 >= (1u << 31))
    return hipErrorInvalidValue;   // the tiled kernel addresses x and w through 32-bit buffer offsets
  if (C <= SC_MAXC && KH <= SC_MAXK && KW <= SC_MAXK && stride <= SC_MAXS && O <= 64 && (O & 15) == 0 &&
      a.K <= SC_KP) {
    // enough workgroups to fill the chip, each reusing its staged weights over `rows` rows
    const int segs = (Wo + SC_W - 1) / SC_W;
    const int rows = max(1, min(SC_MAXR, segs * Ho * B / 448));
    dim3 grid(segs, (Ho + rows - 1) / rows, B);
    auto go = [&](auto kern) { (void)launch(kern, grid, dim3(256), 0, s, a, rows); };
    const bool one = rows == 1, vx = (W * C) % 8 == 0 && ((uintptr_t)x & 15) == 0;
    // the vector path for the channel counts of network stems (RGB, RGBA), the element path
    // otherwise
    if (vx && C == 3) one ? go(k_conv_smallc<3, SC_MAXK, true>) : go(k_conv_smallc<3, SC_MAXIN, true>);
    else if (vx && C == 4) one ? go(k_conv_smallc<4, SC_MAXK, true>) : go(k_conv_smallc<4, SC_MAXIN, true>);
    else switch (C) {
      case 1: one ? go(k_conv_smallc<1, SC_MAXK, false>) : go(k_conv_smallc<1, SC_MAXIN, false>); break;
      case 2: one ? go(k_conv_smallc<2, SC_MAXK, false>) : go(k_conv_smallc<2, SC_MAXIN, false>); break;
      case 3: one ? go(k_conv_smallc<3, SC_MAXK, false>) : go(k_conv_smallc<3, SC_MAXIN, false>); break;
      default: one ? go(k_conv_smallc<4, SC_MAXK, false>) : go(k_conv_smallc<4, SC_MAXIN, false>); break;
    }
    return hipGetLastError();
  }
  if ((C & 63) == 0) return pick_tiled<X_CONV64, true>(a, sp, s);
  return hipErrorInvalidValue;
}

}  // namespace k
}  // namespace tp
