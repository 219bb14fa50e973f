// Host-side launchers of the gfx950 kernels. Every launcher checks the shape
// preconditions its kernel relies on and returns hipErrorInvalidValue instead of
// launching when they do not hold.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <vector>

namespace tp {
namespace k {

enum { ACT_NONE = 0, ACT_RELU = 1, ACT_GELU = 2 };

// One kernel launch as the launchers record it while a forward pass is being captured into
// a graph: the kernel, its launch shape, a copy of every argument (each at its own 8-byte
// aligned offset in `bytes`) and the offsets in `bytes` of the device pointers the arguments
// hold (a pointer argument itself; the pointer fields of a contraction's argument block). The
// runtime uses it to repoint an instantiated graph at other input and output buffers.
struct LaunchRecord {
  const void* func = nullptr;
  dim3 grid, block;
  unsigned shmem = 0;
  std::vector<uint32_t> arg_at;    // offset of each argument in `bytes`
  std::vector<uint8_t> bytes;
  std::vector<uint32_t> ptr_at;    // offsets of pointer values in `bytes`
};

// When set (by the runtime, on the capturing thread), every launcher appends its launches.
extern thread_local std::vector<LaunchRecord>* launch_log;

// Fused epilogue of the bf16 contractions: v = acc + bias[n] (+ res[m][n]); v = act(v);
// out[m][n] = v stored as bf16 or fp32. Row stride of res and out is N.
struct Epilogue {
  const uint16_t* bias = nullptr;   // bf16 [N], may be null
  const void* res = nullptr;        // [M][N], may be null
  int res_f32 = 0;                  // res dtype: 0 bf16, 1 fp32
  int act = 0;                      // ACT_*
  void* out = nullptr;
  int out_f32 = 0;                  // out dtype: 0 bf16, 1 fp32
  int w_packed = 0;                 // weights in 16 x 128 blocks (N % 16 == 0, K % 128 == 0)
  // optional row LayerNorm of the (fp32) result, written to ln_out (bf16 or fp32): then
  // `out` must be fp32 [M][N] scratch, which a contraction split over k does not touch (the
  // reduction normalises in registers when 256 <= N <= 1024 and N % 256 == 0)
  const uint16_t* ln_g = nullptr;
  const uint16_t* ln_b = nullptr;
  float ln_eps = 0.f;
  void* ln_out = nullptr;
  int ln_out_f32 = 0;
};

// Scratch for splitting a contraction over k into fp32 partials (null disables splitting).
struct Split {
  float* partials = nullptr;
  size_t partial_bytes = 0;
};

// y[M][N] = x[M][K] * w[N][K]^T with the epilogue; bf16 in, fp32 accumulate. K % 8 == 0;
// for M > 32, x and w each below 2 GiB (M K 2 and N K 2 bytes < 2^31).
hipError_t linear_bf16(const uint16_t* x, int M, int K, const uint16_t* w, int N, const Epilogue& ep,
                       const Split& sp, hipStream_t s);

// Implicit-GEMM convolution: x NHWC [B][H][W][C] bf16, w OHWI [O][KH][KW][C] bf16,
// y NHWC [B][Ho][Wo][O] via the epilogue (M = B*Ho*Wo rows of N = O). C % 64 == 0 (implicit
// GEMM), or C <= 4 with O <= 64, O % 16 == 0 and a filter of at most 7 x 7, stride <= 2 (the
// small-channel kernel of a network's stem); other channel counts return
// hipErrorInvalidValue. x and w each below 2 GiB; a 1x1 stride-1 convolution is a linear
// layer and has its size limits too.
hipError_t conv_bf16(const uint16_t* x, int B, int H, int W, int C, const uint16_t* w, int O, int KH, int KW,
                     int stride, int pad, const Epilogue& ep, const Split& sp, hipStream_t s);

// fp32 linear: y[M][N] = act(x[M][K] * w[N][K]^T + bias). K % 4 == 0.
hipError_t linear_f32(const float* x, int M, int K, const float* w, int N, const float* bias, int act, float* y,
                      hipStream_t s);

// Row LayerNorm of fp32 x[M][D] (population variance) with bf16 gamma/beta; out bf16 or
// fp32. D % 64 == 0, D <= 1024.
hipError_t layernorm(const float* x, int M, int D, const uint16_t* g, const uint16_t* b, float eps, void* out,
                     int out_f32, hipStream_t s);

// h[r] = LN(tok[ids[r]] + pos[r % S] + type[0]) for r < M, out bf16 [M][D]; ids are
// clamped to [0, vocab).
hipError_t embed_ln(const int32_t* ids, int M, int S, int D, int vocab, const uint16_t* tok, const uint16_t* pos,
                    const uint16_t* type, const uint16_t* g, const uint16_t* b, float eps, uint16_t* out,
                    hipStream_t s);

// Multi-head self-attention, head dim 64, no mask: qkv bf16 [B*S][3*H*64] (Q|K|V blocks,
// heads contiguous inside each) -> out bf16 [B*S][H*64]. S % 32 == 0, S <= 256.
hipError_t attention(const uint16_t* qkv, int B, int S, int H, uint16_t* out, hipStream_t s);

// 3x3 stride-2 pad-1 max-pool, NHWC bf16; C % 8 == 0.
hipError_t maxpool3s2(const uint16_t* x, int B, int H, int W, int C, uint16_t* y, hipStream_t s);

// Mean over HW positions: x [B][HW][C] -> y [B][C], bf16.
hipError_t avgpool(const uint16_t* x, int B, int HW, int C, uint16_t* y, hipStream_t s);

// Copy of `bytes` (multiple of 16) from device-visible pinned host memory to device
// memory by `wgs` workgroups of 16-byte loads.
hipError_t gather_copy(const void* src, void* dst, uint64_t bytes, int wgs, hipStream_t s);

// A single-wave kernel that sleeps for about `us` microseconds (bounded loop).
hipError_t delay(int us, hipStream_t s);

}  // namespace k
}  // namespace tp
