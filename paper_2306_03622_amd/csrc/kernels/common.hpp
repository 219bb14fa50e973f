// Shared device helpers for the gfx950 kernels: bf16 storage conversions, MFMA operand
// types and wave64 reductions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstddef>
#include <cstring>
#include <tuple>
#include <utility>

#include "kernels.hpp"

namespace tp {
namespace k {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float((uint32_t)u << 16); }

// float -> bf16 bits, round to nearest even; NaN stays NaN (quiet). Written as a select, not
// an early return: as a branch it compiled to a divergent if per conversion (exec-mask
// saves and restores around every element of an epilogue)
__device__ __forceinline__ uint16_t f2bf(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t quiet_nan = (u >> 16) | 0x40u;
  return (uint16_t)((u & 0x7fffffffu) > 0x7f800000u ? quiet_nan : rounded);
}

// erf(x) by Abramowitz and Stegun, Handbook of Mathematical Functions, formula 7.1.26:
// 1 - (a1 t + ... + a5 t^5) exp(-x^2) with t = 1 / (1 + p |x|), odd in x, absolute error at
// most 1.5e-7 (plus the hardware reciprocal's and exponential's rounding). Branch-free: the
// library erff chose between two evaluations per element, a divergent branch in every
// GELU epilogue.
__device__ __forceinline__ float erf_as7126(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.f));
  float p = fmaf(1.061405429f, t, -1.453152027f);
  p = fmaf(p, t, 1.421413741f);
  p = fmaf(p, t, -0.284496736f);
  p = fmaf(p, t, 0.254829592f);
  return copysignf(1.f - p * t * __expf(-ax * ax), x);
}

__device__ __forceinline__ float act_apply(float v, int act) {
  if (act == ACT_RELU) return v > 0.f ? v : 0.f;
  if (act == ACT_GELU) return 0.5f * v * (1.f + erf_as7126(v * 0.70710678118654752f));
  return v;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load marked non-temporal (data streamed once, not worth keeping in the caches)
__device__ __forceinline__ uint4 load_nt16(const void* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// branch-free zeroing of a loaded vector (the load itself is always in bounds)
__device__ __forceinline__ uint4 mask_u4(uint4 v, bool ok) {
  const uint32_t m = ok ? 0xffffffffu : 0u;
  return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
}

// butterfly sum over the 64 lanes of a wave in a fixed order (lanes 32 apart first, then 16,
// 8, 4, 2, 1: bit-identical across runs). The four steps inside a 16-lane row move data by
// DPP instead of through the LDS crossbar: rotating a row by 8 pairs the lanes that xor 8
// pairs; the row's values then repeat every 8 lanes, so rotating by 4 pairs values that xor 4
// pairs; the last two steps are quad permutations (LayerNorm-bound launches of BERT-base:
// warm forward -1.3% at batch 1, same bits).
template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
  return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += __shfl_xor(v, 32, 64);
  v += __shfl_xor(v, 16, 64);
  v = dpp_add<0x128>(v);        // row_ror:8
  v = dpp_add<0x124>(v);        // row_ror:4
  v = dpp_add<0x4E>(v);         // quad_perm [2,3,0,1]: xor 2
  return dpp_add<0xB1>(v);      // quad_perm [1,0,3,2]: xor 1
}

// Byte offsets of the device pointers inside a kernel argument of type T (none for values;
// the argument itself for a pointer; argument blocks specialise this).
template <typename T>
struct PtrFields {
  static void add(std::vector<uint32_t>&, uint32_t) {}
};
template <typename T>
struct PtrFields<T*> {
  static void add(std::vector<uint32_t>& v, uint32_t at) { v.push_back(at); }
};

// Launches `kern` with its arguments converted to the kernel's parameter types (the same
// call the triple-chevron form makes), and records the launch in launch_log when one is set.
template <typename... P, typename... A>
hipError_t launch(void (*kern)(P...), dim3 grid, dim3 block, unsigned shmem, hipStream_t s, A&&... a) {
  static_assert(sizeof...(P) == sizeof...(A), "argument count");
  std::tuple<P...> args{P(std::forward<A>(a))...};
  return std::apply(
      [&](auto&... v) -> hipError_t {
        void* argv[] = {static_cast<void*>(&v)...};
        if (launch_log) {
          LaunchRecord r;
          r.func = reinterpret_cast<const void*>(kern);
          r.grid = grid;
          r.block = block;
          r.shmem = shmem;
          auto put = [&](const auto& x) {
            using T = std::decay_t<decltype(x)>;
            const uint32_t at = (uint32_t)((r.bytes.size() + 7) & ~size_t(7));
            r.bytes.resize(at + sizeof(T));
            std::memcpy(r.bytes.data() + at, &x, sizeof(T));
            r.arg_at.push_back(at);
            PtrFields<T>::add(r.ptr_at, at);
          };
          (put(v), ...);
          launch_log->push_back(std::move(r));
        }
        return hipLaunchKernel(reinterpret_cast<const void*>(kern), grid, block, argv, shmem, s);
      },
      args);
}

}  // namespace k
}  // namespace tp
