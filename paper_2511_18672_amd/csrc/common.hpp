// Device-side helpers shared by the gfx950 kernels of the selective-refinement
// step: the request table passed by value to every kernel, token-position
// decoding, bf16 conversion and wave64 reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sphinx.h"

namespace sphinx {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;

// Request geometry, passed by value (kernarg segment) to every kernel.
struct ReqTable {
  int32_t R;
  int32_t frames[SPHINX_MAX_REQUESTS];
  int32_t h[SPHINX_MAX_REQUESTS];
  int32_t w[SPHINX_MAX_REQUESTS];
  int32_t frame_off[SPHINX_MAX_REQUESTS + 1];
  int64_t tok_off[SPHINX_MAX_REQUESTS + 1];  // tok_off[R] = N
};

struct TokPos {
  int r, f, y, x, g;  // request, frame in request, patch row, patch column, global frame
  int64_t elem;       // NCHW element index of (c=0, py=0, px=0) of the token
  int plane;          // h*w of the request (stride between channels)
  int w;              // latent width (stride between rows)
};

__device__ __forceinline__ int find_request(const ReqTable& T, int64_t t) {
  int lo = 0, hi = T.R - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (T.tok_off[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Global frame of token t (the part of decode_token that token-major latents need).
__device__ __forceinline__ int frame_of_token(const ReqTable& T, int64_t t) {
  const int r = find_request(T, t);
  const uint32_t loc = (uint32_t)(t - T.tok_off[r]);
  const uint32_t tpf = ((uint32_t)T.h[r] >> 1) * ((uint32_t)T.w[r] >> 1);
  return T.frame_off[r] + (int)(loc / tpf);
}

__device__ __forceinline__ TokPos decode_token(const ReqTable& T, int64_t t) {
  TokPos p;
  p.r = find_request(T, t);
  const uint32_t loc = (uint32_t)(t - T.tok_off[p.r]);
  const uint32_t wp = (uint32_t)T.w[p.r] >> 1, hp = (uint32_t)T.h[p.r] >> 1;
  const uint32_t tpf = hp * wp;
  const uint32_t f = loc / tpf;
  const uint32_t rem = loc - f * tpf;
  const uint32_t y = rem / wp;
  p.f = (int)f;
  p.y = (int)y;
  p.x = (int)(rem - y * wp);
  p.g = T.frame_off[p.r] + p.f;
  p.w = T.w[p.r];
  p.plane = T.h[p.r] * T.w[p.r];
  p.elem = 16 * T.tok_off[p.r] + ((int64_t)p.f * 4) * p.plane + (int64_t)(2 * p.y) * p.w + 2 * p.x;
  return p;
}

// Workgroups are dealt to the 8 XCDs round-robin by linear id (x fastest).
// Returns the tile that linear workgroup b of `total` should compute so that
// each XCD gets one contiguous range of tiles: XCD x receives q + (x < r)
// workgroups (q = total / 8, r = total % 8), and its k-th workgroup (b = 8k + x)
// takes tile start(x) + k.  A bijection on [0, total) whatever the hardware
// does; with the round-robin dealing, tiles that share operand rows stay in
// one XCD's L2.
__device__ __forceinline__ int xcd_tile(int b, int total) {
  const int x = b & 7, k = b >> 3, q = total >> 3, r = total & 7;
  return x * q + min(x, r) + k;
}

// Direct global->LDS copy, 16 bytes per lane (global_load_lds_dwordx4): lane
// i's 16 bytes land at lds_dst + 16 i, where lds_dst must be wave-uniform.
// Issued through inline asm rather than the builtin: with the builtin in a
// loop the compiler's wait-count analysis treats every later LDS read as
// possibly aliasing a pending copy and waits for all LDS reads (lgkmcnt(0))
// before their first use.  Callers order the copies themselves: each wave
// waits for its copies (s_waitcnt vmcnt) before the barrier that publishes
// them.  The compiler's own vmcnt waits stay correct, since copies it does
// not see only make them stricter.
__device__ __forceinline__ void lds_dma16(const void* gsrc, const void* lds_dst) {
  const uint32_t m0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)lds_dst;
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gsrc), "s"(m0) : "memory", "m0");
}

// The same copy from a wave-uniform base address (an SGPR pair) plus a
// per-lane 32-bit byte offset, so that moving the source costs scalar
// arithmetic only.
__device__ __forceinline__ void lds_dma16_at(const void* sbase, uint32_t voff, const void* lds_dst) {
  const uint32_t m0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)lds_dst;
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(m0)
               : "memory", "m0");
}

__device__ __forceinline__ float bf2f(bf16 v) { return (float)v; }
__device__ __forceinline__ bf16 f2bf(float v) { return (bf16)v; }  // round to nearest even

template <typename T> __device__ __forceinline__ float load_as_f32(const T* p, int64_t i);
template <> __device__ __forceinline__ float load_as_f32<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float load_as_f32<bf16>(const bf16* p, int64_t i) { return (float)p[i]; }

template <typename T> __device__ __forceinline__ T store_from_f32(float v);
template <> __device__ __forceinline__ float store_from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 store_from_f32<bf16>(float v) { return (bf16)v; }

// Lane v of the same row (16 lanes) selected by a DPP control word.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}

// Sum over the 64 lanes of a fully active wave, in every lane (bit-identical
// in all lanes: each step adds two values in both orders' common result).
// Within a row of 16 lanes: quad permutations (lane ^ 1, lane ^ 2), then the
// half-row and row mirrors; across rows: the gfx950 row-pair and half swaps.
// No LDS round trips, unlike a shuffle butterfly.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);  // row_half_mirror: the other quad of the 8-lane half
  v += dpp_f<0x140>(v);  // row_mirror: the other half of the row
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
  return v;
}

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

// GELU, tanh form: 0.5 z (1 + tanh(u)), u = sqrt(2/pi) (z + 0.044715 z^3).
// Since 1 + tanh(u) = 2 / (1 + e^(-2u)), this is z / (1 + 2^(-2u log2 e)): one
// hardware exp2 and one reciprocal (each within about an ulp of fp32), which
// keeps the MLP epilogue cheap next to its MFMAs.  Large negative z gives
// z / inf = -0, large positive z gives z.
__device__ __forceinline__ float gelu_tanh(float z) {
  constexpr float c = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float a = z * fmaf(c * 0.044715f, z * z, c);                         // c (z + 0.044715 z^3)
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(a));
}

}  // namespace sphinx
