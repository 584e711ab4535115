// Gather with noise injection (Alg. 1 add_noise on the selected tokens) and
// scatter/blend back into the NCHW latents (Sec. 3, Sec. 5.3: confident
// regions keep their values).
//
// One thread moves one token: its position is decoded once, its 16 values are
// eight 8-byte (channel, patch-row) pairs in the latent planes and one
// 64-byte row of x_sel ([n][16] fp32).  Neighbouring selected tokens along x
// are neighbours in memory, so a wave touches contiguous runs of each plane.
#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int kTPB = 256;

template <typename T> struct Pair;
template <> struct Pair<float> {
  static __device__ __forceinline__ float2 load(const float* p, int64_t e) {
    return *reinterpret_cast<const float2*>(p + e);
  }
  static __device__ __forceinline__ void store(float* p, int64_t e, float2 v) {
    *reinterpret_cast<float2*>(p + e) = v;
  }
};
template <> struct Pair<bf16> {
  static __device__ __forceinline__ float2 load(const bf16* p, int64_t e) {
    const bf16x2 v = *reinterpret_cast<const bf16x2*>(p + e);
    return make_float2((float)v[0], (float)v[1]);
  }
  static __device__ __forceinline__ void store(bf16* p, int64_t e, float2 v) {
    bf16x2 o;
    o[0] = (bf16)v.x;
    o[1] = (bf16)v.y;
    *reinterpret_cast<bf16x2*>(p + e) = o;
  }
};

// One thread per selected token: decode its position once, read its 8 (c, py)
// pairs of 2 values from the latent planes, write its 64-byte x_sel row as
// four 16-byte stores.
template <typename ST, typename ET>
__global__ __launch_bounds__(kTPB) void k_gather(ReqTable T, const ST* __restrict__ state, const ET* __restrict__ eps,
                                                 const int32_t* __restrict__ idx, int n, const float* __restrict__ a,
                                                 const float* __restrict__ b, float* __restrict__ x) {
  const int64_t j = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  if (j >= n) return;
  const int32_t t = idx[j];
  if (t < 0 || t >= T.tok_off[T.R]) return;  // out-of-range index: nothing is read
  const TokPos tp = decode_token(T, t);
  const float av = a[tp.g], bv = b[tp.g];
  const bool inject = eps != nullptr && bv != 0.0f;
  float v[16];
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const int64_t e = tp.elem + (int64_t)(p >> 1) * tp.plane + (int64_t)(p & 1) * tp.w;
    const float2 z = Pair<ST>::load(state, e);
    v[2 * p] = av * z.x;
    v[2 * p + 1] = av * z.y;
  }
  if (inject) {
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const int64_t e = tp.elem + (int64_t)(p >> 1) * tp.plane + (int64_t)(p & 1) * tp.w;
      const float2 nz = Pair<ET>::load(eps, e);
      v[2 * p] = fmaf(bv, nz.x, v[2 * p]);
      v[2 * p + 1] = fmaf(bv, nz.y, v[2 * p + 1]);
    }
  }
  float4* xr = reinterpret_cast<float4*>(x + j * 16);
#pragma unroll
  for (int q = 0; q < 4; ++q) xr[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
}

template <typename OT>
__global__ __launch_bounds__(kTPB) void k_scatter(ReqTable T, const float* __restrict__ x,
                                                  const int32_t* __restrict__ idx, int n, OT* __restrict__ out) {
  const int64_t j = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  if (j >= n) return;
  const int32_t t = idx[j];
  if (t < 0 || t >= T.tok_off[T.R]) return;  // out-of-range index: nothing is written
  const TokPos tp = decode_token(T, t);
  const float4* xr = reinterpret_cast<const float4*>(x + j * 16);
  float v[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 f = xr[q];
    v[4 * q] = f.x;
    v[4 * q + 1] = f.y;
    v[4 * q + 2] = f.z;
    v[4 * q + 3] = f.w;
  }
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const int64_t e = tp.elem + (int64_t)(p >> 1) * tp.plane + (int64_t)(p & 1) * tp.w;
    Pair<OT>::store(out, e, make_float2(v[2 * p], v[2 * p + 1]));
  }
}

template <typename IT, typename OT>
__global__ __launch_bounds__(kTPB) void k_convert(const IT* __restrict__ in, OT* __restrict__ out, int64_t pairs) {
  for (int64_t i = (int64_t)blockIdx.x * kTPB + threadIdx.x; i < pairs; i += (int64_t)gridDim.x * kTPB)
    Pair<OT>::store(out, 2 * i, Pair<IT>::load(in, 2 * i));
}

inline int grid_for(int64_t threads) { return (int)((threads + kTPB - 1) / kTPB); }
}  // namespace

hipError_t launch_gather(const ReqTable& T, const void* state, sphinx_dtype sdt, const void* eps, sphinx_dtype edt,
                         const int32_t* idx, int n, const float* a, const float* b, float* x, hipStream_t s) {
  const int g = grid_for(n);
  if (sdt == SPHINX_F32 && edt == SPHINX_F32)
    k_gather<float, float><<<g, kTPB, 0, s>>>(T, (const float*)state, (const float*)eps, idx, n, a, b, x);
  else if (sdt == SPHINX_F32 && edt == SPHINX_BF16)
    k_gather<float, bf16><<<g, kTPB, 0, s>>>(T, (const float*)state, (const bf16*)eps, idx, n, a, b, x);
  else if (sdt == SPHINX_BF16 && edt == SPHINX_F32)
    k_gather<bf16, float><<<g, kTPB, 0, s>>>(T, (const bf16*)state, (const float*)eps, idx, n, a, b, x);
  else
    k_gather<bf16, bf16><<<g, kTPB, 0, s>>>(T, (const bf16*)state, (const bf16*)eps, idx, n, a, b, x);
  return hipGetLastError();
}

hipError_t launch_scatter(const ReqTable& T, const float* x, const int32_t* idx, int n, void* out, sphinx_dtype odt,
                          hipStream_t s) {
  const int g = grid_for(n);
  if (odt == SPHINX_F32)
    k_scatter<float><<<g, kTPB, 0, s>>>(T, x, idx, n, (float*)out);
  else
    k_scatter<bf16><<<g, kTPB, 0, s>>>(T, x, idx, n, (bf16*)out);
  return hipGetLastError();
}

hipError_t launch_convert(const void* in, sphinx_dtype idt, void* out, sphinx_dtype odt, int64_t count,
                          hipStream_t s) {
  const int64_t pairs = count / 2;
  const int g = (int)std::min<int64_t>(grid_for(pairs), 8192);
  if (idt == SPHINX_F32 && odt == SPHINX_F32)
    k_convert<float, float><<<g, kTPB, 0, s>>>((const float*)in, (float*)out, pairs);
  else if (idt == SPHINX_F32 && odt == SPHINX_BF16)
    k_convert<float, bf16><<<g, kTPB, 0, s>>>((const float*)in, (bf16*)out, pairs);
  else if (idt == SPHINX_BF16 && odt == SPHINX_F32)
    k_convert<bf16, float><<<g, kTPB, 0, s>>>((const bf16*)in, (float*)out, pairs);
  else
    k_convert<bf16, bf16><<<g, kTPB, 0, s>>>((const bf16*)in, (bf16*)out, pairs);
  return hipGetLastError();
}

}  // namespace sphinx
