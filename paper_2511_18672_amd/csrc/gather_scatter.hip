// Gather with noise injection (Alg. 1 add_noise on the selected tokens) and
// scatter/blend back into the NCHW latents (Sec. 3, Sec. 5.3: confident
// regions keep their values).
//
// One thread moves one (channel, patch-row) pair of a token: 2 horizontally
// adjacent latent values, i.e. 8 threads per token.  Neighbouring selected
// tokens along x are neighbours in memory, so a wave touches contiguous runs of
// the latent planes, and writes to x_sel ([n][16] fp32) are contiguous.
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

template <typename ST, typename ET>
__global__ __launch_bounds__(kTPB) void k_gather(ReqTable T, const ST* __restrict__ state, const ET* __restrict__ eps,
                                                 const int32_t* __restrict__ idx, int n, const float* __restrict__ a,
                                                 const float* __restrict__ b, float* __restrict__ x) {
  const int64_t gid = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  const int64_t j = gid >> 3;
  const int p = (int)(gid & 7);
  if (j >= n) return;
  const int32_t t = idx[j];
  if (t < 0 || t >= T.tok_off[T.R]) return;  // out-of-range index: nothing is read
  const TokPos tp = decode_token(T, t);
  const int c = p >> 1, py = p & 1;
  const int64_t e = tp.elem + (int64_t)c * tp.plane + (int64_t)py * tp.w;
  const float2 z = Pair<ST>::load(state, e);
  const float av = a[tp.g], bv = b[tp.g];
  float2 r = make_float2(av * z.x, av * z.y);
  if (eps != nullptr && bv != 0.0f) {
    const float2 nz = Pair<ET>::load(eps, e);
    r.x = fmaf(bv, nz.x, r.x);
    r.y = fmaf(bv, nz.y, r.y);
  }
  *reinterpret_cast<float2*>(x + j * 16 + p * 2) = r;
}

template <typename OT>
__global__ __launch_bounds__(kTPB) void k_scatter(ReqTable T, const float* __restrict__ x,
                                                  const int32_t* __restrict__ idx, int n, OT* __restrict__ out) {
  const int64_t gid = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  const int64_t j = gid >> 3;
  const int p = (int)(gid & 7);
  if (j >= n) return;
  const int32_t t = idx[j];
  if (t < 0 || t >= T.tok_off[T.R]) return;  // out-of-range index: nothing is written
  const TokPos tp = decode_token(T, t);
  const int c = p >> 1, py = p & 1;
  const int64_t e = tp.elem + (int64_t)c * tp.plane + (int64_t)py * tp.w;
  Pair<OT>::store(out, e, *reinterpret_cast<const float2*>(x + j * 16 + p * 2));
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
  const int g = grid_for((int64_t)n * 8);
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
  const int g = grid_for((int64_t)n * 8);
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
