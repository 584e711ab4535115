// Gather with noise injection (Alg. 1 add_noise on the selected tokens) and
// scatter/blend back into the latents (Sec. 3, Sec. 5.3: confident regions
// keep their values), for NCHW and token-major latents.
//
// NCHW: one thread moves one token.  Its position is decoded once; its 16
// values are eight 8-byte (channel, patch-row) pairs in the latent planes and
// one 64-byte row of x_sel ([n][16] fp32).  Neighbouring selected tokens along
// x are neighbours in memory, so a wave touches contiguous runs of each plane.
//
// Token-major: a token is one contiguous row (64 B in f32, 32 B in bf16) at
// 16*t, in the order of an x_sel row.  Four lanes move one token, four values
// each, so one wave instruction covers 16 whole rows on both sides.  The f32
// rows and x_sel are moved with non-temporal loads and stores (streamed once
// per launch); measured at 2^26 tokens this lifts the rates by 10-17 %.
#include <type_traits>

#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int kTPB = 256;

template <typename T> struct Vec;
template <> struct Vec<float> {
  static __device__ __forceinline__ float2 load2(const float* p, int64_t e) {
    return *reinterpret_cast<const float2*>(p + e);
  }
  static __device__ __forceinline__ void store2(float* p, int64_t e, float2 v) {
    *reinterpret_cast<float2*>(p + e) = v;
  }
  static __device__ __forceinline__ float4 load4(const float* p, int64_t e) {
    return *reinterpret_cast<const float4*>(p + e);
  }
  static __device__ __forceinline__ void store4(float* p, int64_t e, float4 v) {
    *reinterpret_cast<float4*>(p + e) = v;
  }
  // non-temporal forms for rows that are streamed once per launch
  static __device__ __forceinline__ float4 load4nt(const float* p, int64_t e) {
    const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + e));
    return make_float4(v[0], v[1], v[2], v[3]);
  }
  static __device__ __forceinline__ void store4nt(float* p, int64_t e, float4 v) {
    __builtin_nontemporal_store(f32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<f32x4*>(p + e));
  }
};
template <> struct Vec<bf16> {
  static __device__ __forceinline__ float2 load2(const bf16* p, int64_t e) {
    const bf16x2 v = *reinterpret_cast<const bf16x2*>(p + e);
    return make_float2((float)v[0], (float)v[1]);
  }
  static __device__ __forceinline__ void store2(bf16* p, int64_t e, float2 v) {
    bf16x2 o;
    o[0] = (bf16)v.x;
    o[1] = (bf16)v.y;
    *reinterpret_cast<bf16x2*>(p + e) = o;
  }
  static __device__ __forceinline__ float4 load4(const bf16* p, int64_t e) {
    const bf16x2* q = reinterpret_cast<const bf16x2*>(p + e);
    const bf16x2 v0 = q[0], v1 = q[1];
    return make_float4((float)v0[0], (float)v0[1], (float)v1[0], (float)v1[1]);
  }
  static __device__ __forceinline__ void store4(bf16* p, int64_t e, float4 v) {
    bf16x2 o0, o1;
    o0[0] = (bf16)v.x;
    o0[1] = (bf16)v.y;
    o1[0] = (bf16)v.z;
    o1[1] = (bf16)v.w;
    bf16x2* q = reinterpret_cast<bf16x2*>(p + e);
    q[0] = o0;
    q[1] = o1;
  }
  static __device__ __forceinline__ float4 load4nt(const bf16* p, int64_t e) { return load4(p, e); }
  static __device__ __forceinline__ void store4nt(bf16* p, int64_t e, float4 v) { store4(p, e, v); }
};

// Element offset of pair p = (c, py) = (p >> 1, p & 1) of a decoded NCHW token.
__device__ __forceinline__ int64_t nchw_pair(const TokPos& tp, int p) {
  return tp.elem + (int64_t)(p >> 1) * tp.plane + (int64_t)(p & 1) * tp.w;
}

template <typename ST, typename ET>
__global__ __launch_bounds__(kTPB) void k_gather_nchw(ReqTable T, const ST* __restrict__ state,
                                                      const ET* __restrict__ eps, const int32_t* __restrict__ idx,
                                                      int n, const float* __restrict__ a,
                                                      const float* __restrict__ b, GatherCtx C,
                                                      float* __restrict__ x) {
  const int64_t j = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  if (j >= n) return;
  const int32_t t = idx[j];
  if (t < 0 || t >= T.tok_off[T.R]) return;  // out-of-range index: nothing is read
  const TokPos tp = decode_token(T, t);
  const bool ctx = C.wmask != nullptr && C.wmask[t] == 0;
  const float av = ctx ? C.a[tp.g] : a[tp.g], bv = ctx ? C.b[tp.g] : b[tp.g];
  float v[16];
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const float2 z = Vec<ST>::load2(state, nchw_pair(tp, p));
    v[2 * p] = av * z.x;
    v[2 * p + 1] = av * z.y;
  }
  if (eps != nullptr && bv != 0.0f) {
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const float2 nz = Vec<ET>::load2(eps, nchw_pair(tp, p));
      v[2 * p] = fmaf(bv, nz.x, v[2 * p]);
      v[2 * p + 1] = fmaf(bv, nz.y, v[2 * p + 1]);
    }
  }
  float4* xr = reinterpret_cast<float4*>(x + j * 16);
#pragma unroll
  for (int q = 0; q < 4; ++q) xr[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
}

// Token-major gather: lane i moves values 4*(i%4) .. 4*(i%4)+3 of token i/4.
// Token-major gather: four lanes per token, 16 bytes each, and two tokens per
// thread (j and j + half): the second token's index, state and noise loads
// are in flight together with the first's, which doubles the bytes each
// thread keeps in flight (the kernel is bound by load latency, not by HBM).
template <typename ST, typename ET>
__global__ __launch_bounds__(kTPB) void k_gather_tok(ReqTable T, const ST* __restrict__ state,
                                                     const ET* __restrict__ eps, const int32_t* __restrict__ idx,
                                                     int n, const float* __restrict__ a,
                                                     const float* __restrict__ b, GatherCtx C,
                                                     float* __restrict__ x) {
  const int64_t i = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  const int64_t half = ((int64_t)n + 1) >> 1;
  const int64_t j1 = i >> 2;
  if (j1 >= half) return;
  const int q = (int)(i & 3);
  const int64_t js[2] = {j1, j1 + half};
  const int64_t Ntok = T.tok_off[T.R];
  int32_t ts[2];
  bool ok[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    ts[u] = js[u] < n ? idx[js[u]] : -1;
    ok[u] = ts[u] >= 0 && ts[u] < Ntok;  // out-of-range index: nothing is read
  }
  float4 z[2], nz[2];
  float av[2], bv[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    if (!ok[u]) continue;
    const int32_t t = ts[u];
    const int g = frame_of_token(T, t);
    const bool ctx = C.wmask != nullptr && C.wmask[t] == 0;
    av[u] = ctx ? C.a[g] : a[g];
    bv[u] = ctx ? C.b[g] : b[g];
    const int64_t e = 16 * (int64_t)t + 4 * q;
    z[u] = Vec<ST>::load4nt(state, e);
    if (eps != nullptr && bv[u] != 0.0f) nz[u] = Vec<ET>::load4(eps, e);  // noise only where injected
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    if (!ok[u]) continue;
    float4 v = make_float4(av[u] * z[u].x, av[u] * z[u].y, av[u] * z[u].z, av[u] * z[u].w);
    if (eps != nullptr && bv[u] != 0.0f)
      v = make_float4(fmaf(bv[u], nz[u].x, v.x), fmaf(bv[u], nz[u].y, v.y), fmaf(bv[u], nz[u].z, v.z),
                      fmaf(bv[u], nz[u].w, v.w));
    Vec<float>::store4nt(x, 16 * js[u] + 4 * q, v);
  }
}

template <typename OT>
__global__ __launch_bounds__(kTPB) void k_scatter_nchw(ReqTable T, const float* __restrict__ x,
                                                       const int32_t* __restrict__ idx, int n,
                                                       const uint8_t* __restrict__ wmask, OT* __restrict__ out) {
  const int64_t j = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  if (j >= n) return;
  const int32_t t = idx[j];
  if (t < 0 || t >= T.tok_off[T.R]) return;  // out-of-range index: nothing is written
  if (wmask != nullptr && wmask[t] == 0) return;  // context token: not written back
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
  for (int p = 0; p < 8; ++p) Vec<OT>::store2(out, nchw_pair(tp, p), make_float2(v[2 * p], v[2 * p + 1]));
}

template <typename OT>
__global__ __launch_bounds__(kTPB) void k_scatter_tok(int64_t N, const float* __restrict__ x,
                                                      const int32_t* __restrict__ idx, int n,
                                                      const uint8_t* __restrict__ wmask, OT* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  const int64_t j = i >> 2;
  if (j >= n) return;
  const int32_t t = idx[j];
  if (t < 0 || t >= N) return;  // out-of-range index: nothing is written
  if (wmask != nullptr && wmask[t] == 0) return;  // context token: not written back
  Vec<OT>::store4nt(out, 16 * (int64_t)t + 4 * (i & 3), Vec<float>::load4nt(x, 4 * i));
}

// Latent cache store: row j of qkv, columns [D, 3D) (key then value), to row
// idx[j] of the cache, 16 bytes per thread.
__global__ __launch_bounds__(kTPB) void k_kv_store(const uint4* __restrict__ qkv, int n, int row_chunks,
                                                   const int32_t* __restrict__ idx, int64_t N,
                                                   uint4* __restrict__ cache) {
  // row_chunks = 16-byte chunks in D elements; a qkv row has 3, a cache row 2
  const int64_t c = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  const int per = 2 * row_chunks;
  if (c >= (int64_t)n * per) return;
  const int j = (int)(c / per), k = (int)(c - (int64_t)j * per);
  const int32_t t = idx[j];
  if (t < 0 || t >= N) return;  // out-of-range index: nothing is stored
  cache[(int64_t)t * per + k] = qkv[(int64_t)j * 3 * row_chunks + row_chunks + k];
}

// Same-layout f32 copy: four 16-byte non-temporal loads in flight per thread,
// then their stores (the fastest copy form measured on this GPU).
__global__ __launch_bounds__(kTPB) void k_copy_f32(const float* __restrict__ in, float* __restrict__ out,
                                                  int64_t quads) {
  constexpr int U = 4;
  const f32x4* src = reinterpret_cast<const f32x4*>(in);
  f32x4* dst = reinterpret_cast<f32x4*>(out);
  const int64_t stride = (int64_t)gridDim.x * kTPB * U;
  for (int64_t base = (int64_t)blockIdx.x * kTPB * U + threadIdx.x; base < quads; base += stride) {
    f32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + (int64_t)u * kTPB;
      if (i < quads) v[u] = __builtin_nontemporal_load(src + i);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + (int64_t)u * kTPB;
      if (i < quads) __builtin_nontemporal_store(v[u], dst + i);
    }
  }
}

// Same-layout copy with dtype conversion, two values per step.
template <typename IT, typename OT>
__global__ __launch_bounds__(kTPB) void k_convert(const IT* __restrict__ in, OT* __restrict__ out, int64_t pairs) {
  for (int64_t i = (int64_t)blockIdx.x * kTPB + threadIdx.x; i < pairs; i += (int64_t)gridDim.x * kTPB)
    Vec<OT>::store2(out, 2 * i, Vec<IT>::load2(in, 2 * i));
}

// Layout change NCHW <-> token-major with dtype conversion, one token per
// thread (a whole-latent conversion, done once per run at its ends).
template <typename IT, typename OT, bool TO_TOKENS>
__global__ __launch_bounds__(kTPB) void k_relayout(ReqTable T, const IT* __restrict__ in, OT* __restrict__ out) {
  const int64_t t = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  if (t >= T.tok_off[T.R]) return;
  const TokPos tp = decode_token(T, t);
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    if (TO_TOKENS)
      Vec<OT>::store2(out, 16 * t + 2 * p, Vec<IT>::load2(in, nchw_pair(tp, p)));
    else
      Vec<OT>::store2(out, nchw_pair(tp, p), Vec<IT>::load2(in, 16 * t + 2 * p));
  }
}

inline unsigned grid_for(int64_t threads) { return (unsigned)((threads + kTPB - 1) / kTPB); }

template <typename ST, typename ET>
void gather_typed(const ReqTable& T, sphinx_layout lay, const void* state, const void* eps, const int32_t* idx,
                  int n, const float* a, const float* b, const GatherCtx& C, float* x, hipStream_t s) {
  if (lay == SPHINX_LAYOUT_TOKENS)
    k_gather_tok<ST, ET><<<grid_for(4 * (((int64_t)n + 1) >> 1)), kTPB, 0, s>>>(T, (const ST*)state,
                                                                                (const ET*)eps, idx, n, a, b, C, x);
  else
    k_gather_nchw<ST, ET><<<grid_for(n), kTPB, 0, s>>>(T, (const ST*)state, (const ET*)eps, idx, n, a, b, C, x);
}

template <typename IT, typename OT>
void convert_typed(const ReqTable& T, int64_t N, const void* in, sphinx_layout il, void* out, sphinx_layout ol,
                   hipStream_t s) {
  if (il == ol && std::is_same<IT, float>::value && std::is_same<OT, float>::value) {
    const int64_t quads = 4 * N;  // 16 values per token
    k_copy_f32<<<(unsigned)std::min<int64_t>((quads + 4 * kTPB - 1) / (4 * kTPB), 65536), kTPB, 0, s>>>(
        (const float*)in, (float*)out, quads);
  } else if (il == ol) {
    const int64_t pairs = 8 * N;
    k_convert<IT, OT><<<(unsigned)std::min<int64_t>(grid_for(pairs), 8192), kTPB, 0, s>>>((const IT*)in, (OT*)out,
                                                                                          pairs);
  } else if (ol == SPHINX_LAYOUT_TOKENS) {
    k_relayout<IT, OT, true><<<grid_for(N), kTPB, 0, s>>>(T, (const IT*)in, (OT*)out);
  } else {
    k_relayout<IT, OT, false><<<grid_for(N), kTPB, 0, s>>>(T, (const IT*)in, (OT*)out);
  }
}
}  // namespace

hipError_t launch_gather(const ReqTable& T, sphinx_layout lay, const void* state, sphinx_dtype sdt, const void* eps,
                         sphinx_dtype edt, const int32_t* idx, int n, const float* a, const float* b,
                         const GatherCtx& C, float* x, hipStream_t s) {
  if (sdt == SPHINX_F32 && edt == SPHINX_F32)
    gather_typed<float, float>(T, lay, state, eps, idx, n, a, b, C, x, s);
  else if (sdt == SPHINX_F32 && edt == SPHINX_BF16)
    gather_typed<float, bf16>(T, lay, state, eps, idx, n, a, b, C, x, s);
  else if (sdt == SPHINX_BF16 && edt == SPHINX_F32)
    gather_typed<bf16, float>(T, lay, state, eps, idx, n, a, b, C, x, s);
  else
    gather_typed<bf16, bf16>(T, lay, state, eps, idx, n, a, b, C, x, s);
  return hipGetLastError();
}

hipError_t launch_scatter(const ReqTable& T, const float* x, const int32_t* idx, int n, const uint8_t* wmask,
                          void* out, sphinx_dtype odt, sphinx_layout lay, hipStream_t s) {
  const int64_t N = T.tok_off[T.R];
  if (lay == SPHINX_LAYOUT_TOKENS) {
    const unsigned g = grid_for(4 * (int64_t)n);
    if (odt == SPHINX_F32)
      k_scatter_tok<float><<<g, kTPB, 0, s>>>(N, x, idx, n, wmask, (float*)out);
    else
      k_scatter_tok<bf16><<<g, kTPB, 0, s>>>(N, x, idx, n, wmask, (bf16*)out);
  } else {
    const unsigned g = grid_for(n);
    if (odt == SPHINX_F32)
      k_scatter_nchw<float><<<g, kTPB, 0, s>>>(T, x, idx, n, wmask, (float*)out);
    else
      k_scatter_nchw<bf16><<<g, kTPB, 0, s>>>(T, x, idx, n, wmask, (bf16*)out);
  }
  return hipGetLastError();
}

hipError_t launch_kv_store(sphinx_dtype dt, const void* qkv, int n, int D, const int32_t* idx, int64_t N,
                           void* cache, hipStream_t s) {
  const int row_chunks = D * (dt == SPHINX_BF16 ? 2 : 4) / 16;
  k_kv_store<<<grid_for((int64_t)n * 2 * row_chunks), kTPB, 0, s>>>((const uint4*)qkv, n, row_chunks, idx, N,
                                                                     (uint4*)cache);
  return hipGetLastError();
}

hipError_t launch_convert(const ReqTable& T, const void* in, sphinx_dtype idt, sphinx_layout il, void* out,
                          sphinx_dtype odt, sphinx_layout ol, hipStream_t s) {
  const int64_t N = T.tok_off[T.R];
  if (idt == SPHINX_F32 && odt == SPHINX_F32)
    convert_typed<float, float>(T, N, in, il, out, ol, s);
  else if (idt == SPHINX_F32 && odt == SPHINX_BF16)
    convert_typed<float, bf16>(T, N, in, il, out, ol, s);
  else if (idt == SPHINX_BF16 && odt == SPHINX_F32)
    convert_typed<bf16, float>(T, N, in, il, out, ol, s);
  else
    convert_typed<bf16, bf16>(T, N, in, il, out, ol, s);
  return hipGetLastError();
}

}  // namespace sphinx
