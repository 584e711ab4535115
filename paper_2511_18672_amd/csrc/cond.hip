// Conditioning of the denoiser on the step's timestep and token positions.
//
//  * k_cond_rows   collapses runs of frames with equal timestep into one
//                  conditioning row (all active frames of a request share the
//                  step's timestep), giving fmap[g] -> row and the row count U.
//  * k_temb        sinusoidal timestep embedding, 256 wide, in fp64.
//  * k_rowgemm     out[u][n] = act(sum_k X[u][k] W[n][k] + b[n]) for the U rows:
//                  the timestep MLP and the adaLN projections of all blocks in
//                  one pass over the weights (weight-read bound; one wave per
//                  two output columns, fp32 math).
//  * k_pos_tables  fp64 sinusoid tables for patch rows, columns and frames.
//  * k_token_meta  per selected row: global frame, conditioning row, packed
//                  (frame, y, x) position.
#include <type_traits>

#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int kTPB = 256;

__global__ void k_cond_rows(const int32_t* __restrict__ tau, int G, int32_t* __restrict__ fmap,
                            int32_t* __restrict__ utau, int32_t* __restrict__ U) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  int u = 0;
  int prev = 0;
  for (int g = 0; g < G; ++g) {
    const int t = tau[g];
    if (g == 0 || t != prev) {
      utau[u] = t;
      ++u;
      prev = t;
    }
    fmap[g] = u - 1;
  }
  *U = u;
}

__global__ __launch_bounds__(kTPB) void k_temb(const int32_t* __restrict__ utau, const int32_t* __restrict__ U,
                                               float* __restrict__ temb) {
  const int u = blockIdx.x;
  if (u >= *U) return;
  const int c = threadIdx.x;  // 0..255
  const int k = c & 127;
  const double w = exp(-log(1e4) * (double)k / 128.0);
  const double arg = (double)utau[u] * w;
  temb[(int64_t)u * SPHINX_TEMB_DIM + c] = (float)(c < 128 ? cos(arg) : sin(arg));
}

// out[u][n] = act(sum_k X[u][k] W[n][k] + b[n]) for the U conditioning rows.
// One wave per output column: the lanes stream the column's weight row with
// 16-byte loads (8 bf16 or 4 fp32 per vector, vectors lane, lane+64, ...), so
// the launch reads every weight exactly once with full-line accesses; the U
// rows of X are small and come from L1/L2.  Partial dot products are reduced
// across the wave.
template <typename WT>
struct WVec;
template <>
struct WVec<bf16> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void get(const bf16* p, float* w) {
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = (float)v[i];
  }
};
template <>
struct WVec<float> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void get(const float* p, float* w) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = v[i];
  }
};

constexpr int kGemvMaxVec = 4;  // K <= 4 * 64 * (elements per vector)
// NV = ceil(K / (64 * elements per vector)) vectors per lane, known at compile
// time: every lane issues its NV loads back to back (an out-of-range vector
// reloads the row's last one and is zeroed), instead of waiting after each
// guarded load.
constexpr int kRowgemmCols = 2;  // output columns per wave

template <typename WT, bool SILU_OUT, int NV>
__global__ __launch_bounds__(kTPB) void k_rowgemm(const float* __restrict__ X, int ldx, const int32_t* __restrict__ Up,
                                                  int K, int N, const WT* __restrict__ W, const WT* __restrict__ bias,
                                                  float* __restrict__ out, int ldo) {
  constexpr int VN = WVec<WT>::N;
  constexpr int C = kRowgemmCols;
  // C output columns per wave: their weight loads are in flight together and
  // each X load serves all of them (a column past N repeats column N - 1 and
  // is not stored)
  const int n0 = (blockIdx.x * (kTPB / kWave) + (int)(threadIdx.x / kWave)) * C;
  if (n0 >= N) return;
  const int lane = lane_id();
  const int U = *Up;
  const int nvec = K / VN;
  float bv[C];
  float w[C][NV][VN];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int n = min(n0 + c, N - 1);
    bv[c] = load_as_f32(bias, n);
    const WT* wr = W + (int64_t)n * K;
#pragma unroll
    for (int i = 0; i < NV; ++i) WVec<WT>::get(wr + min(lane + kWave * i, nvec - 1) * VN, w[c][i]);
  }
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (lane + kWave * i >= nvec)
#pragma unroll
        for (int e = 0; e < VN; ++e) w[c][i][e] = 0.0f;
  for (int u = 0; u < U; ++u) {
    const float* xr = X + (int64_t)u * ldx;
    float acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c) acc[c] = 0.0f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = min(lane + kWave * i, nvec - 1);  // zero weights past the row
#pragma unroll
      for (int e = 0; e < VN; e += 4) {
        const f32x4 xv = *reinterpret_cast<const f32x4*>(xr + v * VN + e);
#pragma unroll
        for (int c = 0; c < C; ++c) {
          acc[c] = fmaf(w[c][i][e], xv[0], acc[c]);
          acc[c] = fmaf(w[c][i][e + 1], xv[1], acc[c]);
          acc[c] = fmaf(w[c][i][e + 2], xv[2], acc[c]);
          acc[c] = fmaf(w[c][i][e + 3], xv[3], acc[c]);
        }
      }
    }
#pragma unroll
    for (int c = 0; c < C; ++c) acc[c] = wave_sum(acc[c]);
    if (lane == 0) {
#pragma unroll
      for (int c = 0; c < C; ++c)
        if (n0 + c < N) {
          float v = acc[c] + bv[c];
          if (SILU_OUT) v = silu(v);
          out[(int64_t)u * ldo + n0 + c] = v;
        }
    }
  }
}

__global__ __launch_bounds__(kTPB) void k_pos_tables(int D, int hp, int wp, int nf, float* __restrict__ Ty,
                                                     float* __restrict__ Tx, float* __restrict__ Tf) {
  const int64_t i = (int64_t)blockIdx.x * kTPB + threadIdx.x;
  const int half = D / 2, q = D / 4;
  const int64_t ny = (int64_t)hp * half, nx = (int64_t)wp * half, nfr = (int64_t)nf * D;
  if (i < ny + nx) {
    const bool is_y = i < ny;
    const int64_t li = is_y ? i : i - ny;
    const int pos = (int)(li / half), c = (int)(li % half);
    const int k = c % q;
    const double nu = exp(-log(1e4) * (double)k / (double)q);
    const double arg = (double)pos * nu;
    (is_y ? Ty : Tx)[li] = (float)(c < q ? sin(arg) : cos(arg));
  } else if (i < ny + nx + nfr) {
    const int64_t li = i - ny - nx;
    const int f = (int)(li / D), c = (int)(li % D);
    const int k = c % half;
    const double mu = exp(-log(1e4) * (double)k / (double)half);
    const double arg = (double)f * mu;
    Tf[li] = (float)(c < half ? sin(arg) : cos(arg));
  }
}

__global__ __launch_bounds__(kTPB) void k_token_meta(ReqTable T, const int32_t* __restrict__ idx, int n,
                                                     const int32_t* __restrict__ fmap, int32_t* __restrict__ gframe,
                                                     int32_t* __restrict__ crow, int32_t* __restrict__ posc) {
  const int j = blockIdx.x * kTPB + threadIdx.x;
  if (j >= n) return;
  const int32_t t = idx[j];
  if (t < 0 || t >= T.tok_off[T.R]) {  // out-of-range index: point at frame 0, position 0
    gframe[j] = 0;
    crow[j] = fmap[0];
    posc[j] = 0;
    return;
  }
  const TokPos p = decode_token(T, t);
  gframe[j] = p.g;
  crow[j] = fmap[p.g];
  posc[j] = (p.f << 20) | (p.y << 10) | p.x;
}
}  // namespace

hipError_t launch_cond_rows(const int32_t* tau, int G, int32_t* fmap, int32_t* utau, int32_t* U, hipStream_t s) {
  k_cond_rows<<<1, 64, 0, s>>>(tau, G, fmap, utau, U);
  return hipGetLastError();
}

hipError_t launch_temb(const int32_t* utau, const int32_t* U, int Gmax, float* temb, hipStream_t s) {
  k_temb<<<Gmax, SPHINX_TEMB_DIM, 0, s>>>(utau, U, temb);
  return hipGetLastError();
}

hipError_t launch_rowgemm(const float* X, int ldx, const int32_t* U, int K, const void* W, const void* b,
                          sphinx_dtype wdt, int N, bool silu_out, float* out, int ldo, hipStream_t s) {
  const int cols = kRowgemmCols * (kTPB / kWave);  // output columns per workgroup
  const int g = (N + cols - 1) / cols;
  const int nv = (K / (wdt == SPHINX_BF16 ? 8 : 4) + kWave - 1) / kWave;  // vectors per lane, 1..4
  auto go = [&](auto wt, auto silu, auto nvc) {
    typedef decltype(wt) WT;
    k_rowgemm<WT, decltype(silu)::value, decltype(nvc)::value>
        <<<g, kTPB, 0, s>>>(X, ldx, U, K, N, (const WT*)W, (const WT*)b, out, ldo);
  };
  auto by_nv = [&](auto wt, auto silu) {
    if (nv <= 1) go(wt, silu, std::integral_constant<int, 1>{});
    else if (nv == 2) go(wt, silu, std::integral_constant<int, 2>{});
    else if (nv == 3) go(wt, silu, std::integral_constant<int, 3>{});
    else go(wt, silu, std::integral_constant<int, 4>{});
  };
  if (wdt == SPHINX_BF16) {
    if (silu_out) by_nv(bf16{}, std::true_type{});
    else by_nv(bf16{}, std::false_type{});
  } else {
    if (silu_out) by_nv(float{}, std::true_type{});
    else by_nv(float{}, std::false_type{});
  }
  return hipGetLastError();
}

hipError_t launch_pos_tables(int D, int hp, int wp, int nf, float* Ty, float* Tx, float* Tf, hipStream_t s) {
  const int64_t total = (int64_t)hp * (D / 2) + (int64_t)wp * (D / 2) + (int64_t)nf * D;
  k_pos_tables<<<(int)((total + kTPB - 1) / kTPB), kTPB, 0, s>>>(D, hp, wp, nf, Ty, Tx, Tf);
  return hipGetLastError();
}

hipError_t launch_token_meta(const ReqTable& T, const int32_t* idx, int n, const int32_t* fmap, int32_t* gframe,
                             int32_t* crow, int32_t* posc, hipStream_t s) {
  k_token_meta<<<(n + kTPB - 1) / kTPB, kTPB, 0, s>>>(T, idx, n, fmap, gframe, crow, posc);
  return hipGetLastError();
}

}  // namespace sphinx
