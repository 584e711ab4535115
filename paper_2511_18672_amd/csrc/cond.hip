// Conditioning of the denoiser on the step's timestep and token positions.
//
//  * k_cond_rows   collapses runs of frames with equal timestep into one
//                  conditioning row (all active frames of a request share the
//                  step's timestep), giving fmap[g] -> row and the row count U.
//  * k_temb        sinusoidal timestep embedding, 256 wide, in fp64.
//  * k_rowgemm     out[u][n] = act(sum_k X[u][k] W[n][k] + b[n]) for the U rows:
//                  the timestep MLP and the adaLN projections of all blocks in
//                  one pass over the weights (weight-read bound; fp32 math).
//  * k_pos_tables  fp64 sinusoid tables for patch rows, columns and frames.
//  * k_token_meta  per selected row: global frame, conditioning row, packed
//                  (frame, y, x) position.
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

// 64 output columns per workgroup, conditioning rows processed 16 at a time.
template <typename WT, bool SILU_OUT>
__global__ __launch_bounds__(kTPB) void k_rowgemm(const float* __restrict__ X, int ldx, const int32_t* __restrict__ Up,
                                                  int K, const WT* __restrict__ W, const WT* __restrict__ bias,
                                                  float* __restrict__ out, int ldo) {
  __shared__ float s_w[64][65];
  __shared__ float s_x[16][64];
  const int U = *Up;
  const int n0 = blockIdx.x * 64;
  const int tn = threadIdx.x & 63, rg = threadIdx.x >> 6;
  for (int r0 = 0; r0 < U; r0 += 16) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < K; k0 += 64) {
      {  // weight tile: 64 columns x 64 k, stored [k][n]
        const int row = threadIdx.x >> 2, kc = (threadIdx.x & 3) * 16;
        const WT* src = W + (int64_t)(n0 + row) * K + k0 + kc;
#pragma unroll
        for (int i = 0; i < 16; ++i) s_w[kc + i][row] = load_as_f32(src, i);
      }
      {  // input tile: 16 rows x 64 k
        const int row = threadIdx.x >> 4, kc = (threadIdx.x & 15) * 4;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          s_x[row][kc + i] = (r0 + row < U) ? X[(int64_t)(r0 + row) * ldx + k0 + kc + i] : 0.0f;
      }
      __syncthreads();
#pragma unroll 8
      for (int k = 0; k < 64; ++k) {
        const float w = s_w[k][tn];
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = fmaf(s_x[rg + 4 * i][k], w, acc[i]);
      }
      __syncthreads();
    }
    const float bv = load_as_f32(bias, n0 + tn);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = r0 + rg + 4 * i;
      if (r < U) {
        float v = acc[i] + bv;
        if (SILU_OUT) v = silu(v);
        out[(int64_t)r * ldo + n0 + tn] = v;
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
  const int g = N / 64;
  if (wdt == SPHINX_BF16) {
    if (silu_out)
      k_rowgemm<bf16, true><<<g, kTPB, 0, s>>>(X, ldx, U, K, (const bf16*)W, (const bf16*)b, out, ldo);
    else
      k_rowgemm<bf16, false><<<g, kTPB, 0, s>>>(X, ldx, U, K, (const bf16*)W, (const bf16*)b, out, ldo);
  } else {
    if (silu_out)
      k_rowgemm<float, true><<<g, kTPB, 0, s>>>(X, ldx, U, K, (const float*)W, (const float*)b, out, ldo);
    else
      k_rowgemm<float, false><<<g, kTPB, 0, s>>>(X, ldx, U, K, (const float*)W, (const float*)b, out, ldo);
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
