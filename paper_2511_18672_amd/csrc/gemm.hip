// GEMMs of the denoiser blocks: C[M][N] = A[M][K] W[N][K]^T + b with a fused
// epilogue:
//   EPI_BIAS  : out = C                         (QKV projection)      -> bf16/fp32
//   EPI_GELU  : out = GELU_tanh(C)              (MLP first layer)     -> bf16/fp32
//   EPI_GATED : h  += (1 + gate[row]) * C       (out-proj, MLP second layer; fp32 residual)
// M = selected tokens (ragged), N, K multiples of the tile sizes.
//
// bf16 path (gfx950 MFMA): block tile 128x128, K step 64, 256 threads = 4 waves
// in a 2x2 grid, each wave a 64x64 tile of 2x2 v_mfma_f32_32x32x16_bf16.  A and
// W are both K-contiguous, so every operand fragment is one 16-byte LDS read.
// LDS rows are padded by 16 bytes against bank conflicts.  Global loads run
// two K steps ahead (two register sets, two LDS buffers, K loop unrolled by
// two), which hides the L2/HBM latency behind the MFMAs.  Rows past M are
// clamped to the last row and not stored.  The epilogue stages the fp32
// tile in LDS and finishes it with 16-byte row-contiguous loads and stores.
//
// fp32 path: a plain 64x64 SIMT tile (used by fp32 models only).
#include "kernels.hpp"

namespace sphinx {

namespace {
template <int EPI, typename OT>
__device__ __forceinline__ void epi_store(const GemmEpi& e, int m, int n, float v) {
  if constexpr (EPI == EPI_GATED) {
    float* h = reinterpret_cast<float*>(e.out);
    const int64_t o = (int64_t)m * e.ldo + n;
    h[o] = fmaf(1.0f + e.gate[(int64_t)e.crow[m] * e.ldg + n], v, h[o]);
  } else {
    if constexpr (EPI == EPI_GELU) v = gelu_tanh(v);
    reinterpret_cast<OT*>(e.out)[(int64_t)m * e.ldo + n] = store_from_f32<OT>(v);
  }
}

constexpr int BM = 128, BN = 128, BK = 64, LDK = BK + 8;
constexpr int CLD = BN + 4;  // fp32 staging row of the epilogue
constexpr int kGemmSmem = 2 * (BM + BN) * LDK * 2;
static_assert(BM * CLD * 4 <= kGemmSmem, "epilogue staging must fit in the operand buffers");

template <int EPI>
__global__ __launch_bounds__(256, 2) void k_gemm_bf16(const bf16* __restrict__ A, const bf16* __restrict__ W,
                                                      const bf16* __restrict__ bias, int M, int N, int K, GemmEpi e) {
  // one LDS block: two A and two B operand buffers, reused as the fp32 C tile
  __shared__ __attribute__((aligned(16))) unsigned char smem[kGemmSmem];
  bf16(*sA)[BM * LDK] = reinterpret_cast<bf16(*)[BM * LDK]>(smem);
  bf16(*sB)[BN * LDK] = reinterpret_cast<bf16(*)[BN * LDK]>(smem + 2 * BM * LDK * sizeof(bf16));
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int lrow = tid >> 3, lch = (tid & 7) * 8;
  const int g = lane >> 5, r32 = lane & 31;
  // Row pointers of this thread's four A and four W rows.  Rows past M are
  // clamped to M-1: they are computed like any other row and never stored.
  const bf16* pa[4];
  const bf16* pw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = lrow + 32 * i;
    pa[i] = A + (int64_t)min(m0 + r, M - 1) * K + lch;
    pw[i] = W + (int64_t)(n0 + r) * K + lch;
  }
  // Two register sets: the global loads run two K steps ahead of the MFMAs.
  bf16x8 ra0[4], rb0[4], ra1[4], rb1[4];
  auto gload = [&](int k0, bf16x8 (&ra)[4], bf16x8 (&rb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = *reinterpret_cast<const bf16x8*>(pa[i] + k0);
      rb[i] = *reinterpret_cast<const bf16x8*>(pw[i] + k0);
    }
  };
  auto sstore = [&](int buf, const bf16x8 (&ra)[4], const bf16x8 (&rb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = lrow + 32 * i;
      *reinterpret_cast<bf16x8*>(&sA[buf][r * LDK + lch]) = ra[i];
      *reinterpret_cast<bf16x8*>(&sB[buf][r * LDK + lch]) = rb[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[2], bw[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&sA[buf][(wm * 64 + i * 32 + r32) * LDK + ks * 16 + g * 8]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bw[j] = *reinterpret_cast<const bf16x8*>(&sB[buf][(wn * 64 + j * 32 + r32) * LDK + ks * 16 + g * 8]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bw[j], acc[i][j], 0, 0, 0);
    }
  };

  // K loop unrolled by two so that LDS buffers and register sets are static:
  // even steps read LDS buffer 0 (register set 0 was stored there), odd steps
  // buffer 1 (set 1).
  const int KT = K / BK;
  gload(0, ra0, rb0);
  if (KT > 1) gload(BK, ra1, rb1);
  sstore(0, ra0, rb0);
  __syncthreads();
  for (int kt = 0; kt < KT; kt += 2) {
    if (kt + 2 < KT) gload((kt + 2) * BK, ra0, rb0);
    compute(0);
    if (kt + 1 < KT) sstore(1, ra1, rb1);
    __syncthreads();
    if (kt + 1 >= KT) break;
    if (kt + 3 < KT) gload((kt + 3) * BK, ra1, rb1);
    compute(1);
    if (kt + 2 < KT) sstore(0, ra0, rb0);
    __syncthreads();
  }

  // Epilogue through LDS: each wave parks its 64x64 fp32 tile (register r of
  // block (i, j) is row 8*(r/4) + 4*g + r%4, column r32), then every thread
  // finishes 4-wide row segments with coalesced 16-byte loads and stores.
  float* sC = reinterpret_cast<float*>(smem);  // [BM][CLD], reuses the operand buffers
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sC[(wm * 64 + i * 32 + (r >> 2) * 8 + g * 4 + (r & 3)) * CLD + wn * 64 + j * 32 + r32] = acc[i][j][r];
  __syncthreads();
  const int c4 = (tid & 31) * 4;  // column inside the tile
  const int n = n0 + c4;
  float4 bv;
  {
    const bf16x4 b4 = *reinterpret_cast<const bf16x4*>(bias + n);
    bv = make_float4((float)b4[0], (float)b4[1], (float)b4[2], (float)b4[3]);
  }
#pragma unroll
  for (int q0 = 0; q0 < BM / 8; q0 += 4) {
    float4 v[4], hv[4], gv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = (q0 + u) * 8 + (tid >> 5);
      const int m = m0 + row;
      v[u] = *reinterpret_cast<const float4*>(&sC[row * CLD + c4]);
      v[u].x += bv.x;
      v[u].y += bv.y;
      v[u].z += bv.z;
      v[u].w += bv.w;
      if constexpr (EPI == EPI_GATED) {
        if (m < M) {
          hv[u] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(e.out) + (int64_t)m * e.ldo + n);
          gv[u] = *reinterpret_cast<const float4*>(e.gate + (int64_t)e.crow[m] * e.ldg + n);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int m = m0 + (q0 + u) * 8 + (tid >> 5);
      if (m >= M) continue;
      if constexpr (EPI == EPI_GATED) {
        float4 h = hv[u];
        h.x = fmaf(1.0f + gv[u].x, v[u].x, h.x);
        h.y = fmaf(1.0f + gv[u].y, v[u].y, h.y);
        h.z = fmaf(1.0f + gv[u].z, v[u].z, h.z);
        h.w = fmaf(1.0f + gv[u].w, v[u].w, h.w);
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(e.out) + (int64_t)m * e.ldo + n) = h;
      } else {
        if constexpr (EPI == EPI_GELU) {
          v[u].x = gelu_tanh(v[u].x);
          v[u].y = gelu_tanh(v[u].y);
          v[u].z = gelu_tanh(v[u].z);
          v[u].w = gelu_tanh(v[u].w);
        }
        bf16x4 o;
        o[0] = (bf16)v[u].x;
        o[1] = (bf16)v[u].y;
        o[2] = (bf16)v[u].z;
        o[3] = (bf16)v[u].w;
        *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(e.out) + (int64_t)m * e.ldo + n) = o;
      }
    }
  }
}

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ A, const float* __restrict__ W,
                                                  const float* __restrict__ bias, int M, int N, int K, GemmEpi e) {
  __shared__ float sA[16][65];
  __shared__ float sB[16][65];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int li = tid + 256 * q;
      const int r = li >> 4, k = li & 15;
      sA[k][r] = (m0 + r < M) ? A[(int64_t)(m0 + r) * K + k0 + k] : 0.0f;
      sB[k][r] = W[(int64_t)(n0 + r) * K + k0 + k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[k][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[k][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty + 16 * i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx + 16 * j;
      epi_store<EPI, float>(e, m, n, acc[i][j] + bias[n]);
    }
  }
}
}  // namespace

hipError_t launch_gemm(int epi, sphinx_dtype dt, const void* A, const void* W, const void* bias, int M, int N, int K,
                       const GemmEpi& e, hipStream_t s) {
  if (dt == SPHINX_BF16) {
    const dim3 grid(N / BN, (M + BM - 1) / BM);
    const bf16 *a = (const bf16*)A, *w = (const bf16*)W, *b = (const bf16*)bias;
    if (epi == EPI_BIAS) k_gemm_bf16<EPI_BIAS><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
    else if (epi == EPI_GELU) k_gemm_bf16<EPI_GELU><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
    else k_gemm_bf16<EPI_GATED><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
  } else {
    const dim3 grid(N / 64, (M + 63) / 64);
    const float *a = (const float*)A, *w = (const float*)W, *b = (const float*)bias;
    if (epi == EPI_BIAS) k_gemm_f32<EPI_BIAS><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
    else if (epi == EPI_GELU) k_gemm_f32<EPI_GELU><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
    else k_gemm_f32<EPI_GATED><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
  }
  return hipGetLastError();
}

}  // namespace sphinx
