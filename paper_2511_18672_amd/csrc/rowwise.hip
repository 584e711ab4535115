// Row-wise kernels of the denoiser:
//  * k_embed   h = x W_pe^T + b_pe + [Ty(y) || Tx(x)] + Tf(f)          (fp32;
//              k_embed_mfma on the matrix cores for bf16 weights at D = 128 k)
//  * k_ln_mod  a = LN(h) * (1 + scale[row]) + shift[row]  -> bf16/fp32  (one wave per row, or per two rows)
//  * k_final   eps_hat = (LN(h) (1 + scale) + shift) W_out^T + b_out, then the
//              DDIM update x <- c1 x + c2 eps_hat in place.  bf16 weights at
//              D = 128, 512, 1024, 1152: k_final_mfma, 16 rows per workgroup on the matrix
//              cores; otherwise one wave per row, the 16 outputs reduced with a
//              butterfly reduce-scatter.
// LayerNorm: biased variance, eps 1e-6, no affine; statistics in fp32 from the
// row held in registers (two passes over registers, one read of HBM).
#include <algorithm>
#include <atomic>

#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int kTPB = 256;
constexpr int kRowsPerBlock = kTPB / kWave;
constexpr int kMaxPer = 32;  // D <= 2048

// 16 weights of one output column as floats (a [..][16] row of WT).
template <typename WT>
__device__ __forceinline__ void load16(const WT* p, float (&w)[16]);
template <>
__device__ __forceinline__ void load16<bf16>(const bf16* p, float (&w)[16]) {
  const bf16x8 a = reinterpret_cast<const bf16x8*>(p)[0], b = reinterpret_cast<const bf16x8*>(p)[1];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    w[k] = (float)a[k];
    w[8 + k] = (float)b[k];
  }
}
template <>
__device__ __forceinline__ void load16<float>(const float* p, float (&w)[16]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 v = reinterpret_cast<const f32x4*>(p)[q];
    w[4 * q] = v[0];
    w[4 * q + 1] = v[1];
    w[4 * q + 2] = v[2];
    w[4 * q + 3] = v[3];
  }
}

// Output-weight table of k_final in LDS: column c's 16 weights are 32 (bf16)
// or 64 (fp32) bytes, i.e. CPC 16-byte chunks.  Chunk q of column c sits at
// chunk (CPC c + q) ^ x(c), x(c) < 4 CPC flipping only the chunk's place
// among the 4 columns sharing c >> 2, with x(c) = (c >> 3) & 7 for bf16 and
// (c >> 2) & 15 for fp32: the 16 lanes of one read pass, which take columns
// 4 (l + 64 i) + e, then hit 16 different 16-byte bank groups.
template <typename WT>
__device__ __forceinline__ int wt_chunk(int c, int q) {
  constexpr int CPC = 16 * (int)sizeof(WT) / 16;
  const int x = sizeof(WT) == 2 ? (c >> 3) & 7 : (c >> 2) & 15;
  return (CPC * c + q) ^ x;
}

// The reader's form of wt_chunk for column c = 4 (l + 64 i) + e of lane l:
// x(c) depends on the lane only, so chunk = 4 CPC (l + 64 i) + ((CPC e + q)
// ^ x_l), and the i term is an immediate offset.
template <typename WT>
__device__ __forceinline__ int wt_lane_off(int lane, int e, int q) {
  constexpr int CPC = 16 * (int)sizeof(WT) / 16;
  const int xl = sizeof(WT) == 2 ? (lane >> 1) & 7 : lane & 15;
  return 16 * (4 * CPC * lane + ((CPC * e + q) ^ xl));
}

template <typename WT>
__device__ __forceinline__ void load16_at(const unsigned char* tab, const int (&off)[16 * (int)sizeof(WT) / 16],
                                          int i, float (&w)[16]) {
  constexpr int VE = 16 / (int)sizeof(WT), CPC = 16 / VE;
  typedef WT vec_t __attribute__((ext_vector_type(16 / sizeof(WT))));
#pragma unroll
  for (int q = 0; q < CPC; ++q) {
    const vec_t v = *reinterpret_cast<const vec_t*>(tab + off[q] + 4096 * CPC * i);
#pragma unroll
    for (int u = 0; u < VE; ++u) w[q * VE + u] = (float)v[u];
  }
}

// One thread per four consecutive columns and a block of kEmbedRows rows,
// grid (row blocks, column blocks): the thread's 4 x 16 weights stay in
// registers across the rows (the weight matrix is read once per row block,
// not once per row); per row 16-byte loads of the position tables and one
// 16-byte store of h (x and the packed position are wave-uniform).
constexpr int kEmbedRows = 8;

template <typename WT>
__global__ __launch_bounds__(kTPB) void k_embed(const float* __restrict__ x, int n, int D, const WT* __restrict__ pe_w,
                                                const WT* __restrict__ pe_b, const float* __restrict__ Ty,
                                                const float* __restrict__ Tx, const float* __restrict__ Tf,
                                                const int32_t* __restrict__ posc, float* __restrict__ h) {
  const int quads = D >> 2;
  const int qd = (int)blockIdx.y * kTPB + (int)threadIdx.x;
  if (qd >= quads) return;
  const int c0 = 4 * qd;
  float w[4][16], b[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    load16<WT>(pe_w + (int64_t)(c0 + e) * 16, w[e]);
    b[e] = load_as_f32(pe_b, c0 + e);
  }
  const int half = D / 2;
  const int j0 = (int)blockIdx.x * kEmbedRows, j1 = min(j0 + kEmbedRows, n);
#pragma unroll 2
  for (int j = j0; j < j1; ++j) {
    const int pc = posc[j];
    const int f = pc >> 20, y = (pc >> 10) & 1023, xx = pc & 1023;
    float xr[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 v = reinterpret_cast<const f32x4*>(x + (int64_t)j * 16)[q];
      xr[4 * q] = v[0];
      xr[4 * q + 1] = v[1];
      xr[4 * q + 2] = v[2];
      xr[4 * q + 3] = v[3];
    }
    const f32x4 pos = (c0 < half) ? *reinterpret_cast<const f32x4*>(Ty + (int64_t)y * half + c0)
                                  : *reinterpret_cast<const f32x4*>(Tx + (int64_t)xx * half + (c0 - half));
    const f32x4 tf = *reinterpret_cast<const f32x4*>(Tf + (int64_t)f * D + c0);
    f32x4 out;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v = b[e];
#pragma unroll
      for (int k = 0; k < 16; ++k) v = fmaf(xr[k], w[e][k], v);
      out[e] = v + pos[e] + tf[e];
    }
    *reinterpret_cast<f32x4*>(h + (int64_t)j * D + c0) = out;
  }
}

// k_embed on the matrix cores (bf16 weights, D a multiple of 128).  The patch
// embedding is a GEMM with a 16-deep contraction: a wave computes a 32 x 32
// tile of h with v_mfma_f32_32x32x16_bf16 (K = 16, one MFMA per operand) on a
// hi/lo bf16 split of the fp32 latents, x = bf16(x) + bf16(x - bf16(x)), two
// MFMAs (bf16 products are exact in fp32, accumulation is fp32).  Lane l holds
// latent row l % 32, values 8 (l / 32) .. + 7 (the A layout) and column
// c0 + l % 32's weights at the same 8 positions (the B layout: 16 contiguous
// bytes of W_pe); the result gives lane l column c0 + l % 32 of rows
// 8 (i / 4) + 4 (l / 32) + i % 4, i < 16, to which it adds the bias and the
// position tables.  The 32 columns of a wave lie on one side of D / 2 (D is a
// multiple of 128), so the y or x table is a wave-uniform choice.  Workgroup:
// 32 rows x 128 columns, four waves side by side.
__global__ __launch_bounds__(kTPB) void k_embed_mfma(const float* __restrict__ x, int n, int D,
                                                     const bf16* __restrict__ pe_w, const bf16* __restrict__ pe_b,
                                                     const float* __restrict__ Ty, const float* __restrict__ Tx,
                                                     const float* __restrict__ Tf, const int32_t* __restrict__ posc,
                                                     float* __restrict__ h) {
  const int lane = (int)threadIdx.x & 63, wave = (int)threadIdx.x >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const int row0 = (int)blockIdx.x * 32;
  const int c = (int)blockIdx.y * 128 + wave * 32 + l32;
  const float* xr = x + (int64_t)min(row0 + l32, n - 1) * 16 + 8 * g;  // rows past n repeat row n - 1
  const f32x4 x0 = reinterpret_cast<const f32x4*>(xr)[0], x1 = reinterpret_cast<const f32x4*>(xr)[1];
  const bf16x8 wv = *reinterpret_cast<const bf16x8*>(pe_w + (int64_t)c * 16 + 8 * g);
  bf16x8 xhi, xlo;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float v = e < 4 ? x0[e] : x1[e - 4];
    const bf16 hi = (bf16)v;
    xhi[e] = hi;
    xlo[e] = (bf16)(v - (float)hi);
  }
  f32x16 acc = {};
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xhi, wv, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xlo, wv, acc, 0, 0, 0);
  const float bc = (float)pe_b[c];
  const int half = D >> 1;
  const bool left = c < half;
  const float* tp = left ? Ty + c : Tx + (c - half);
  // every row's position and table loads first, then the sums and stores
  int pc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) pc[i] = posc[min(row0 + 8 * (i >> 2) + 4 * g + (i & 3), n - 1)];
  float pos[16], tf[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int f = pc[i] >> 20, y = (pc[i] >> 10) & 1023, xx = pc[i] & 1023;
    pos[i] = tp[(int64_t)(left ? y : xx) * half];
    tf[i] = Tf[(int64_t)f * D + c];
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int row = row0 + 8 * (i >> 2) + 4 * g + (i & 3);
    if (row < n) h[(int64_t)row * D + c] = ((acc[i] + bc) + pos[i]) + tf[i];
  }
}

template <int V> struct VecF;
template <> struct VecF<1> {
  typedef float T;
  static __device__ __forceinline__ float get(const T& v, int i) { return v; }
};
template <> struct VecF<2> {
  typedef float2 T;
  static __device__ __forceinline__ float get(const T& v, int i) { return i == 0 ? v.x : v.y; }
};
template <> struct VecF<4> {
  typedef float4 T;
  static __device__ __forceinline__ float get(const T& v, int i) {
    return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
  }
};

template <typename OT, int V> struct VecStore;
template <typename OT> struct VecStore<OT, 1> {
  static __device__ __forceinline__ void put(OT* p, const float (&v)[1]) { *p = store_from_f32<OT>(v[0]); }
};
template <> struct VecStore<float, 2> {
  static __device__ __forceinline__ void put(float* p, const float (&v)[2]) {
    *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
  }
};
template <> struct VecStore<float, 4> {
  static __device__ __forceinline__ void put(float* p, const float (&v)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};
template <> struct VecStore<bf16, 2> {
  static __device__ __forceinline__ void put(bf16* p, const float (&v)[2]) {
    bf16x2 o;
    o[0] = (bf16)v[0];
    o[1] = (bf16)v[1];
    *reinterpret_cast<bf16x2*>(p) = o;
  }
};
template <> struct VecStore<bf16, 4> {
  static __device__ __forceinline__ void put(bf16* p, const float (&v)[4]) {
    bf16x4 o;
    o[0] = (bf16)v[0];
    o[1] = (bf16)v[1];
    o[2] = (bf16)v[2];
    o[3] = (bf16)v[3];
    *reinterpret_cast<bf16x4*>(p) = o;
  }
};

// One wave per row; lane handles V consecutive values per 64*V-wide chunk, so
// every load and store of a wave is one contiguous 256*V- (fp32) or 128*V-byte run.
// CH: chunks of 64 V columns per row when known at compile time (then all
// row loads issue back to back; instantiated for D = 512, 1024, 2048 with
// V = 4 and D = 1152 with V = 2), 0 for any D.
// HALF: the last of the CH chunks covers only lanes 0..31 (D = 64 V (CH - 1) + 32 V,
// e.g. D = 1152 in float4 chunks).
template <typename OT, int V, int CH, int R = 1, bool HALF = false>
__global__ __launch_bounds__(kTPB) void k_ln_mod(const float* __restrict__ h, int n, int D,
                                                 const float* __restrict__ mod, int ldm, int sh_off, int sc_off,
                                                 const int32_t* __restrict__ crow, OT* __restrict__ out) {
  typedef typename VecF<V>::T VT;
  static_assert(R == 1 || CH > 0, "several rows per wave need a compile-time chunk count");
  static_assert(!HALF || CH > 0, "a half last chunk needs a compile-time chunk count");
  constexpr int kMaxChunks = CH > 0 ? CH : kMaxPer / V;
  const int row0 = (blockIdx.x * kRowsPerBlock + (int)(threadIdx.x / kWave)) * R;
  if (row0 >= n) return;
  const int lane = lane_id();
  const int chunks = CH > 0 ? CH : D / (kWave * V);
  auto live = [&](int i) { return CH > 0 ? (!HALF || i + 1 < CH || lane < kWave / 2) : i < chunks; };
  // all rows' loads first; a row past n repeats row n - 1 and is not stored
  VT v[R][kMaxChunks];
  const float* m[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int row = min(row0 + j, n - 1);
    const float* hr = h + (int64_t)row * D;
    m[j] = mod + (int64_t)crow[row] * ldm;
#pragma unroll
    for (int i = 0; i < kMaxChunks; ++i) {
      if (HALF && i + 1 == CH)  // lanes 32..63 load a duplicate of lanes 0..31 and drop it
        v[j][i] = *reinterpret_cast<const VT*>(hr + (i * kWave + (lane & (kWave / 2 - 1))) * V);
      else if (CH > 0 || i < chunks)
        v[j][i] = *reinterpret_cast<const VT*>(hr + (i * kWave + lane) * V);
    }
  }
#pragma unroll
  for (int j = 0; j < R; ++j) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxChunks; ++i)
      if (live(i))
#pragma unroll
        for (int e = 0; e < V; ++e) s += VecF<V>::get(v[j][i], e);
    const float mu = wave_sum(s) / (float)D;
    float s2 = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxChunks; ++i)
      if (live(i)) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
          const float d = VecF<V>::get(v[j][i], e) - mu;
          s2 = fmaf(d, d, s2);
        }
      }
    const float rstd = rsqrtf(wave_sum(s2) / (float)D + 1e-6f);
    if (row0 + j >= n) break;
    OT* o = out + (int64_t)(row0 + j) * D;
#pragma unroll
    for (int i = 0; i < kMaxChunks; ++i)
      if (live(i)) {
        const int c = (i * kWave + lane) * V;
        const VT sh = *reinterpret_cast<const VT*>(m[j] + sh_off + c);
        const VT sc = *reinterpret_cast<const VT*>(m[j] + sc_off + c);
        float r[V];
#pragma unroll
        for (int e = 0; e < V; ++e)
          r[e] = fmaf((VecF<V>::get(v[j][i], e) - mu) * rstd, 1.0f + VecF<V>::get(sc, e), VecF<V>::get(sh, e));
        VecStore<OT, V>::put(o + c, r);
      }
  }
}

// One wave per row; lane owns the column quads lane + 64 i.  The output
// weights sit transposed in LDS (a column's 16 weights in two (bf16) or four
// (fp32) 16-byte chunks, swizzled as wt_chunk describes), so a column costs
// two or four conflict-free 16-byte LDS reads.
constexpr int kMaxQuads = 8;  // D <= 2048
template <typename WT>
__global__ __launch_bounds__(kTPB) void k_final(const float* __restrict__ h, int n, int D,
                                                const float* __restrict__ mod, int ldm, int sh_off, int sc_off,
                                                const int32_t* __restrict__ crow, const int32_t* __restrict__ gframe,
                                                const WT* __restrict__ out_w, const WT* __restrict__ out_b,
                                                const float* __restrict__ c1, const float* __restrict__ c2,
                                                float* __restrict__ x) {
  extern __shared__ __attribute__((aligned(16))) unsigned char s_raw[];
  WT* s_wt = reinterpret_cast<WT*>(s_raw);  // [D][16]
  {  // transposed fill, [16][D] -> [D][16]: sixteen independent 16-byte loads per thread
    constexpr int VE = 16 / (int)sizeof(WT);
    typedef WT vec_t __attribute__((ext_vector_type(16 / sizeof(WT))));
    for (int c0 = (int)threadIdx.x * VE; c0 < D; c0 += kTPB * VE) {
      vec_t wk[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) wk[k] = *reinterpret_cast<const vec_t*>(out_w + (int64_t)k * D + c0);
#pragma unroll
      for (int i = 0; i < VE; ++i)
#pragma unroll
        for (int q = 0; q < 16 / VE; ++q) {
          vec_t col;
#pragma unroll
          for (int u = 0; u < VE; ++u) col[u] = wk[q * VE + u][i];
          reinterpret_cast<vec_t*>(s_wt)[wt_chunk<WT>(c0 + i, q)] = col;
        }
    }
  }
  __syncthreads();
  const int lane = lane_id();
  const int quads = D >> 2;
  constexpr int CPC = 16 * (int)sizeof(WT) / 16;
  int woff[4][CPC];  // byte offsets of this lane's weight chunks (column quad 0)
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int q = 0; q < CPC; ++q) woff[e][q] = wt_lane_off<WT>(lane, e, q);
  // this lane's output after the reduce-scatter below
  const int kout = ((lane >> 5) & 1) * 8 + ((lane >> 4) & 1) * 4 + ((lane >> 3) & 1) * 2 + ((lane >> 2) & 1);
  const float bout = load_as_f32(out_b, kout);
  for (int row = blockIdx.x * kRowsPerBlock + (int)(threadIdx.x / kWave); row < n;
       row += gridDim.x * kRowsPerBlock) {
    // the row's conditioning index, frame, DDIM coefficients and state are
    // loaded up front, beside the row itself, so that only the modulation
    // loads wait for the statistics
    const int cr = crow[row], gf = gframe[row];
    float* xp = x + (int64_t)row * 16 + kout;
    const float c1g = c1[gf], c2g = c2[gf], xold = *xp;
    const float* hr = h + (int64_t)row * D;
    f32x4 v[kMaxQuads];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxQuads; ++i) {
      const int q = lane + kWave * i;
      v[i] = (q < quads) ? reinterpret_cast<const f32x4*>(hr)[q] : f32x4{0.f, 0.f, 0.f, 0.f};
      s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
    }
    const float mu = wave_sum(s) / (float)D;
    float s2 = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxQuads; ++i)
      if (lane + kWave * i < quads)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float d = v[i][e] - mu;
          s2 = fmaf(d, d, s2);
        }
    const float rstd = rsqrtf(wave_sum(s2) / (float)D + 1e-6f);
    const float* m = mod + (int64_t)cr * ldm;
    float acc[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k] = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxQuads; ++i) {
      const int q = lane + kWave * i;
      if (q < quads) {
        const f32x4 sc = *reinterpret_cast<const f32x4*>(m + sc_off + 4 * q);
        const f32x4 sh = *reinterpret_cast<const f32x4*>(m + sh_off + 4 * q);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float a = fmaf((v[i][e] - mu) * rstd, 1.0f + sc[e], sh[e]);
          float w[16];
          load16_at<WT>(s_raw, woff[e], i, w);
#pragma unroll
          for (int k = 0; k < 16; ++k) acc[k] = fmaf(a, w[k], acc[k]);
        }
      }
    }
    // butterfly reduce-scatter: after the four halving steps lane holds output
    // k = 8*b5 + 4*b4 + 2*b3 + b2 (b = lane bits), summed over lanes that differ
    // in those bits; the last two steps sum over lane bits 1 and 0.
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int mask = 32 >> st;
      const int cnt = 16 >> st;
      const bool up = (lane & mask) != 0;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (i < cnt / 2) {
          const float send = up ? acc[i] : acc[i + cnt / 2];
          const float keep = up ? acc[i + cnt / 2] : acc[i];
          acc[i] = keep + __shfl_xor(send, mask, kWave);
        }
    }
    float e = acc[0];
    e += __shfl_xor(e, 2, kWave);
    e += __shfl_xor(e, 1, kWave);
    if ((lane & 3) == 0) *xp = fmaf(c2g, e + bout, c1g * xold);
  }
}

// k_final on the matrix cores (bf16 weights, D = 128 KPW): the output
// projection is a GEMM with 16 columns, so a workgroup takes 16 rows and
// v_mfma_f32_16x16x32_bf16 does the 16 x D x 16 product.  Wave w owns the
// D/4 columns [32 KPW w, 32 KPW (w+1)); lane l holds row r = l % 16 at columns
// 32 (KPW w + kb) + 8 (l / 16) + 0..7, which is the A-operand layout of the
// MFMA (and its B operand, the weights of output r at the same columns, is 16
// contiguous bytes of out_w).
//  * LayerNorm statistics: each wave's mean and squared deviations over its
//    columns (the four lanes of a row reduced with two shuffles), combined
//    across the waves through LDS as equal-size groups (Chan et al.).
//  * The modulated value a is fp32; it enters the MFMA as a_hi = bf16(a) and
//    a_lo = bf16(a - a_hi), two MFMAs per 32 columns, so the products keep
//    about 17 significant bits of a (bf16 x bf16 products are exact in fp32
//    and the MFMA accumulates in fp32).
//  * Rows, weights and modulation are loaded up front (PF of the KPW column
//    blocks' modulation; the rest one block at a time, PF blocks ahead), so a
//    workgroup waits on memory about once.
//  * The four waves' 16 x 16 partial sums meet in LDS; thread t finishes row
//    t / 16, output t % 16 with the bias and the DDIM update.
// Modulation blocks loaded ahead at D = 1024 and 1152: 3 (162 and 176 VGPRs)
// measured 17.0 and 19.6 us at 9677 and 10194 rows, all of them up front (238
// and 256 VGPRs, fewer waves per SIMD) 17.9 and 24.6 us.
constexpr int kFinalAhead = 3;

template <int KPW, int PF>
__global__ __launch_bounds__(kTPB) void k_final_mfma(const float* __restrict__ h, int n, int D,
                                                     const float* __restrict__ mod, int ldm, int sh_off, int sc_off,
                                                     const int32_t* __restrict__ crow,
                                                     const int32_t* __restrict__ gframe, const bf16* __restrict__ out_w,
                                                     const bf16* __restrict__ out_b, const float* __restrict__ c1,
                                                     const float* __restrict__ c2, float* __restrict__ x) {
  static_assert(PF >= 1 && PF <= KPW, "modulation blocks loaded ahead");
  constexpr int WCOLS = 32 * KPW;  // columns per wave
  __shared__ float s_stat[4][16][2];
  __shared__ float s_acc[4][16][17];
  const int tid = (int)threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int row0 = (int)blockIdx.x * 16;
  const int row = min(row0 + r, n - 1);  // rows past n repeat row n - 1 and are not stored
  const int cb = WCOLS * wave + 8 * g;   // the lane's column at kb = 0
  const float* hr = h + (int64_t)row * D + cb;
  const float* m = mod + (int64_t)crow[row] * ldm + cb;
  const bf16* wr = out_w + (int64_t)r * D + cb;
  f32x4 hv[KPW][2], sc[KPW][2], sh[KPW][2];
  bf16x8 wv[KPW];
#pragma unroll
  for (int kb = 0; kb < KPW; ++kb) {
    hv[kb][0] = *reinterpret_cast<const f32x4*>(hr + 32 * kb);
    hv[kb][1] = *reinterpret_cast<const f32x4*>(hr + 32 * kb + 4);
  }
#pragma unroll
  for (int kb = 0; kb < KPW; ++kb) wv[kb] = *reinterpret_cast<const bf16x8*>(wr + 32 * kb);
  auto load_mod = [&](int kb) {
    sc[kb][0] = *reinterpret_cast<const f32x4*>(m + sc_off + 32 * kb);
    sc[kb][1] = *reinterpret_cast<const f32x4*>(m + sc_off + 32 * kb + 4);
    sh[kb][0] = *reinterpret_cast<const f32x4*>(m + sh_off + 32 * kb);
    sh[kb][1] = *reinterpret_cast<const f32x4*>(m + sh_off + 32 * kb + 4);
  };
#pragma unroll
  for (int kb = 0; kb < PF; ++kb) load_mod(kb);
  // statistics of the wave's columns of the row, then of the whole row
  float s = 0.f;
#pragma unroll
  for (int kb = 0; kb < KPW; ++kb)
#pragma unroll
    for (int e = 0; e < 4; ++e) s += hv[kb][0][e] + hv[kb][1][e];
  s += __shfl_xor(s, 16, kWave);
  s += __shfl_xor(s, 32, kWave);
  const float mw = s / (float)WCOLS;
  float q = 0.f;
#pragma unroll
  for (int kb = 0; kb < KPW; ++kb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float d0 = hv[kb][0][e] - mw, d1 = hv[kb][1][e] - mw;
      q = fmaf(d0, d0, q);
      q = fmaf(d1, d1, q);
    }
  q += __shfl_xor(q, 16, kWave);
  q += __shfl_xor(q, 32, kWave);
  if (g == 0) {
    s_stat[wave][r][0] = mw;
    s_stat[wave][r][1] = q;
  }
  __syncthreads();
  float mu = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) mu += s_stat[w][r][0];
  mu *= 0.25f;
  float m2 = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float d = s_stat[w][r][0] - mu;
    m2 += fmaf((float)WCOLS * d, d, s_stat[w][r][1]);
  }
  const float rstd = rsqrtf(m2 / (float)D + 1e-6f);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < KPW; ++kb) {
    if (kb + PF < KPW) load_mod(kb + PF);
    bf16x8 ahi, alo;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int hf = e >> 2, i = e & 3;
      const float a = fmaf((hv[kb][hf][i] - mu) * rstd, 1.0f + sc[kb][hf][i], sh[kb][hf][i]);
      const bf16 hi = (bf16)a;
      ahi[e] = hi;
      alo[e] = (bf16)(a - (float)hi);
    }
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, wv[kb], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, wv[kb], acc, 0, 0, 0);
  }
  // lane l holds rows 4 (l / 16) + i, output l % 16 of the wave's partial sum
#pragma unroll
  for (int i = 0; i < 4; ++i) s_acc[wave][4 * g + i][r] = acc[i];
  __syncthreads();
  const int orow = tid >> 4, on = tid & 15;
  const int grow = row0 + orow;
  if (grow < n) {
    const float e = (s_acc[0][orow][on] + s_acc[1][orow][on]) + (s_acc[2][orow][on] + s_acc[3][orow][on]);
    const int gf = gframe[grow];
    float* xp = x + (int64_t)grow * 16 + on;
    *xp = fmaf(c2[gf], e + (float)out_b[on], c1[gf] * *xp);
  }
}
}  // namespace

hipError_t launch_embed(const float* x, int n, int D, const void* pe_w, const void* pe_b, sphinx_dtype wdt,
                        const float* Ty, const float* Tx, const float* Tf, const int32_t* posc, float* h,
                        hipStream_t s) {
  if (wdt == SPHINX_BF16 && D % 128 == 0) {  // matrix cores: 32 rows x 128 columns per workgroup
    const dim3 gm((unsigned)((n + 31) / 32), (unsigned)(D / 128));  // rows in x: no 65535 limit
    k_embed_mfma<<<gm, kTPB, 0, s>>>(x, n, D, (const bf16*)pe_w, (const bf16*)pe_b, Ty, Tx, Tf, posc, h);
    return hipGetLastError();
  }
  const dim3 g((unsigned)((n + kEmbedRows - 1) / kEmbedRows), (unsigned)((D / 4 + kTPB - 1) / kTPB));
  if (wdt == SPHINX_BF16)
    k_embed<bf16><<<g, kTPB, 0, s>>>(x, n, D, (const bf16*)pe_w, (const bf16*)pe_b, Ty, Tx, Tf, posc, h);
  else
    k_embed<float><<<g, kTPB, 0, s>>>(x, n, D, (const float*)pe_w, (const float*)pe_b, Ty, Tx, Tf, posc, h);
  return hipGetLastError();
}

hipError_t launch_ln_mod(const float* h, int n, int D, const float* mod, int ldm, int sh_off, int sc_off,
                         const int32_t* crow, void* out, sphinx_dtype odt, hipStream_t s) {
  const int g = (n + kRowsPerBlock - 1) / kRowsPerBlock;
  // two rows per wave where a lane holds four float4 chunks of a row (D = 1024:
  // 13.2 -> 12.3 us at 9677 rows); at D = 1152 two rows per wave measured
  // slower (15.2 -> 16.2 us with float2 chunks), and float4 chunks with a half
  // last one beat nine float2 chunks (15.4 -> 14.8 us)
  const int g2 = (n + 2 * kRowsPerBlock - 1) / (2 * kRowsPerBlock);
  // 16-byte vectors need every row and every modulation chunk on a 16-byte boundary
  const bool v4 = (D % (kWave * 4) == 0) && (ldm % 4 == 0) && (sh_off % 4 == 0) && (sc_off % 4 == 0);
  const bool v2 = (D % (kWave * 2) == 0) && (ldm % 2 == 0) && (sh_off % 2 == 0) && (sc_off % 2 == 0);
  const int ch4 = v4 ? D / (kWave * 4) : 0;
  const int ch2 = (!v4 && v2) ? D / (kWave * 2) : 0;  // 9 at D = 1152
  // D = 1152 in float4 chunks: four full, the fifth on half the lanes
  const bool v4h = (ldm % 4 == 0) && (sh_off % 4 == 0) && (sc_off % 4 == 0);
  if (odt == SPHINX_BF16) {
    bf16* o = (bf16*)out;
    if (ch4 == 4) k_ln_mod<bf16, 4, 4, 2><<<g2, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (ch4 == 2) k_ln_mod<bf16, 4, 2><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (ch4 == 8) k_ln_mod<bf16, 4, 8><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (v4) k_ln_mod<bf16, 4, 0><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (ch2 == 9 && v4h) k_ln_mod<bf16, 4, 5, 1, true><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (ch2 == 9) k_ln_mod<bf16, 2, 9><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (v2) k_ln_mod<bf16, 2, 0><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else k_ln_mod<bf16, 1, 0><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
  } else {
    float* o = (float*)out;
    if (ch4 == 4) k_ln_mod<float, 4, 4><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (ch4 == 2) k_ln_mod<float, 4, 2><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (ch4 == 8) k_ln_mod<float, 4, 8><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (v4) k_ln_mod<float, 4, 0><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (ch2 == 9) k_ln_mod<float, 2, 9><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else if (v2) k_ln_mod<float, 2, 0><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
    else k_ln_mod<float, 1, 0><<<g, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, o);
  }
  return hipGetLastError();
}

hipError_t launch_final(const float* h, int n, int D, const float* mod, int ldm, int sh_off, int sc_off,
                        const int32_t* crow, const int32_t* gframe, const void* out_w, const void* out_b,
                        sphinx_dtype wdt, const float* c1, const float* c2, float* x, hipStream_t s) {
  // bf16 weights at D = 128 KPW (KPW 1, 4, 8, 9: the widths the tests cover) with 16-byte aligned
  // modulation rows: the matrix-core kernel, one workgroup per 16 rows
  const bool mod4 = (ldm % 4 == 0) && (sh_off % 4 == 0) && (sc_off % 4 == 0);
  if (wdt == SPHINX_BF16 && mod4 && D % 128 == 0) {
    const unsigned gb = (unsigned)((n + 15) / 16);
    const bf16 *w = (const bf16*)out_w, *b = (const bf16*)out_b;
    switch (D / 128) {
      case 1:
        k_final_mfma<1, 1><<<gb, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, gframe, w, b, c1, c2, x);
        return hipGetLastError();
      case 4:
        k_final_mfma<4, 4><<<gb, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, gframe, w, b, c1, c2, x);
        return hipGetLastError();
      case 8:
        k_final_mfma<8, kFinalAhead><<<gb, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, gframe, w, b, c1, c2, x);
        return hipGetLastError();
      case 9:
        k_final_mfma<9, kFinalAhead><<<gb, kTPB, 0, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, gframe, w, b, c1, c2, x);
        return hipGetLastError();
      default:
        break;
    }
  }
  // Grid-stride over rows: as many workgroups as fit on the device at once
  // (each fills its LDS weight table once), so that all of them run in one
  // round.  (A fixed 1024 left a quarter of them for a second round at three
  // workgroups per CU.)
  // The resident count is queried once per device, weight type and D (the
  // query is not cheap enough to repeat every step).
  const int rows_blocks = (n + kRowsPerBlock - 1) / kRowsPerBlock;
  const size_t lds = 16 * (size_t)D * (wdt == SPHINX_BF16 ? sizeof(bf16) : sizeof(float));
  struct Entry {
    std::atomic<int> key{-1}, blocks{0};
  };
  static Entry cache[64][2];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  Entry& ent = cache[dev][wdt == SPHINX_BF16 ? 0 : 1];
  int resident = ent.key.load(std::memory_order_acquire) == D ? ent.blocks.load(std::memory_order_relaxed) : 0;
  if (resident <= 0) {
    int per_cu = 0, cus = 0;
    const hipError_t err = wdt == SPHINX_BF16
                               ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_final<bf16>, kTPB, lds)
                               : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_final<float>, kTPB, lds);
    if (err != hipSuccess || per_cu <= 0) per_cu = 2;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
    resident = per_cu * cus;
    ent.blocks.store(resident, std::memory_order_relaxed);
    ent.key.store(D, std::memory_order_release);
  }
  const int g = std::min(rows_blocks, resident);
  if (wdt == SPHINX_BF16)
    k_final<bf16><<<g, kTPB, lds, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, gframe, (const bf16*)out_w,
                                       (const bf16*)out_b, c1, c2, x);
  else
    k_final<float><<<g, kTPB, lds, s>>>(h, n, D, mod, ldm, sh_off, sc_off, crow, gframe, (const float*)out_w,
                                        (const float*)out_b, c1, c2, x);
  return hipGetLastError();
}

// Forwarded rows per frame (the spatial segments of a factorised denoiser),
// as frame boundaries of the forwarded rows (idx ascending): first[g] = the
// first row whose token lies in frame g or later (g = 0..G; tokens below 0
// count as frame -1, tokens at or past N as frame G).  Row j writes first[g]
// for every g after the frame of row j-1 up to its own, so that with idx
// ascending every entry is written exactly once, without atomics.
__global__ __launch_bounds__(256) void k_frame_bounds(ReqTable T, const int32_t* __restrict__ idx, int n, int G,
                                                      int32_t* __restrict__ first) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j > n) return;
  const int64_t N = T.tok_off[T.R];
  auto frame = [&](int32_t t) { return t < 0 ? -1 : t >= N ? G : frame_of_token(T, t); };
  const int fp = j == 0 ? -1 : frame(idx[j - 1]);
  const int fc = j == n ? G : frame(idx[j]);
  for (int g = max(fp + 1, 0); g <= min(fc, G); ++g) first[g] = j;
}
// Token -> forwarded row map: pos[t] = j for t = idx[j], -1 elsewhere.
__global__ __launch_bounds__(256) void k_fill_neg(int32_t* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = -1;
}
__global__ __launch_bounds__(256) void k_pos_scatter(const int32_t* __restrict__ idx, int n, int64_t N,
                                                     int32_t* __restrict__ pos) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j < n && idx[j] >= 0 && idx[j] < N) pos[idx[j]] = j;
}

hipError_t launch_frame_bounds(const ReqTable& T, const int32_t* idx, int n, int G, int32_t* first, hipStream_t s) {
  k_frame_bounds<<<(unsigned)(n / 256 + 1), 256, 0, s>>>(T, idx, n, G, first);
  return hipGetLastError();
}

hipError_t launch_pos_map(int64_t N, const int32_t* idx, int n, int32_t* pos, hipStream_t s) {
  k_fill_neg<<<(unsigned)((N + 255) / 256), 256, 0, s>>>(pos, N);
  k_pos_scatter<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(idx, n, N, pos);
  return hipGetLastError();
}

}  // namespace sphinx
