// Varlen non-causal attention over the selected tokens of each request
// (joint spatio-temporal attention of the denoiser blocks restricted to the
// gathered tokens, Sec. 5.3 / Alg. 1 partial_step on the masked tokens).
//
// bf16 path, head_dim 64, gfx950 MFMA (flash-attention style, online softmax):
//  * one workgroup = 128 queries of one segment and one head, 4 waves x 32
//    queries; K/V tiles of 64 keys are staged in LDS (K row-major, V
//    transposed to [d][key]);
//  * scores are computed transposed, S^T = K Q^T with v_mfma_f32_32x32x16_bf16:
//    every lane then owns one query and 16 of each 32 keys, so the row max and
//    row sum need no cross-lane traffic except one exchange with lane^32;
//  * P^T stays in registers and is fed directly as the B operand of
//    O^T = V^T P^T.  The MFMA sums over k-slots; a slot (g = lane/32, j) of
//    P^T holds key 16*half + 8*(j/4) + 4*g + j%4 of the 32-key block, and the
//    V^T A-operand is read with the same key permutation (two 8-byte LDS reads);
//  * the output O^T lands with the query on the lane, so the final 1/l
//    normalisation is lane-local;
//  * softmax in base 2 with the 1/sqrt(d) scale folded into log2(e)/sqrt(d);
//    P is rounded to bf16 for the PV product, the running sum uses fp32 P.
// Workgroups of the longest segment are scheduled first.
//
// fp32 path (fp32 models, head_dim <= 64): one thread per (query, head).
#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int AQ = 128;  // queries per workgroup
constexpr int AK = 64;   // keys per LDS tile
constexpr int HD = 64;   // head_dim of the bf16 path
constexpr int KLD = HD + 8;
constexpr int VLD = AK + 8;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__global__ __launch_bounds__(256, 2) void k_attn_bf16(const bf16* __restrict__ qkv, bf16* __restrict__ o, int D,
                                                      float scale_log2, SegTable S) {
  __shared__ __attribute__((aligned(16))) bf16 sK[AK * KLD];
  __shared__ __attribute__((aligned(16))) bf16 sV[HD * VLD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, r32 = lane & 31;
  const int head = blockIdx.y;
  int s = 0;
  while (s + 1 < S.nseg && S.tile_prefix[s + 1] <= (int)blockIdx.x) ++s;
  const int qt = (int)blockIdx.x - S.tile_prefix[s];
  const int seg0 = S.start[s], L = S.len[s];
  const int64_t ld = 3 * (int64_t)D;
  const bf16* Qg = qkv + head * HD;
  const bf16* Kg = qkv + D + head * HD;
  const bf16* Vg = qkv + 2 * D + head * HD;
  const bf16x8 zero8 = {};

  const int ql = qt * AQ + wave * 32 + r32;
  bf16x8 qf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
    qf[ks] = (ql < L) ? *reinterpret_cast<const bf16x8*>(Qg + (int64_t)(seg0 + ql) * ld + ks * 16 + g * 8) : zero8;

  f32x16 oacc[2] = {f32x16{}, f32x16{}};
  float m_run = -INFINITY, l_run = 0.0f;
  const int nkt = (L + AK - 1) / AK;
  for (int kt = 0; kt < nkt; ++kt) {
    const int kbase = kt * AK;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int key = (tid >> 3) + 32 * i, ch = (tid & 7) * 8;
      const bf16x8 v = (kbase + key < L)
                           ? *reinterpret_cast<const bf16x8*>(Kg + (int64_t)(seg0 + kbase + key) * ld + ch)
                           : zero8;
      *reinterpret_cast<bf16x8*>(&sK[key * KLD + ch]) = v;
    }
    {
      const int p = tid & 31, c = tid >> 5;
      const int k0 = kbase + 2 * p;
      const bf16x8 v0 = (k0 < L) ? *reinterpret_cast<const bf16x8*>(Vg + (int64_t)(seg0 + k0) * ld + c * 8) : zero8;
      const bf16x8 v1 =
          (k0 + 1 < L) ? *reinterpret_cast<const bf16x8*>(Vg + (int64_t)(seg0 + k0 + 1) * ld + c * 8) : zero8;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        bf16x2 pr;
        pr[0] = v0[i];
        pr[1] = v1[i];
        *reinterpret_cast<bf16x2*>(&sV[(c * 8 + i) * VLD + 2 * p]) = pr;
      }
    }
    __syncthreads();

    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&sK[(kb * 32 + r32) * KLD + ks * 16 + g * 8]);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sacc[kb], 0, 0, 0);
      }
    }
    // sacc[kb][r] = score of key kbase + 32*kb + 8*(r/4) + 4*g + r%4 with query r32
    if (kbase + AK > L) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kbase + kb * 32 + (r >> 2) * 8 + g * 4 + (r & 3) >= L) sacc[kb][r] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(m_run, mx * scale_log2);
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    float psum = 0.0f;
    bf16x8 pf[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pv = fast_exp2(fmaf(sacc[kb][r], scale_log2, -m_new));
        psum += pv;
        pf[kb][r >> 3][r & 7] = (bf16)pv;
      }
    l_run = fmaf(l_run, alpha, psum);
#pragma unroll
    for (int db = 0; db < 2; ++db) oacc[db] *= alpha;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const bf16* vrow = &sV[(db * 32 + r32) * VLD + kb * 32 + hf * 16 + g * 4];
          const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow);
          const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 8);
          const bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kb][hf], oacc[db], 0, 0, 0);
        }
    __syncthreads();
  }
  l_run += __shfl_xor(l_run, 32, kWave);
  if (ql < L) {
    const float inv = 1.0f / l_run;
    bf16* orow = o + (int64_t)(seg0 + ql) * D + head * HD;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        bf16x4 ov;
#pragma unroll
        for (int t = 0; t < 4; ++t) ov[t] = (bf16)(oacc[db][rr * 4 + t] * inv);
        *reinterpret_cast<bf16x4*>(orow + db * 32 + rr * 8 + g * 4) = ov;
      }
  }
}

constexpr int kF32Max = 64;

__global__ __launch_bounds__(128) void k_attn_f32(const float* __restrict__ qkv, float* __restrict__ o, int D, int d,
                                                  int heads, int n, float scale, SegTable S) {
  const int gid = blockIdx.x * 128 + threadIdx.x;
  if (gid >= n * heads) return;
  const int j = gid / heads, h = gid % heads;
  int s = 0;
  while (s + 1 < S.nseg_by_start && S.start_sorted[s + 1] <= j) ++s;
  const int seg0 = S.start_sorted[s], L = S.len_sorted[s];
  const int64_t ld = 3 * (int64_t)D;
  float q[kF32Max], acc[kF32Max];
#pragma unroll
  for (int c = 0; c < kF32Max; ++c) {
    q[c] = (c < d) ? qkv[(int64_t)j * ld + h * d + c] : 0.0f;
    acc[c] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  for (int t = seg0; t < seg0 + L; ++t) {
    const float* kr = qkv + (int64_t)t * ld + D + h * d;
    const float* vr = qkv + (int64_t)t * ld + 2 * D + h * d;
    float sc = 0.0f;
#pragma unroll
    for (int c = 0; c < kF32Max; ++c)
      if (c < d) sc = fmaf(q[c], kr[c], sc);
    sc *= scale;
    const float mn = fmaxf(m, sc);
    const float corr = expf(m - mn);
    const float p = expf(sc - mn);
    l = fmaf(l, corr, p);
#pragma unroll
    for (int c = 0; c < kF32Max; ++c)
      if (c < d) acc[c] = fmaf(acc[c], corr, p * vr[c]);
    m = mn;
  }
#pragma unroll
  for (int c = 0; c < kF32Max; ++c)
    if (c < d) o[(int64_t)j * D + h * d + c] = acc[c] / l;
}
}  // namespace

hipError_t launch_attention(sphinx_dtype dt, const void* qkv, void* o, int D, int heads, int head_dim, int n,
                            const SegTable& S, hipStream_t s) {
  if (dt == SPHINX_BF16) {
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)head_dim);
    const dim3 grid(S.tile_prefix[S.nseg], heads);
    k_attn_bf16<<<grid, 256, 0, s>>>((const bf16*)qkv, (bf16*)o, D, scale_log2, S);
  } else {
    const float scale = 1.0f / sqrtf((float)head_dim);
    k_attn_f32<<<(n * heads + 127) / 128, 128, 0, s>>>((const float*)qkv, (float*)o, D, head_dim, heads, n, scale, S);
  }
  return hipGetLastError();
}

}  // namespace sphinx
