// GEMMs of the denoiser blocks: C[M][N] = A[M][K] W[N][K]^T + b with a fused
// epilogue:
//   EPI_BIAS  : out = C                         (QKV projection)      -> bf16/fp32
//   EPI_GELU  : out = GELU_tanh(C)              (MLP first layer)     -> bf16/fp32
//   EPI_GATED : h  += (1 + gate[row]) * C       (out-proj, MLP second layer; fp32 residual)
// M = selected tokens (ragged); N and K multiples of 128 on the bf16 path.
//
// bf16 path (gfx950 MFMA): k_gemm_dma_* (described with their code).  Operand
// offsets are 32-bit: the caller guarantees M*K and N*K below 2^31 elements.
//
// fp32 path: a plain 64x64 SIMT tile (used by fp32 models only).
#include <atomic>
#include <type_traits>

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
    if constexpr (EPI == EPI_BIAS) v = n < e.qcols ? v * e.qscale : v;
    reinterpret_cast<OT*>(e.out)[(int64_t)m * e.ldo + n] = store_from_f32<OT>(v);
  }
}

// ---------------------------------------------------------------------------
// bf16 GEMM with direct global->LDS copies (global_load_lds_dwordx4).
//  * Block tile 128x128x64, 4 waves in 2x2, each a 64x64 tile of 2x2
//    v_mfma_f32_32x32x16_bf16; two workgroups per CU.
//  * Operand tiles are unpadded 128-byte rows (A rows, then W rows, of one
//    64-wide K step); chunk c of row r sits at c ^ ((r >> 1) & 7), which spreads
//    the 16 rows of one ds_read_b128 pass (same chunk) over all 64 LDS banks.
//    Each wave copies 8 rows per instruction: lane i of copy q writes slot i%8
//    of row 8q + i/8 and reads the global chunk the permutation puts there, so
//    the copy needs no registers and no LDS stores; its source is a
//    wave-uniform scalar base (A or W, moved by scalar adds per K step) plus a
//    fixed per-lane byte offset, so it needs no VALU either.
//  * On gfx950 VALU work does not overlap other waves' MFMAs, so the loop is
//    kept free of it: the K loop is unrolled over the ring, making every
//    fragment address a loop-invariant base plus an immediate offset.
//  * K steps live in a 2-slot ring.  The wait for the next step's copies and
//    the workgroup barrier sit inside the last 16-deep k-step of the current
//    one, so the next step's first fragments are read (and the following
//    copies issued) while the last MFMAs of the current step run; inside a
//    step each k-step's fragment reads are issued before the previous
//    k-step's MFMAs.  Barriers carry no memory fence: each wave waits for its
//    own copies (vmcnt) and LDS reads (lgkmcnt) first.
//  * Every output starts at its bias and accumulates its k-steps of 16 in
//    ascending k, whatever the tile shape, so all variants give bit-identical
//    results.
//  * A 192-row variant (wave tiles 96x64, 80 KB of LDS, epilogue staged one
//    wave row at a time) is launched where its smaller tile count packs into
//    fewer rounds of two workgroups per CU; same results.
//  * Launches whose 128-, 192- or 256-row tiles all fit on the CUs at once
//    (few selected tokens) run the smallest such tile, one eight-wave
//    workgroup per CU with a ring of 3 or 4 stages; same results.
namespace dma {

// s_waitcnt immediate: vmcnt(vm) expcnt(7) lgkmcnt(0) (gfx9 encoding: vmcnt in
// bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8)
constexpr int wait_vm_lgkm0(int vm) { return 0x0070 | (vm & 15) | ((vm >> 4) << 14); }

// EH: the fp32 epilogue tile is staged in EH row halves (EH = 2 when the
// whole tile would need more LDS than the operand ring).  NW waves in 2 rows
// of NW/2 (4: 2x2, 8: 2x4).
template <int BM, int BN, int NS, int EH = 1, int NW = 4>
struct DmaCfg {
  static constexpr int BK = 64;
  static constexpr int NT = 64 * NW, WGN = NW / 2;  // threads; waves along N
  static constexpr int WM = BM / 2, WN = BN / WGN, TI = WM / 32, TJ = WN / 32;
  static constexpr int STAGE = (BM + BN) * 128;     // bytes per K-step
  static constexpr int COPIES = (BM + BN) / 8 / NW; // copy instructions per wave per stage
  static constexpr int CLD = BN + 4;                // epilogue staging row (fp32)
  static constexpr int EROWS = BM / EH;             // tile rows staged at once
  static constexpr int SMEM = NS * STAGE > EROWS * CLD * 4 ? NS * STAGE : EROWS * CLD * 4;
  static_assert(EH == 1 || EH == 2, "whole tile or two halves (one per wave row)");
  static_assert(NW == 4 || NW == 8, "2x2 or 2x4 waves");
  static_assert(COPIES * 8 * NW == BM + BN && BM % 8 == 0, "each copy instruction moves 8 rows of A or of W");
};

// Tile of a one-dimensional grid of BM x BN tiles; workgroups are dealt to the
// 8 XCDs round-robin.  Wide N (more than 8 column tiles, and W at least a
// quarter of A): tiles in plain N-fastest order, so XCD x always gets the
// column tiles n = x (mod 8) and keeps that eighth of W in its L2 for the
// whole kernel.  Otherwise renumbered (xcd_tile) so that each XCD takes
// consecutive row blocks of A with all their column tiles: A is fetched into
// one L2 instead of eight, W into all eight.
template <int BM, int BN>
__device__ __forceinline__ void grid_tile(int M, int N, int& m0, int& n0) {
  const int nt = N / BN;
  if (nt > 8 && M < 4 * N) {
    m0 = ((int)blockIdx.x / nt) * BM;
    n0 = ((int)blockIdx.x % nt) * BN;
  } else {
    const int tile = xcd_tile((int)blockIdx.x, (int)gridDim.x);
    m0 = (tile / nt) * BM;
    n0 = (tile % nt) * BN;
  }
}

template <int EPI, int BM, int BN, int NS, int EH = 1, int NW = 4>
__device__ __forceinline__ void gemm_dma_body(const bf16* __restrict__ A, const bf16* __restrict__ W,
                                              const bf16* __restrict__ bias, int M, int N, int K, GemmEpi e,
                                              unsigned char* smem, int m0, int n0) {
  typedef DmaCfg<BM, BN, NS, EH, NW> C;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int g = lane >> 5, r32 = lane & 31;

  // copy sources: instruction i of this wave fills rows 8q .. 8q+7 of the
  // stage (q = wave * COPIES + i; rows < BM are A rows, the rest W rows)
  // (the operand, A or W, is wave-uniform: a scalar base; the lane's byte
  // offset from it is fixed, so moving to the next K step is scalar arithmetic)
  const bf16* src[C::COPIES];
  uint32_t voff[C::COPIES];
#pragma unroll
  for (int i = 0; i < C::COPIES; ++i) {
    const int q = wave * C::COPIES + i;
    const int row = 8 * q + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    if (8 * q < BM) {
      src[i] = A;
      voff[i] = 2u * (uint32_t)(min(m0 + row, M - 1) * K + c * 8);
    } else {
      src[i] = W;
      voff[i] = 2u * (uint32_t)((n0 + row - BM) * K + c * 8);
    }
  }
  auto copy_stage = [&](int kt, int slot) {
    unsigned char* base = smem + slot * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::COPIES; ++i)
      lds_dma16_at(src[i] + kt * C::BK, voff[i], base + (wave * C::COPIES + i) * 1024);
  };
  // fragment offsets inside a stage (k-step ks of 16)
  int foff[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) foff[ks] = r32 * 128 + (((2 * ks + g) ^ ((r32 >> 1) & 7)) << 4);
  const int a_row0 = wm * C::WM, b_row0 = BM + wn * C::WN;

  // acc[i][j] is the transposed output block: the MFMA takes the W fragment
  // as its A operand, so lane l holds row a_row0 + 32 i + l%32 of the tile and,
  // in registers 4q .. 4q+3, its four consecutive columns wn WN + 32 j + 8q +
  // 4(l/32) .. +3.  The accumulators start at the bias of their column, so the
  // epilogue adds no bias.
  f32x16 acc[C::TI][C::TJ];
#pragma unroll
  for (int j = 0; j < C::TJ; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bf16x4 b4 = *reinterpret_cast<const bf16x4*>(bias + n0 + wn * C::WN + j * 32 + 8 * q + 4 * g);
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < C::TI; ++i) acc[i][j][4 * q + t] = (float)b4[t];
    }

  const int KT = K / C::BK;  // even (K is a multiple of 128)
  static_assert(NS >= 2 && NS <= 4, "ring of 2 to 4 stages");
  // Stage j lives in slot j % NS.  The wait for stage kt+1 and the barrier sit
  // inside the last k-step of tile kt: after it every wave has read all of
  // stage kt (so its slot can be refilled with stage kt+NS) and stage kt+1 has
  // landed (so its first fragments can be read while the last MFMAs of tile
  // kt run).  With NS > 2 every K step refills its slot, near the end with a
  // copy of the last stage into a slot that is not read again, so that at
  // each wait exactly the NS - 2 newest stages may still be in flight.
  auto sync_stage = [&]() {
    __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0((NS - 2) * C::COPIES));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
#pragma unroll
  for (int st = 0; st < NS; ++st) copy_stage(NS == 2 ? st : min(st, KT - 1), st);
  // stage 0 must land before the first reads; the later ones may stay in flight
  __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0((NS - 1) * C::COPIES));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  bf16x8 fa[4][C::TI], fb[4][C::TJ];  // one register set per k-step
  auto read = [&](const unsigned char* st, int ks, int buf) {
#pragma unroll
    for (int i = 0; i < C::TI; ++i)
      fa[buf][i] = *reinterpret_cast<const bf16x8*>(st + (a_row0 + 32 * i) * 128 + foff[ks]);
#pragma unroll
    for (int j = 0; j < C::TJ; ++j)
      fb[buf][j] = *reinterpret_cast<const bf16x8*>(st + (b_row0 + 32 * j) * 128 + foff[ks]);
  };
  // One K step in ring slot SLOT (a compile-time constant, so that every
  // fragment address is a loop-invariant base plus an immediate offset).
  auto step = [&](int kt, auto SLOT) {
    constexpr int slot = decltype(SLOT)::value, nslot = slot + 1 == NS ? 0 : slot + 1;
    const unsigned char* st = smem + slot * C::STAGE;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if (ks < 3) {
        read(st, ks + 1, ks + 1);
      } else if (kt + 1 < KT) {
        sync_stage();
        if constexpr (NS == 2) {
          if (kt + NS < KT) copy_stage(kt + NS, slot);
        } else {
          copy_stage(min(kt + NS, KT - 1), slot);
        }
        read(smem + nslot * C::STAGE, 0, 0);
      }
      // the next k-step's reads are issued before this k-step's MFMAs
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < C::TI; ++i)
#pragma unroll
        for (int j = 0; j < C::TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[ks][j], fa[ks][i], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  read(smem, 0, 0);
  // whole trips over the ring, then (NS > 2) the last KT % NS stages; with two
  // slots KT is even (K is a multiple of 128, which launch_gemm checks)
  if constexpr (NS == 2) {
    for (int kt = 0; kt < KT; kt += 2) {
      step(kt, std::integral_constant<int, 0>{});
      step(kt + 1, std::integral_constant<int, 1>{});
    }
  } else {
    int kt = 0;
    for (; kt + NS <= KT; kt += NS) {
      step(kt, std::integral_constant<int, 0>{});
      step(kt + 1, std::integral_constant<int, 1>{});
      step(kt + 2, std::integral_constant<int, 2>{});
      if constexpr (NS > 3) step(kt + 3, std::integral_constant<int, 3>{});
    }
    if (kt < KT) step(kt, std::integral_constant<int, 0>{});
    if (kt + 1 < KT) step(kt + 1, std::integral_constant<int, 1>{});
    if constexpr (NS > 3)
      if (kt + 2 < KT) step(kt + 2, std::integral_constant<int, 2>{});
  }
  __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  // epilogue: fp32 tile staged in LDS (whole, or one wave row's half at a
  // time), then 16-byte row-contiguous I/O.  Outputs and the residual are
  // addressed as a wave-uniform tile base plus the thread's 32-bit byte offset
  // (at most EROWS rows of ldo elements), which grows by a fixed stride per
  // pass; tiles wholly inside M skip the per-row checks, and the query scale
  // is a tile-uniform branch.
  float* sC = reinterpret_cast<float*>(smem);
  constexpr int TPR = BN / 4;          // threads per row (one float4 each)
  constexpr int RPP = C::NT / TPR;     // rows per pass
  constexpr int NP = C::EROWS / RPP;   // row passes per staged half
  constexpr int OSZ = EPI == EPI_GATED ? 4 : 2;  // output bytes: fp32 residual or bf16 activation
  const int c4 = (tid % TPR) * 4, rsub = tid / TPR;
  const uint32_t off0 = (uint32_t)(rsub * e.ldo + c4) * OSZ, ostep = (uint32_t)(RPP * e.ldo) * OSZ;
  auto epilogue = [&](auto FULL, auto QT) {
    constexpr bool kFull = decltype(FULL)::value, kQ = decltype(QT)::value;
#pragma unroll
    for (int h = 0; h < EH; ++h) {
      const int mh = m0 + h * C::EROWS;  // first row of this half
      char* obase = reinterpret_cast<char*>(e.out) + ((int64_t)mh * e.ldo + n0) * OSZ;
      // gated residual: every pass's residual and gate loads are issued before
      // the staging (rows past M read row M - 1 and are not stored), so their
      // latencies overlap instead of following one another pass by pass
      float4 hres[EPI == EPI_GATED ? NP : 1], gres[EPI == EPI_GATED ? NP : 1];
      if constexpr (EPI == EPI_GATED) {
        int cr[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const int m = mh + p * RPP + rsub;
          cr[p] = e.crow[kFull ? m : min(m, M - 1)];
        }
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          // in a tile that crosses M the clamped row may lie before this half
          // (a whole half past M reads row M - 1): address it absolutely there
          if constexpr (kFull)
            hres[p] = *reinterpret_cast<const float4*>(obase + off0 + p * ostep);
          else
            hres[p] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(e.out) +
                                                       (int64_t)min(mh + p * RPP + rsub, M - 1) * e.ldo + n0 + c4);
          gres[p] = *reinterpret_cast<const float4*>(e.gate + (int64_t)cr[p] * e.ldg + n0 + c4);
        }
      }
      if (EH == 1 || wm == h) {  // four consecutive columns per 16-byte LDS store
        float* srow = sC + (a_row0 - h * C::EROWS + r32) * C::CLD + wn * C::WN + 4 * g;
#pragma unroll
        for (int i = 0; i < C::TI; ++i)
#pragma unroll
          for (int j = 0; j < C::TJ; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              *reinterpret_cast<float4*>(srow + i * 32 * C::CLD + j * 32 + 8 * q) =
                  make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
      }
      __syncthreads();
      if constexpr (EPI == EPI_GATED) {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const float4 v = *reinterpret_cast<const float4*>(&sC[(p * RPP + rsub) * C::CLD + c4]);
          const float4 gv = gres[p];
          float4 hv = hres[p];
          hv.x = fmaf(1.0f + gv.x, v.x, hv.x);
          hv.y = fmaf(1.0f + gv.y, v.y, hv.y);
          hv.z = fmaf(1.0f + gv.z, v.z, hv.z);
          hv.w = fmaf(1.0f + gv.w, v.w, hv.w);
          if (kFull || mh + p * RPP + rsub < M) *reinterpret_cast<float4*>(obase + off0 + p * ostep) = hv;
        }
      } else {
#pragma unroll 4
        for (int p = 0; p < NP; ++p) {
          if (!kFull && mh + p * RPP + rsub >= M) continue;
          float4 v = *reinterpret_cast<const float4*>(&sC[(p * RPP + rsub) * C::CLD + c4]);
          if constexpr (EPI == EPI_GELU) {
            v.x = gelu_tanh(v.x);
            v.y = gelu_tanh(v.y);
            v.z = gelu_tanh(v.z);
            v.w = gelu_tanh(v.w);
          }
          if constexpr (kQ) {
            v.x *= e.qscale;
            v.y *= e.qscale;
            v.z *= e.qscale;
            v.w *= e.qscale;
          }
          bf16x4 o;
          o[0] = (bf16)v.x;
          o[1] = (bf16)v.y;
          o[2] = (bf16)v.z;
          o[3] = (bf16)v.w;
          *reinterpret_cast<bf16x4*>(obase + off0 + p * ostep) = o;
        }
      }
      if (h + 1 < EH) __syncthreads();  // the next half reuses the staging rows
    }
  };
  // a column tile is all queries or none (qcols is a multiple of 128)
  const bool qtile = EPI == EPI_BIAS && n0 < e.qcols;
  if (m0 + BM <= M) {
    if (qtile) epilogue(std::true_type{}, std::true_type{});
    else epilogue(std::true_type{}, std::false_type{});
  } else {
    if (qtile) epilogue(std::false_type{}, std::true_type{});
    else epilogue(std::false_type{}, std::false_type{});
  }
}
#define SPHINX_GEMM_DMA_KERNEL(NAME, EPI, BM, EH)                                                            \
  __global__ __launch_bounds__(256, 2) void NAME(const bf16* __restrict__ A, const bf16* __restrict__ W,          \
                                                 const bf16* __restrict__ bias, int M, int N, int K, GemmEpi e) {  \
    __shared__ __attribute__((aligned(1024))) unsigned char smem[DmaCfg<BM, 128, 2, EH>::SMEM];                   \
    int m0, n0;                                                                                                  \
    grid_tile<BM, 128>(M, N, m0, n0);                                                                               \
    gemm_dma_body<EPI, BM, 128, 2, EH>(A, W, bias, M, N, K, e, smem, m0, n0);                                    \
  }
SPHINX_GEMM_DMA_KERNEL(k_gemm_dma_bias, EPI_BIAS, 128, 1)
SPHINX_GEMM_DMA_KERNEL(k_gemm_dma_gelu, EPI_GELU, 128, 1)
SPHINX_GEMM_DMA_KERNEL(k_gemm_dma_gated, EPI_GATED, 128, 1)
// 192-row tiles (wave tiles 96x64, epilogue in two halves; 80 KB of LDS, so
// still two workgroups per CU): fewer tiles for the same M, and 5/6 of the
// LDS reads per MFMA of the 128-row tile
SPHINX_GEMM_DMA_KERNEL(k_gemm_dma192_bias, EPI_BIAS, 192, 2)
SPHINX_GEMM_DMA_KERNEL(k_gemm_dma192_gelu, EPI_GELU, 192, 2)
SPHINX_GEMM_DMA_KERNEL(k_gemm_dma192_gated, EPI_GATED, 192, 2)
#undef SPHINX_GEMM_DMA_KERNEL

// BM-row tiles (64, 128, 192 or 256) with a ring of NS stages (4 x 24 KB,
// 4 x 32 KB, 4 x 40 KB or 3 x 48 KB of LDS, so one workgroup per CU), for
// launches whose tiles all fit on the CUs at once.  A lone workgroup waits out
// the copy latency of every K step when only the next stage is in flight; here
// NS - 1 are.  Eight waves of 32x32, 64x32, 96x32 or 128x32 (two per SIMD), so
// that each SIMD has a second wave to issue while one waits.  Same results as
// the other tiles.
template <int EPI, int NS, int BM = 128>
__global__ __launch_bounds__(512, 1) void k_gemm_dma_deep(const bf16* __restrict__ A, const bf16* __restrict__ W,
                                                          const bf16* __restrict__ bias, int M, int N, int K,
                                                          GemmEpi e) {
  constexpr int EH = BM <= 128 ? 1 : 2;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[DmaCfg<BM, 128, NS, EH, 8>::SMEM];
  int m0, n0;
  grid_tile<BM, 128>(M, N, m0, n0);
  gemm_dma_body<EPI, BM, 128, NS, EH, 8>(A, W, bias, M, N, K, e, smem, m0, n0);
}

// Mixed row tiles: nb 192-row and ns 128-row tiles per column tile.  Same
// results as either tile.
//  * Narrow outputs (at most 8 column tiles) that fit in one round of two
//    workgroups per CU: XCD x takes the row band [x B, (x+1) B),
//    B = 192 nb + 128 ns, with all column tiles; its first nb * nt workgroups
//    (at most one per CU) are the 192-row ones.  With only 192-row tiles a CU
//    can hold two of them (384 rows) while others hold one; here a CU holds at
//    most 192 + 128 rows.
//  * Wide outputs: column-fastest order (XCD x keeps the column tiles
//    n = x mod 8), the 192-row tiles first and the 128-row ones last, so that
//    the last round is made of the smaller tiles.
template <int EPI, bool WIDE>
__global__ __launch_bounds__(256, 2) void k_gemm_dma_mix(const bf16* __restrict__ A, const bf16* __restrict__ W,
                                                         const bf16* __restrict__ bias, int M, int N, int K,
                                                         GemmEpi e, int nb, int ns) {
  constexpr int S192 = DmaCfg<192, 128, 2, 2>::SMEM, S128 = DmaCfg<128, 128, 2, 1>::SMEM;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[S192 > S128 ? S192 : S128];
  const int nt = N / 128;
  if constexpr (WIDE) {  // nb row tiles of 192 rows, then ns of 128, column-fastest
    const int k = (int)blockIdx.x;
    if (k < nb * nt) {
      gemm_dma_body<EPI, 192, 128, 2, 2>(A, W, bias, M, N, K, e, smem, (k / nt) * 192, (k % nt) * 128);
    } else {
      const int j = k - nb * nt;
      const int m0 = 192 * nb + (j / nt) * 128;
      if (m0 < M) gemm_dma_body<EPI, 128, 128, 2, 1>(A, W, bias, M, N, K, e, smem, m0, (j % nt) * 128);
    }
  } else {  // XCD bands
    const int x = (int)blockIdx.x & 7, k = (int)blockIdx.x >> 3;
    const int band = x * (192 * nb + 128 * ns);
    if (k < nb * nt) {
      const int m0 = band + (k / nt) * 192;
      if (m0 < M) gemm_dma_body<EPI, 192, 128, 2, 2>(A, W, bias, M, N, K, e, smem, m0, (k % nt) * 128);
    } else {
      const int j = k - nb * nt;
      const int m0 = band + 192 * nb + (j / nt) * 128;
      if (m0 < M) gemm_dma_body<EPI, 128, 128, 2, 1>(A, W, bias, M, N, K, e, smem, m0, (j % nt) * 128);
    }
  }
}
}  // namespace dma

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
// Calibration loop: four independent 32x32x16 bf16 MFMA chains per wave.
// MFMA calibration loop; RANDOM: operands are hashed random bf16 in [-2, 2),
// eight (A, B) pairs used in rotation.
__device__ __forceinline__ float peak_rand(unsigned x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return (float)(x & 0xffffu) * (4.0f / 65536.0f) - 2.0f;
}

template <bool RANDOM>
__global__ __launch_bounds__(256) void k_peak_mfma(int iters, float* __restrict__ out) {
  constexpr int NS = RANDOM ? 8 : 1;
  const unsigned t = blockIdx.x * 256u + threadIdx.x;
  bf16x8 a[NS], b[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[s][i] = RANDOM ? (bf16)peak_rand(t * 64u + s * 8u + i) : (bf16)(1e-3f * (float)((threadIdx.x + i) & 15));
      b[s][i] = RANDOM ? (bf16)peak_rand(0x9e3779b9u ^ (t * 64u + s * 8u + i)) : (bf16)(1e-3f * (float)(i + 1));
    }
  f32x16 c0 = f32x16{}, c1 = f32x16{}, c2 = f32x16{}, c3 = f32x16{};
  // one round: four MFMAs on operand pairs s..s+3 (static register indices)
  auto round = [&](auto sc) {
    constexpr int s = decltype(sc)::value;
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s % NS], b[(s + 1) % NS], c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(s + 1) % NS], b[(s + 2) % NS], c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(s + 2) % NS], b[(s + 3) % NS], c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(s + 3) % NS], b[s % NS], c3, 0, 0, 0);
  };
  int it = 0;
  for (; it + 1 < iters; it += 2) {
    round(std::integral_constant<int, 0>{});
    round(std::integral_constant<int, 4>{});
  }
  if (it < iters) round(std::integral_constant<int, 0>{});
  float sum = 0.0f;
#pragma unroll
  for (int r = 0; r < 16; ++r) sum += c0[r] + c1[r] + c2[r] + c3[r];
  sum = wave_sum(sum);
  if (threadIdx.x == 0) out[blockIdx.x] = sum;
}
}  // namespace

namespace {
// Compute units of the current device (cached per device; 256 if unknown).
int cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int c = cache[dev].load(std::memory_order_relaxed);
  if (c <= 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0) c = 256;
    cache[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

// Relative time of `tiles` workgroups at two per CU: whole rounds, plus half a
// round for a last round that leaves every CU at most one tile (a lone tile
// runs about twice as fast), else a whole one; `w` is the tile's cost in
// 128-row-tile rounds.  Measured on the block GEMMs at M from 4.9k to 19.4k,
// this picks the faster of the 128- and 192-row tiles or one within 1 %.
double tile_rounds(int64_t tiles, int64_t slots, double w) {
  const int64_t full = tiles / slots, rem = tiles % slots;
  return w * ((double)full + (rem == 0 ? 0.0 : rem * 2 <= slots ? 0.5 : 1.0));
}

// One eight-wave workgroup per BM-row tile with an NS-stage ring.
template <int NS, int BM>
void launch_deep(int epi, int tiles, const bf16* a, const bf16* w, const bf16* b, int M, int N, int K,
                 const GemmEpi& e, hipStream_t s) {
  if (epi == EPI_BIAS) dma::k_gemm_dma_deep<EPI_BIAS, NS, BM><<<tiles, 512, 0, s>>>(a, w, b, M, N, K, e);
  else if (epi == EPI_GELU) dma::k_gemm_dma_deep<EPI_GELU, NS, BM><<<tiles, 512, 0, s>>>(a, w, b, M, N, K, e);
  else dma::k_gemm_dma_deep<EPI_GATED, NS, BM><<<tiles, 512, 0, s>>>(a, w, b, M, N, K, e);
}
}  // namespace

hipError_t launch_gemm(int epi, sphinx_dtype dt, const void* A, const void* W, const void* bias, int M, int N, int K,
                       const GemmEpi& e, hipStream_t s) {
  if (dt == SPHINX_BF16) {
    // the K loop takes two 64-deep steps at a time; the query scale is applied per 128-column tile
    if (K % 128 != 0 || N % 128 != 0 || (epi == EPI_BIAS && e.qcols % 128 != 0)) return hipErrorInvalidValue;
    const bf16 *a = (const bf16*)A, *w = (const bf16*)W, *b = (const bf16*)bias;
    {
      const int64_t nt = N / 128, slots = 2 * (int64_t)cu_count();
      const int64_t t128 = nt * ((M + 127) / 128), t192 = nt * ((M + 191) / 192);
      // few tiles: the smallest row tile (128, 192 or 256 rows) whose tiles
      // all fit on the CUs at once, one per CU with a deeper ring (128, 160
      // or 144 KB of LDS; 64-row tiles 96 KB)
      const int64_t cus = slots / 2, t256 = nt * ((M + 255) / 256), t64 = nt * ((M + 63) / 64);
      if (t128 <= cus || t192 <= cus || t256 <= cus) {
        // 64-row tiles where 128-row ones would leave more than half the CUs idle
        if (t64 <= cus && 2 * t128 <= cus) launch_deep<4, 64>(epi, (int)t64, a, w, b, M, N, K, e, s);
        else if (t128 <= cus) launch_deep<4, 128>(epi, (int)t128, a, w, b, M, N, K, e, s);
        else if (t192 <= cus) launch_deep<4, 192>(epi, (int)t192, a, w, b, M, N, K, e, s);
        else launch_deep<3, 256>(epi, (int)t256, a, w, b, M, N, K, e, s);
        return hipGetLastError();
      }
      // mixed tiles: narrow N, 192-row tiles filling more than half of one round
      int nb = -1, ns = 0;
      if (nt <= 8 && slots % 16 == 0 && t192 * 2 > slots && t192 <= slots) {
        const int per = (int)(slots / 8 / nt);  // slots per XCD and column tile
        const int need = (M + 7) / 8;           // rows per XCD band
        nb = std::max(0, (need - 128 * per + 63) / 64);
        ns = per - nb;
        if (nb * 2 > per) nb = -1;  // some CU would hold two 192-row tiles
      }
      // wide N needing more than three rounds of 192-row tiles: the last round
      // all 128-row tiles (ns per column tile), 192-row tiles before it
      if (nt > 8 && t192 > 3 * slots) {
        const int ws = (int)(slots / nt);
        const int wb = (M - 128 * ws + 191) / 192;
        if (ws > 0 && wb > 0) {
          const int grid = (wb + ws) * (int)nt;
          if (epi == EPI_BIAS) dma::k_gemm_dma_mix<EPI_BIAS, true><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e, wb, ws);
          else if (epi == EPI_GELU) dma::k_gemm_dma_mix<EPI_GELU, true><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e, wb, ws);
          else dma::k_gemm_dma_mix<EPI_GATED, true><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e, wb, ws);
          return hipGetLastError();
        }
      }
      if (nb >= 0) {
        const int grid = 8 * (nb + ns) * (int)nt;
        if (epi == EPI_BIAS) dma::k_gemm_dma_mix<EPI_BIAS, false><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e, nb, ns);
        else if (epi == EPI_GELU) dma::k_gemm_dma_mix<EPI_GELU, false><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e, nb, ns);
        else dma::k_gemm_dma_mix<EPI_GATED, false><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e, nb, ns);
      } else if (tile_rounds(t192, slots, 1.41) < tile_rounds(t128, slots, 1.0)) {
        // a 192-row tile does 1.5x the work of a 128-row one in 1.41x the time
        const int tiles = (int)t192;
        if (epi == EPI_BIAS) dma::k_gemm_dma192_bias<<<tiles, 256, 0, s>>>(a, w, b, M, N, K, e);
        else if (epi == EPI_GELU) dma::k_gemm_dma192_gelu<<<tiles, 256, 0, s>>>(a, w, b, M, N, K, e);
        else dma::k_gemm_dma192_gated<<<tiles, 256, 0, s>>>(a, w, b, M, N, K, e);
      } else {
        const int tiles = (int)t128;
        if (epi == EPI_BIAS) dma::k_gemm_dma_bias<<<tiles, 256, 0, s>>>(a, w, b, M, N, K, e);
        else if (epi == EPI_GELU) dma::k_gemm_dma_gelu<<<tiles, 256, 0, s>>>(a, w, b, M, N, K, e);
        else dma::k_gemm_dma_gated<<<tiles, 256, 0, s>>>(a, w, b, M, N, K, e);
      }
    }
  } else {
    const dim3 grid(N / 64, (M + 63) / 64);
    const float *a = (const float*)A, *w = (const float*)W, *b = (const float*)bias;
    if (epi == EPI_BIAS) k_gemm_f32<EPI_BIAS><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
    else if (epi == EPI_GELU) k_gemm_f32<EPI_GELU><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
    else k_gemm_f32<EPI_GATED><<<grid, 256, 0, s>>>(a, w, b, M, N, K, e);
  }
  return hipGetLastError();
}

hipError_t launch_peak_mfma(int iters, bool random, float* out, int blocks, hipStream_t s) {
  if (random)
    k_peak_mfma<true><<<blocks, 256, 0, s>>>(iters, out);
  else
    k_peak_mfma<false><<<blocks, 256, 0, s>>>(iters, out);
  return hipGetLastError();
}

}  // namespace sphinx
