// Varlen non-causal attention over the selected tokens of each request
// (joint spatio-temporal attention of the denoiser blocks restricted to the
// gathered tokens, Sec. 5.3 / Alg. 1 partial_step on the masked tokens).
//
// bf16 path, head_dim 64 or 72, gfx950 MFMA (flash-attention style, online softmax):
//  * one workgroup = 128 queries of one segment and one head, 4 waves x 32
//    queries; K/V tiles of 64 keys are copied global->LDS directly;
//  * scores are computed transposed, S^T = K Q^T with v_mfma_f32_32x32x16_bf16:
//    every lane then owns one query and 16 of each 32 keys, so the row max and
//    row sum need no cross-lane traffic except one exchange with lane^32;
//  * P^T stays in registers and is fed directly as the B operand of
//    O^T = V^T P^T; the V^T fragments come from LDS transpose reads in the
//    key order of the P^T k-slots;
//  * the output O^T lands with the query on the lane, so the final 1/l
//    normalisation is lane-local;
//  * softmax in base 2: q arrives from the QKV projection already multiplied
//    by log2(e)/sqrt(d) (rounded to bf16 once, after the scale);
//    the running max starts at zero (when the first tile's maxima are
//    moderate) or at the first tile's, and is only moved (and O, l rescaled)
//    when a tile's probabilities would sum past 2^64, so no tile max is
//    computed in the common case; P is rounded to bf16 for the PV
//    product and the row sum adds the same rounded values (v_dot2 with ones);
//  * only the last key tile of a segment is masked.
// Workgroups of the longest segment are scheduled first, and the linear
// workgroup order is remapped so that each XCD works on whole heads.
// head_dim 72 pads QK^T with one 8-deep k-step and computes O^T in three
// 32-row blocks (rows 72..95 are dropped).  Both head dims run the
// software-pipelined kernels k_attn_bf16_dma and k_attn_bf16_dma72 (described
// with their code).  Row bases are 64-bit and per-lane copy offsets stay
// within one 64-key tile, so any segment the ABI accepts is addressable.
//
// fp32 path (fp32 models, head_dim <= 64): one thread per (query, head).

#include <type_traits>

#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int AQ = 128;  // queries per workgroup
constexpr int AK = 64;   // keys per LDS tile
// A tile's probabilities are exp2 of its scores minus the running max, with
// no per-tile max in the common case; the max is moved (and O, l rescaled)
// only when a tile's row sum of probabilities exceeds this bound, so every
// probability stays below 2^64 and every accumulator far from overflow.
constexpr float kPsumMax = 18446744073709551616.0f;  // 2^64
static_assert(AQ == kAttnQueryTile, "host tile size must match the kernel");

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Three-way max as one instruction.  Written out because the compiler
// otherwise first quiets each MFMA result that enters a two-operand max (an
// extra instruction per value); scores are never signalling NaNs.
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

__device__ __forceinline__ float max_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max3(__uint_as_float(r[0]), __uint_as_float(r[1]), __uint_as_float(r[1]));
}

// Scores of keys at or past L set to -inf (scores s0: keys 0..31, s1: keys
// 32..63 of the tile starting at key kbase, slot r = key 8*(r/4) + 4*g + r%4).
__device__ __forceinline__ void mask_tail(f32x16& s0, f32x16& s1, int g, int kbase, int L) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int key = kbase + (r >> 2) * 8 + g * 4 + (r & 3);
    if (key >= L) s0[r] = -INFINITY;
    if (key + 32 >= L) s1[r] = -INFINITY;
  }
}

// Row max of one 64-key tile (lanes l and l^32 hold the two halves of the
// same query's keys).  With MASK, keys past L are set to -inf first.
template <bool MASK>
__device__ __forceinline__ float tile_max(f32x16& s0, f32x16& s1, int g, int kbase, int L) {
  if (MASK) mask_tail(s0, s1, g, kbase, L);
  // four independent chains of four max3 over the 32 values, then one max3 and a max
  float m4[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float t = max3(s0[4 * q], s0[4 * q + 1], s0[4 * q + 2]);
    t = max3(t, s0[4 * q + 3], s1[4 * q]);
    t = max3(t, s1[4 * q + 1], s1[4 * q + 2]);
    m4[q] = t;
  }
  const float m = max3(max3(m4[0], m4[1], s1[3]), max3(m4[2], m4[3], s1[7]), max3(s1[11], s1[15], s1[15]));
  return max_across_halves(m);
}

// ---------------------------------------------------------------------------
// head_dim 64, software-pipelined, with direct global->LDS copies
// (global_load_lds_dwordx4) and the LDS transpose read (ds_read_b64_tr_b16).
//  * Iteration t of the key loop issues QK(t+1) (8 MFMAs on the next K tile)
//    and PV(t-1) (8 MFMAs with the probabilities kept from the previous
//    iteration) while computing the softmax of tile t, whose scores came from
//    the previous iteration.  Neither MFMA group depends on that softmax, so
//    the region is one straight-line block: all fragment reads first, then 16
//    steps of one MFMA and one pair of probabilities, fenced so the compiler
//    keeps the order.
//  * K and V tiles are stored unpadded, 64 rows of 128 B, with the 16-byte
//    chunks of row r permuted: K chunk c at c ^ ((r >> 1) & 7), V chunk c at
//    c ^ 2(r & 3).  LDS has 64 four-byte banks and serves a 16-byte read to 16
//    lanes per pass; a 128-byte row covers half the banks, so the 16 rows of
//    one ds_read_b128 pass (same chunk) must spread over both halves and all
//    eight chunk slots, which the K permutation does; the V permutation does
//    the same for the four rows of each transpose-read lane group.
//  * Each wave copies 8 rows per instruction: lane i of copy n writes the 16
//    bytes at row 8(2w + n) + i/8, slot i%8 of the tile and reads them from
//    the global chunk that the permutation puts there: no registers, no LDS
//    stores and no VALU transposition.
//  * The V^T A fragment of a 32-row block db is two transpose reads: within a
//    16-lane group, output lane i gets element i%4 of what input lane
//    4e + i/4 addressed, so input lane j addresses V row (key) 4g + j/4 (+8
//    for the second read) at d = 32 db + 16 (b & 1) + 4 (j % 4), b = lane/16;
//    this gives each lane the 8 keys of its P^T k-slots for d = 32 db + l%32.
//  * Tiles live in 3-slot rings: the copies issued in iteration t land by the
//    end of iteration t+1 (a per-wave vmcnt wait that leaves the newest copies
//    in flight, then the workgroup barrier; no memory fence).
namespace dma {
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
constexpr int kRing = 3;  // tiles in flight per operand

// Tile geometry per head dimension.  head_dim 64: 128-byte rows, PV in two
// 32-row blocks of O^T, QK in four 16-deep k-steps.  head_dim 72: 144-byte
// rows (nine 16-byte chunks; nine is odd, so the 16 rows of a read pass fall
// on 16 different bank groups without a swizzle), PV in three blocks (rows
// 72..95 of the third are computed and dropped), QK in four 16-deep k-steps
// and one 8-deep k-step (dims 64..71, v_mfma_f32_32x32x8_bf16).
template <int HD>
struct Geo;
template <>
struct Geo<64> {
  static constexpr int RB = 128, DB = 2, NPV = 8, NQK = 8, TILE = AK * RB, PAD = 0, COPIES = 2, VR = 3;
};
template <>
struct Geo<72> {
  // PAD: a third-block V^T read of the last key row runs up to 40 bytes past
  // its tile (into dims that are dropped); the pad keeps it inside the ring.
  // VR: V ring of two slots (46 KB of LDS, three workgroups per CU); V(t) is
  // copied in the iteration before its PV and waited for at its end.
  static constexpr int RB = 144, DB = 3, NPV = 12, NQK = 10, TILE = AK * RB, PAD = 64, COPIES = 3, VR = 2;
};

template <int HD>
struct Smem {
  char k[kRing][Geo<HD>::TILE];
  char v[Geo<HD>::VR][Geo<HD>::TILE];
  char pad[Geo<HD>::PAD + 16];
};

// acc + p.x + p.y as one v_dot2c with (1, 1) in bf16.  A volatile statement,
// so that each step's dot product stays in its step: as plain arithmetic the
// compiler gathers the sixteen of a tile into one chain after the last MFMA.
__device__ __forceinline__ float rowsum_add(float acc, bf16x2 p) {
  asm volatile("v_dot2c_f32_bf16_e32 %0, 0x3f803f80, %1" : "+v"(acc) : "v"(__builtin_bit_cast(unsigned, p)));
  return acc;
}

__device__ __forceinline__ bf16x8 tr_pair(const char* p0, const char* p1) {
  const v4s a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)p0);
  const v4s b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)p1);
  const v4s r[2] = {a, b};
  return *reinterpret_cast<const bf16x8*>(r);
}

// Per-lane byte offsets inside a tile (loop invariant).
// head_dim 64: the swizzled chunk index only flips bits 5-6 of the K offset
// with the k-step and bit 6 of the V offset with the block, so one offset of
// each suffices.  head_dim 72: unswizzled, the k-step and the block add
// constants.
template <int HD>
struct LaneOff {
  int k0;  // QK A fragment of k-step 0, key rows 0..31 (rows 32..63: + 32 RB)
  int v0;  // PV A fragment of block 0, first transpose read (second: + 8 RB)
  __device__ int k(int ks) const { return HD == 64 ? k0 ^ (ks << 5) : k0 + 32 * ks; }
  __device__ int v(int db) const { return HD == 64 ? v0 ^ (db << 6) : v0 + 64 * db; }
  int k4o;  // head_dim 72, k-step 4 (8 deep): dims 64 + 4 g .. + 3 of key row r32
  __device__ int k4() const { return k4o; }
};

template <int HD>
__device__ __forceinline__ LaneOff<HD> lane_offsets(int lane) {
  LaneOff<HD> o;
  const int r32 = lane & 31, g = lane >> 5;
  const int j = lane & 15, b = lane >> 4;
  const int row = 4 * g + (j >> 2);
  const int byte = 32 * (b & 1) + 8 * (j & 3);
  if constexpr (HD == 64) {
    o.k0 = r32 * 128 + ((g ^ ((r32 >> 1) & 7)) << 4);  // chunk 2 ks + g, XOR-swizzled by row pair
    const int chunk = (byte >> 4) ^ (2 * (row & 3));
    o.v0 = row * 128 + (chunk << 4) + (byte & 8);
    o.k4o = 0;
  } else {
    o.k0 = r32 * 144 + 16 * g;  // chunk 2 ks + g
    o.v0 = row * 144 + byte;
    o.k4o = r32 * 144 + 128 + 8 * g;
  }
  return o;
}

template <int HD>
__device__ __forceinline__ void qk(const char* sK, const LaneOff<HD>& lo, const bf16x8 (&qf)[4], const v4s& q4,
                                   f32x16& s0, f32x16& s1) {
  constexpr int RB = Geo<HD>::RB;
  s0 = f32x16{};
  s1 = f32x16{};
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(sK + lo.k(ks));
    const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(sK + lo.k(ks) + 32 * RB);
    s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[ks], s0, 0, 0, 0);
    s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[ks], s1, 0, 0, 0);
  }
  if constexpr (HD == 72) {
    const v4s k0 = *reinterpret_cast<const v4s*>(sK + lo.k4());
    const v4s k1 = *reinterpret_cast<const v4s*>(sK + lo.k4() + 32 * RB);
    s0 = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(k0, q4, s0, 0, 0, 0);
    s1 = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(k1, q4, s1, 0, 0, 0);
  }
}

// O^T += V^T P^T; P^T k-slot (g, j) of (kb, hf) is key 32 kb + 16 hf + 8 (j/4) + 4 g + j%4.
template <int HD>
__device__ __forceinline__ void pv(const char* sV, const LaneOff<HD>& lo, const bf16x8 (&pf)[2][2],
                                   f32x16 (&oacc)[Geo<HD>::DB]) {
  constexpr int RB = Geo<HD>::RB;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int db = 0; db < Geo<HD>::DB; ++db) {
        const char* p = sV + lo.v(db) + (32 * kb + 16 * hf) * RB;
        const bf16x8 vf = tr_pair(p, p + 8 * RB);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kb][hf], oacc[db], 0, 0, 0);
      }
}

// One iteration's MFMA work interleaved by hand with the softmax of the
// previous tile: one MFMA per step (PV(t-1) first: 8 steps at head_dim 64,
// 12 at 72; then QK(t+1), the head-dim k-steps of the two 32-key blocks
// alternately, from a zero accumulator) and, in the first 16 steps, softmax
// work on two
// consecutive probability
// pairs, software-pipelined so that no instruction of a step waits on another
// of the same step: the exponentials of pair st+1 and the bf16 pack and
// row-sum dot product of pair st.  PV first lets the previous probabilities
// die while the new ones are made, and the QK accumulators only come alive in
// the second half, which keeps the register footprint low enough for three
// waves per SIMD; so does reading the operand fragment of a step from LDS two
// steps ahead (a ring of three).  Each step is fenced so the compiler keeps
// the order.
// PV step st: probability block (kb, hf) and O^T block db.
template <int HD>
__device__ __forceinline__ void pv_step(int st, int& kb, int& hf, int& db) {
  if constexpr (HD == 64) {
    kb = st >> 2;
    hf = (st >> 1) & 1;
    db = st & 1;
  } else {
    kb = st / 6;
    hf = (st / 3) & 1;
    db = st % 3;
  }
}

template <int HD>
__device__ __forceinline__ bf16x8 step_frag(const char* sK, const char* sV, const LaneOff<HD>& lo, int st) {
  constexpr int RB = Geo<HD>::RB, NPV = Geo<HD>::NPV;
  if (st < NPV) {
    int kb, hf, db;
    pv_step<HD>(st, kb, hf, db);
    const char* p = sV + lo.v(db) + (32 * kb + 16 * hf) * RB;
    return tr_pair(p, p + 8 * RB);
  }
  const int ks = (st - NPV) >> 1;
  const int wofs = ((st - NPV) & 1) ? 32 * RB : 0;
  if (HD == 72 && ks == 4) {  // 8 deep: the low half carries the operand
    const v4s k = *reinterpret_cast<const v4s*>(sK + lo.k4() + wofs);
    const v4s r[2] = {k, k};
    return *reinterpret_cast<const bf16x8*>(r);
  }
  return *reinterpret_cast<const bf16x8*>(sK + lo.k(ks) + wofs);
}

template <int HD>
__device__ __forceinline__ void region(const char* sK, const char* sV, const LaneOff<HD>& lo,
                                       const bf16x8 (&qf)[4], const v4s& q4, const f32x16& c0,
                                       const f32x16& c1, float& psum_out, const bf16x8 (&pp)[2][2],
                                       bf16x8 (&pn)[2][2], f32x16& n0, f32x16& n1,
                                       f32x16 (&oacc)[Geo<HD>::DB]) {
  constexpr int NPV = Geo<HD>::NPV, NSTEP = NPV + Geo<HD>::NQK;
  bf16x8 fr[3];
  fr[0] = step_frag<HD>(sK, sV, lo, 0);
  fr[1] = step_frag<HD>(sK, sV, lo, 1);
  // pair st: score block w = st & 1 (c0 or c1), rows r, r+1 with r = 8 (st >> 3) + 2 ((st >> 1) & 3)
  auto score = [&](int st, int e) -> float {
    const int r = (st >> 3) * 8 + 2 * ((st >> 1) & 3) + e;
    return (st & 1) ? c1[r] : c0[r];
  };
  float ex[16][2];
#pragma unroll
  for (int e = 0; e < 2; ++e) ex[0][e] = fast_exp2(score(0, e));
  __builtin_amdgcn_sched_barrier(0);
  float psum = 0.0f;
  const f32x16 zero16 = {};
#pragma unroll
  for (int st = 0; st < NSTEP; ++st) {
    if (st + 2 < NSTEP) fr[(st + 2) % 3] = step_frag<HD>(sK, sV, lo, st + 2);
    if (st < NPV) {
      int kb, hf, db;
      pv_step<HD>(st, kb, hf, db);
      oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[st % 3], pp[kb][hf], oacc[db], 0, 0, 0);
    } else {
      // the first k-step accumulates from zero: the scores arrive unshifted
      const int ks = (st - NPV) >> 1;
      if (HD == 72 && ks == 4) {
        const v4s a = *reinterpret_cast<const v4s*>(&fr[st % 3]);
        if ((st - NPV) & 1)
          n1 = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(a, q4, n1, 0, 0, 0);
        else
          n0 = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(a, q4, n0, 0, 0, 0);
      } else if ((st - NPV) & 1) {
        n1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[st % 3], qf[ks], ks == 0 ? zero16 : n1, 0, 0, 0);
      } else {
        n0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[st % 3], qf[ks], ks == 0 ? zero16 : n0, 0, 0, 0);
      }
    }
    if (st + 1 < 16)
#pragma unroll
      for (int e = 0; e < 2; ++e) ex[st + 1][e] = fast_exp2(score(st + 1, e));
    if (st < 16) {
      const int hf = st >> 3, i = (st >> 1) & 3, w = st & 1;
      bf16x2 pr;
      pr[0] = (bf16)ex[st][0];
      pr[1] = (bf16)ex[st][1];
      psum = rowsum_add(psum, pr);
      pn[w][hf][2 * i] = pr[0];
      pn[w][hf][2 * i + 1] = pr[1];
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  // Pin the probabilities here: otherwise the compiler sinks their whole
  // computation past the next iteration's branches, next to their use,
  // undoing the interleaving with this iteration's MFMAs.
#pragma unroll
  for (int w = 0; w < 2; ++w)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) asm volatile("" : "+v"(pn[w][hf]));
  asm volatile("" : "+v"(psum));
  psum_out = psum;
}

// Probabilities exp2(s - delta) of a tile's shifted scores, rounded to bf16 in
// P^T operand order; returns their row sum (of the rounded values).
__device__ __forceinline__ float probs(const f32x16& s0, const f32x16& s1, float delta, bf16x8 (&pf)[2][2]) {
  const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
  float psum = 0.0f;
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = hf * 8 + 2 * i;
      bf16x2 a, b;
      a[0] = (bf16)fast_exp2(s0[r] - delta);
      a[1] = (bf16)fast_exp2(s0[r + 1] - delta);
      b[0] = (bf16)fast_exp2(s1[r] - delta);
      b[1] = (bf16)fast_exp2(s1[r + 1] - delta);
      psum = __builtin_amdgcn_fdot2_f32_bf16(a, ones, psum, false);
      psum = __builtin_amdgcn_fdot2_f32_bf16(b, ones, psum, false);
      pf[0][hf][2 * i] = a[0];
      pf[0][hf][2 * i + 1] = a[1];
      pf[1][hf][2 * i] = b[0];
      pf[1][hf][2 * i + 1] = b[1];
    }
  return psum;
}
}  // namespace dma

template <int HD>
__device__ __forceinline__ void attn_body_dma(const AttnIO& io, int D, int heads, const SegTable& S,
                                              dma::Smem<HD>& sm) {
  typedef dma::Geo<HD> G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, r32 = lane & 31;
  const int ntiles = S.tile_prefix[S.nseg];
  const int work = ntiles * heads;
  // Workgroups are dealt to the 8 XCDs round-robin by linear id; renumbered so
  // that XCD x runs the contiguous units [x q, (x+1) q), i.e. whole heads, and
  // keeps a head's K and V in its L2.
  int lid = (int)blockIdx.x;
  if (work % 8 == 0) lid = (lid & 7) * (work >> 3) + (lid >> 3);
  const int head = lid / ntiles, tile = lid - head * ntiles;
  int s = 0;
  while (s + 1 < S.nseg && S.tile_prefix[s + 1] <= tile) ++s;
  const int qt = tile - S.tile_prefix[s];
  const int seg0 = S.start[s], Lq = S.len[s];
  const int kv0 = S.kv_start[s], L = S.kv_len[s];  // L: keys of the segment
  const int ldq = io.ldq, ld = io.ldkv;
  const bf16x8 zero8 = {};

  // V buffer 2 (that of "tile -1") starts all zero: the first iteration's PV
  // multiplies it by zero probabilities.  (So does the pad behind it, which
  // third-block reads of head_dim 72 run into.)
  for (int i = tid; i < G::TILE / 16; i += 256) reinterpret_cast<bf16x8*>(sm.v[G::VR - 1])[i] = zero8;
  if (G::PAD > 0 && tid < (G::PAD + 16) / 16) reinterpret_cast<bf16x8*>(sm.pad)[tid] = zero8;

  const int ql = qt * AQ + wave * 32 + r32;
  bf16x8 qf[4];
  dma::v4s q4 = {};  // head_dim 72: dims 64 + 4 g .. + 3
  const bf16* Qg = static_cast<const bf16*>(io.q) + (int64_t)seg0 * ldq + head * HD;
  // q is stored scaled by log2(e)/sqrt(d): scores come out of the MFMAs in base-2 units
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
    qf[ks] = (ql < Lq) ? *reinterpret_cast<const bf16x8*>(Qg + (int64_t)ql * ldq + ks * 16 + g * 8) : zero8;
  if constexpr (HD == 72) {
    bf16x4 v = {};
    if (ql < Lq) v = *reinterpret_cast<const bf16x4*>(Qg + (int64_t)ql * ldq + 64 + g * 4);
    q4 = __builtin_bit_cast(dma::v4s, v);
  }


  // Copy sources.  head_dim 64: lane i of copy n (n = 0, 1) fills row
  // 8(2 wave + n) + i/8, slot i%8 of a tile.  head_dim 72: a wave fills rows
  // 16 wave .. +15, 144 chunks, chunk t = 64 n + i by copy n (n = 0, 1, 2; the
  // third copy with 16 lanes), at row t/9, slot t%9.  The tile's first key row
  // is a wave-uniform base address; each lane keeps its byte offset from it.
  // In a tile that runs past the segment's last key the rows past it repeat
  // that key.
  const bf16* Kg = static_cast<const bf16*>(io.k) + (int64_t)kv0 * ld + head * HD;
  const bf16* Vg = static_cast<const bf16*>(io.v) + (int64_t)kv0 * ld + head * HD;
  auto copy_row = [&](int n) {
    return HD == 64 ? 8 * (2 * wave + n) + (lane >> 3) : 16 * wave + (64 * n + lane) / 9;
  };
  auto k_chunk = [&](int row) { return (lane & 7) ^ ((row >> 1) & 7); };
  auto v_chunk = [&](int row) { return (lane & 7) ^ (2 * (row & 3)); };
  auto chunk72 = [&](int n) { return (64 * n + lane) % 9; };
  auto active = [&](int n) { return HD == 64 || n < 2 || lane < 16; };
  auto dst = [&](char* tile, int n) {
    return HD == 64 ? tile + (2 * wave + n) * 1024 : tile + wave * 2304 + n * 1024;
  };
  uint32_t koff[G::COPIES], voff;
#pragma unroll
  for (int n = 0; n < G::COPIES; ++n) {
    const int row = copy_row(n);
    koff[n] = 2u * (uint32_t)(row * ld + (HD == 64 ? k_chunk(row) : chunk72(n)) * 8);
  }
  voff = 2u * (uint32_t)(copy_row(0) * ld + v_chunk(copy_row(0)) * 8);  // head_dim 64; copy 1: 8 rows on
  auto copy_k = [&](int kbase, int buf) {
    const bf16* base = Kg + (int64_t)kbase * ld;
    if (kbase + AK <= L) {
#pragma unroll
      for (int n = 0; n < G::COPIES; ++n)
        if (active(n)) lds_dma16_at(base, koff[n], dst(sm.k[buf], n));
    } else {
#pragma unroll
      for (int n = 0; n < G::COPIES; ++n) {
        const int row = copy_row(n);
        const int c = HD == 64 ? k_chunk(row) : chunk72(n);
        const uint32_t off = 2u * (uint32_t)(min(row, L - 1 - kbase) * ld + c * 8);
        if (active(n)) lds_dma16_at(base, off, dst(sm.k[buf], n));
      }
    }
  };
  auto copy_v = [&](int kbase, int buf) {
    const bf16* base = Vg + (int64_t)kbase * ld;
    if (kbase + AK <= L) {
#pragma unroll
      for (int n = 0; n < G::COPIES; ++n) {
        if constexpr (HD == 64)
          lds_dma16_at(base + n * 8 * ld, voff, dst(sm.v[buf], n));
        else if (active(n))
          lds_dma16_at(base, koff[n], dst(sm.v[buf], n));  // same layout as K
      }
    } else {
#pragma unroll
      for (int n = 0; n < G::COPIES; ++n) {
        const int row = copy_row(n);
        const int c = HD == 64 ? v_chunk(row) : chunk72(n);
        const uint32_t off = 2u * (uint32_t)(min(row, L - 1 - kbase) * ld + c * 8);
        if (active(n)) lds_dma16_at(base, off, dst(sm.v[buf], n));
      }
    }
  };
  // Barrier after this wave's LDS operations and all but its newest `keep`
  // copies (the copies issued in the current iteration stay in flight); no
  // memory fence is needed beyond that (the LDS reads of the iteration have
  // all been consumed by MFMAs).  The empty asm statements keep the compiler
  // from moving memory operations across the barrier.
  auto land = [&](auto keep) {
    if (decltype(keep)::value == 4)
      __builtin_amdgcn_s_waitcnt(0x0074);  // vmcnt(4) lgkmcnt(0)
    else if (decltype(keep)::value == 3)
      __builtin_amdgcn_s_waitcnt(0x0073);  // vmcnt(3) lgkmcnt(0)
    else if (decltype(keep)::value == 6)
      __builtin_amdgcn_s_waitcnt(0x0076);  // vmcnt(6) lgkmcnt(0)
    else
      __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  // copies that stay in flight at the end of an iteration: head_dim 64 both
  // of its copies (K(t+3), V(t+1)), head_dim 72 only K(t+3) (V(t) is needed
  // in the next iteration)
  using Keep4 = std::integral_constant<int, HD == 64 ? 4 : 3>;
  using Keep0 = std::integral_constant<int, 0>;

  const dma::LaneOff<HD> lo = dma::lane_offsets<HD>(lane);
  f32x16 oacc[G::DB];
#pragma unroll
  for (int db = 0; db < G::DB; ++db) oacc[db] = f32x16{};
  float m_run, l_run = 0.0f;
  const int nkt = (L + AK - 1) / AK;

  // Tile j of K and of V lives in ring slot j % 3.  Iteration t: softmax of
  // tile t, QK(t+1), PV(t-1); copies K(t+3) (clamped to the last tile: a
  // harmless duplicate near the end) and V(t+1), which land by the end of
  // iteration t+1.
  int slot = 0;  // t % 3
  // No per-tile max: a tile's probabilities are exp2 of its scores minus the
  // running max.  Only when a tile's row sum exceeds kPsumMax (some score
  // more than about 64 above the running max) does `rebase` move the max to
  // the tile's, rescale O (which then holds the tiles up to t-1) and l, and
  // recompute the tile's probabilities.  QK accumulates from zero.  A wave
  // whose first-tile maxima all lie in [-64, 32] keeps the running max at
  // zero (exp2 of such scores neither overflows nor loses the row sum to
  // underflow), so its probabilities are exp2 of the MFMA output with no
  // further arithmetic.  Otherwise, and after a rebase, the wave is `shifted`
  // (wave-uniform): each tile's scores have the running max subtracted
  // before their exponentials.
  bool shifted = false;
  // The scores of one 32-key block w of tile t once more, shifted by the
  // current max (rare path: the tile's score registers are reused as soon as
  // its probabilities are made, and a loop tile's K slot in LDS is refilled by
  // then).  K rows are read from global memory in the fragment layout of the
  // LDS reads (row r32 of the block, dims 16 ks + 8 g .. + 7; head_dim 72:
  // dims 64 + 4 g .. + 3 for the 8-deep step).  Rows past the segment repeat
  // its last key and their scores are masked.
  auto rescore = [&](int t, int w) -> f32x16 {
    const int key = t * AK + 32 * w + r32;
    const bf16* row = Kg + (int64_t)min(key, L - 1) * ld;
    f32x16 c = f32x16{};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(row + ks * 16 + g * 8), qf[ks], c,
                                                  0, 0, 0);
    if constexpr (HD == 72)
      c = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(*reinterpret_cast<const dma::v4s*>(row + 64 + g * 4), q4, c, 0, 0,
                                                    0);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int k = t * AK + 32 * w + (r >> 2) * 8 + g * 4 + (r & 3);
      c[r] = k < L ? c[r] - m_run : -INFINITY;
    }
    return c;
  };
  // Rebase for tile t, whose probabilities passed the bound: the running max
  // moves to the tile's max where that is larger, O (which then holds the tiles
  // up to t-1) and l are rescaled, and the tile's probabilities are made again
  // from rescored scores, one 32-key block at a time.  Returns their row sum.
  auto rebase = [&](int t, bf16x8 (&pf)[2][2]) -> float {
    float mx = -INFINITY;
#pragma unroll 1
    for (int w = 0; w < 2; ++w) {  // one block at a time: few registers on this rare path
      const f32x16 c = rescore(t, w);
#pragma unroll
      for (int r = 0; r < 16; r += 2) mx = max3(mx, c[r], c[r + 1]);
    }
    mx = max_across_halves(mx);  // the same in lanes l and l^32
    const float delta = mx > 0.0f ? mx : 0.0f;
    const float alpha = fast_exp2(-delta);
#pragma unroll
    for (int db = 0; db < G::DB; ++db) oacc[db] *= alpha;
    l_run *= alpha;
    m_run += delta;
    shifted = true;
    const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
    float psum = 0.0f;
    bf16x8 q0[2], q1[2];  // probabilities of blocks 0 and 1
#pragma unroll 1
    for (int w = 0; w < 2; ++w) {
      const f32x16 c = rescore(t, w);  // now shifted by the new max
      bf16x8 h[2];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          bf16x2 pr;
          pr[0] = (bf16)fast_exp2(c[hf * 8 + 2 * i]);
          pr[1] = (bf16)fast_exp2(c[hf * 8 + 2 * i + 1]);
          psum = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, psum, false);
          h[hf][2 * i] = pr[0];
          h[hf][2 * i + 1] = pr[1];
        }
      if (w == 0) {
        q0[0] = h[0];
        q0[1] = h[1];
      } else {
        q1[0] = h[0];
        q1[1] = h[1];
      }
    }
    pf[0][0] = q0[0];
    pf[0][1] = q0[1];
    pf[1][0] = q1[0];
    pf[1][1] = q1[1];
    return psum;
  };
  auto settle = [&](f32x16& c0, f32x16& c1) {  // what a tile's scores still owe
    if (shifted)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        c0[r] -= m_run;
        c1[r] -= m_run;
      }
  };
  // K6: t mod 6 when the caller knows it at compile time (then every ring slot
  // is a constant and the LDS addresses are immediate offsets from loop-invariant
  // lane bases), or -1 (slots from the running `slot`).
  auto iter = [&](int t, auto K6, f32x16& c0, f32x16& c1, f32x16& n0, f32x16& n1, bf16x8 (&pp)[2][2],
                  bf16x8 (&pn)[2][2]) {
    constexpr int k6 = decltype(K6)::value;
    const int sl = k6 >= 0 ? k6 % 3 : slot;       // t % 3
    const int par = k6 >= 0 ? k6 % 2 : (t & 1);   // t % 2
    const int s1 = sl == 2 ? 0 : sl + 1, s2 = sl == 0 ? 2 : sl - 1;  // (t+1) % 3, (t-1) % 3
    int vs;  // V slot of PV(t-1)
    if constexpr (HD == 64) {
      copy_k(min(t + 3, nkt - 1) * AK, sl);
      copy_v((t + 1) * AK, s1);
      vs = s2;
    } else {
      copy_v(t * AK, par);  // first, so that the end-of-iteration wait can leave K(t+3) in flight
      copy_k(min(t + 3, nkt - 1) * AK, sl);
      vs = par ^ 1;
    }
    settle(c0, c1);
    // head_dim 64: the wave in its MFMA region goes first, ahead of the
    // serial work of the other waves on its SIMD
    if constexpr (HD == 64) __builtin_amdgcn_s_setprio(1);
    float psum;
    dma::region<HD>(sm.k[s1], sm.v[vs], lo, qf, q4, c0, c1, psum, pp, pn, n0, n1, oacc);
    if constexpr (HD == 64) __builtin_amdgcn_s_setprio(0);
    if (__ballot(!(psum <= kPsumMax)) != 0) psum = rebase(t, pn);
    l_run += psum;
    land(Keep4{});
    slot = s1;
  };

  copy_k(0, 0);
  copy_k(min(1, nkt - 1) * AK, 1);
  copy_k(min(2, nkt - 1) * AK, 2);
  if constexpr (HD == 64) {
    copy_v(0, 0);
    land(Keep4{});  // K(0) and K(1) have landed
  } else {
    land(std::integral_constant<int, 6>{});  // K(0) has landed
  }
  f32x16 a0, a1, b0, b1;
  dma::qk<HD>(sm.k[0], lo, qf, q4, a0, a1);
  {  // the running max starts at zero or at tile 0's (keys past L masked);
     // tile 0's scores are settled like every other tile's
    const float m0 = tile_max<true>(a0, a1, g, 0, L);
    shifted = __ballot(!(m0 >= -64.0f && m0 <= 32.0f)) != 0;
    m_run = shifted ? m0 : 0.0f;
  }
  // iteration 0 copies K(3) into slot 0: every wave must be done reading K(0)
  // (and, at head_dim 72, K(1) must have landed)
  land(Keep4{});
  bf16x8 pa[2][2] = {{zero8, zero8}, {zero8, zero8}}, pb[2][2];
  using IC0 = std::integral_constant<int, 0>;
  using IC1 = std::integral_constant<int, 1>;
  using IC2 = std::integral_constant<int, 2>;
  using IC3 = std::integral_constant<int, 3>;
  using IC4 = std::integral_constant<int, 4>;
  using IC5 = std::integral_constant<int, 5>;
  using ICR = std::integral_constant<int, -1>;
  int t = 0;
  // head_dim 64: six tiles per trip, so both ring phases are known (t % 6 == 0
  // here): 348.8 -> 343.0 us at the headline.  At head_dim 72 the same unroll
  // gained nothing and pushed spills into the kernel, so it keeps two per trip.
  if constexpr (HD == 64) {
    for (; t + 6 < nkt; t += 6) {
      iter(t, IC0{}, a0, a1, b0, b1, pa, pb);
      iter(t + 1, IC1{}, b0, b1, a0, a1, pb, pa);
      iter(t + 2, IC2{}, a0, a1, b0, b1, pa, pb);
      iter(t + 3, IC3{}, b0, b1, a0, a1, pb, pa);
      iter(t + 4, IC4{}, a0, a1, b0, b1, pa, pb);
      iter(t + 5, IC5{}, b0, b1, a0, a1, pb, pa);
    }
  }
  for (; t + 2 < nkt; t += 2) {
    iter(t, ICR{}, a0, a1, b0, b1, pa, pb);
    iter(t + 1, ICR{}, b0, b1, a0, a1, pb, pa);
  }
  if (t + 1 < nkt) {
    iter(t, ICR{}, a0, a1, b0, b1, pa, pb);
    a0 = b0;
    a1 = b1;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) pa[kb][hf] = pb[kb][hf];
    ++t;
  }
  {  // last tile t = nkt - 1 (possibly partial); head_dim 64: V(t) was copied in iteration t-1
    int sprev, scur;
    if constexpr (HD == 64) {
      sprev = slot == 0 ? 2 : slot - 1;
      scur = slot;
    } else {
      copy_v(t * AK, t & 1);
      sprev = (t + 1) & 1;
      scur = t & 1;
    }
    settle(a0, a1);
    if (L % AK != 0) mask_tail(a0, a1, g, t * AK, L);
    float psum = dma::probs(a0, a1, 0.0f, pb);
    dma::pv<HD>(sm.v[sprev], lo, pa, oacc);  // PV(t-1) before a rebase, which rescales it too
    if (__ballot(!(psum <= kPsumMax)) != 0) psum = rebase(t, pb);
    l_run += psum;
    land(Keep0{});
    dma::pv<HD>(sm.v[scur], lo, pb, oacc);
  }
  l_run += __shfl_xor(l_run, 32, kWave);
  if (ql < Lq) {
    const float inv = 1.0f / l_run;
    bf16* orow = static_cast<bf16*>(io.o) + (int64_t)(seg0 + ql) * D + head * HD;
#pragma unroll
    for (int db = 0; db < G::DB; ++db)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr)
        if (db * 32 + rr * 8 < HD) {  // head_dim 72: of the third block only dims 64..71
          bf16x4 ov;
#pragma unroll
          for (int q = 0; q < 4; ++q) ov[q] = (bf16)(oacc[db][rr * 4 + q] * inv);
          *reinterpret_cast<bf16x4*>(orow + db * 32 + rr * 8 + g * 4) = ov;
        }
  }
}

__global__ __launch_bounds__(256, 3) void k_attn_bf16_dma(AttnIO io, int D, int heads, SegTable S) {
  __shared__ __attribute__((aligned(1024))) dma::Smem<64> sm;
  attn_body_dma<64>(io, D, heads, S, sm);
}

// head_dim 72: 46 KB of LDS, three workgroups per CU.
__global__ __launch_bounds__(256, 3) void k_attn_bf16_dma72(AttnIO io, int D, int heads, SegTable S) {
  __shared__ __attribute__((aligned(1024))) dma::Smem<72> sm;
  attn_body_dma<72>(io, D, heads, S, sm);
}

constexpr int kF32Max = 64;

// q is stored scaled by log2(e)/sqrt(d): base-2 online softmax.
__global__ __launch_bounds__(128) void k_attn_f32(AttnIO io, int D, int d, int heads, int n, SegTable S) {
  const int gid = blockIdx.x * 128 + threadIdx.x;
  if (gid >= n * heads) return;
  const int j = gid / heads, h = gid % heads;
  int s = 0;
  while (s + 1 < S.nseg && !(j >= S.start[s] && j < S.start[s] + S.len[s])) ++s;
  const int kv0 = S.kv_start[s], L = S.kv_len[s];
  const float* qp = static_cast<const float*>(io.q);
  const float* kp = static_cast<const float*>(io.k);
  const float* vp = static_cast<const float*>(io.v);
  float* o = static_cast<float*>(io.o);
  float q[kF32Max], acc[kF32Max];
#pragma unroll
  for (int c = 0; c < kF32Max; ++c) {
    q[c] = (c < d) ? qp[(int64_t)j * io.ldq + h * d + c] : 0.0f;
    acc[c] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  for (int t = kv0; t < kv0 + L; ++t) {
    const float* kr = kp + (int64_t)t * io.ldkv + h * d;
    const float* vr = vp + (int64_t)t * io.ldkv + h * d;
    float sc = 0.0f;
#pragma unroll
    for (int c = 0; c < kF32Max; ++c)
      if (c < d) sc = fmaf(q[c], kr[c], sc);
    const float mn = fmaxf(m, sc);
    const float corr = exp2f(m - mn);
    const float p = exp2f(sc - mn);
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

hipError_t launch_attention(sphinx_dtype dt, const AttnIO& io, int D, int heads, int head_dim, int n,
                            const SegTable& S, hipStream_t s) {
  if (dt == SPHINX_BF16) {
    const int grid = S.tile_prefix[S.nseg] * heads;
    if (head_dim == 64)
      k_attn_bf16_dma<<<grid, 256, 0, s>>>(io, D, heads, S);
    else
      k_attn_bf16_dma72<<<grid, 256, 0, s>>>(io, D, heads, S);
  } else {
    k_attn_f32<<<(n * heads + 127) / 128, 128, 0, s>>>(io, D, head_dim, heads, n, S);
  }
  return hipGetLastError();
}

}  // namespace sphinx

// ---------------------------------------------------------------------------
// Temporal attention of a factorised denoiser: the forwarded tokens at one
// (y, x) position of a request attend to each other across frames (to all of
// the request's frames at that position through the latent cache).  A column
// holds at most 64 tokens, so this is a few dot products per query: one
// workgroup per column (members found with one ballot), one wave per head,
// one lane per query.  Each wave stages its head's key and value rows in LDS
// in chunks with 16-byte loads; the lanes then read them as broadcasts.  fp32
// math with an online softmax in base 2 (q is stored scaled by
// log2(e)/sqrt(d)).
// ---------------------------------------------------------------------------
namespace sphinx {
namespace {

template <typename T>
struct TempVec;  // 16 bytes of a row as floats
template <>
struct TempVec<bf16> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void get(const bf16* p, float* o) {
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = (float)v[i];
  }
};
template <>
struct TempVec<float> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void get(const float* p, float* o) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = v[i];
  }
};

// HD: the head dimension when EXACT, else an upper bound with the runtime d
// (fp32 models); a multiple of the 16-byte vector.
template <typename T, int HD, bool EXACT>
__global__ __launch_bounds__(256) void k_attn_temporal(ReqTable RT, AttnIO io, int D, int d_rt, int heads,
                                                       const int32_t* __restrict__ pos, int cached) {
  constexpr int VN = TempVec<T>::N;             // elements per 16-byte vector
  constexpr int NV = HD / VN;                   // vectors per head row (upper bound)
  constexpr int KC = sizeof(T) == 2 ? 32 : 16;  // keys per staged chunk
  const int d = EXACT ? HD : d_rt;
  const int vpr = EXACT ? NV : d_rt / VN;
  __shared__ int rows[64];                    // forwarded row of each query member
  __shared__ int krows[64];                   // key rows (qkv rows, or cache token rows)
  __shared__ int nq_s, nk_s;
  __shared__ __attribute__((aligned(16))) T stage[4][2][KC * HD];
  int c = (int)blockIdx.x, r = 0;
  for (;; ++r) {
    const int cols = (RT.h[r] >> 1) * (RT.w[r] >> 1);
    if (c < cols || r + 1 == RT.R) break;
    c -= cols;
  }
  const int F = RT.frames[r];
  const int64_t tpf = (int64_t)(RT.h[r] >> 1) * (RT.w[r] >> 1);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (wave == 0) {  // members of the column in frame order
    int p = -1;
    int64_t t = 0;
    if (lane < F) {
      t = RT.tok_off[r] + lane * tpf + c;
      p = pos[t];
    }
    const uint64_t bq = __ballot(p >= 0);
    const int iq = __popcll(bq & ((1ull << lane) - 1ull));
    if (p >= 0) rows[iq] = p;
    if (cached) {
      if (lane < F) krows[lane] = (int)t;
    } else if (p >= 0) {
      krows[iq] = p;
    }
    if (lane == 0) {
      nq_s = __popcll(bq);
      nk_s = cached ? F : __popcll(bq);
    }
  }
  __syncthreads();
  const int nq = nq_s, nk = nk_s;
  if (nq == 0) return;
  const T* Q = static_cast<const T*>(io.q);
  const T* K = static_cast<const T*>(io.k);
  const T* V = static_cast<const T*>(io.v);
  T* O = static_cast<T*>(io.o);
  T* sk = stage[wave][0];
  T* sv = stage[wave][1];
  for (int h = wave; h < heads; h += 4) {
    float q[HD], acc[HD];
    const bool mine = lane < nq;
    const int qr = mine ? rows[lane] : rows[0];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      if (EXACT || v < vpr) TempVec<T>::get(Q + (int64_t)qr * io.ldq + h * d + v * VN, q + v * VN);
      else
#pragma unroll
        for (int i = 0; i < VN; ++i) q[v * VN + i] = 0.0f;
    }
#pragma unroll
    for (int e = 0; e < HD; ++e) acc[e] = 0.0f;
    float m = -INFINITY, l = 0.0f;
    for (int k0 = 0; k0 < nk; k0 += KC) {
      const int cnt = min(KC, nk - k0);
      // this wave's chunk of key and value rows into LDS (16-byte copies)
      for (int i = lane; i < cnt * vpr; i += kWave) {
        const int row = i / vpr, v = i - row * vpr;
        const int64_t src = (int64_t)krows[k0 + row] * io.ldkv + h * d + v * VN;
        *reinterpret_cast<uint4*>(sk + row * HD + v * VN) = *reinterpret_cast<const uint4*>(K + src);
        *reinterpret_cast<uint4*>(sv + row * HD + v * VN) = *reinterpret_cast<const uint4*>(V + src);
      }
      __builtin_amdgcn_s_waitcnt(0);  // the wave's own LDS writes are complete (lockstep wave)
      asm volatile("" ::: "memory");
      if (mine) {
        for (int j = 0; j < cnt; ++j) {
          float part[4] = {0.0f, 0.0f, 0.0f, 0.0f};  // independent partial dot products
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            if (EXACT || v < vpr) {
              float kv[VN];
              TempVec<T>::get(sk + j * HD + v * VN, kv);
#pragma unroll
              for (int i = 0; i < VN; ++i) part[i & 3] = fmaf(q[v * VN + i], kv[i], part[i & 3]);
            }
          }
          const float sc = (part[0] + part[1]) + (part[2] + part[3]);
          const float mn = fmaxf(m, sc);
          const float corr = exp2f(m - mn), p = exp2f(sc - mn);
          l = fmaf(l, corr, p);
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            if (EXACT || v < vpr) {
              float vv[VN];
              TempVec<T>::get(sv + j * HD + v * VN, vv);
#pragma unroll
              for (int i = 0; i < VN; ++i) acc[v * VN + i] = fmaf(acc[v * VN + i], corr, p * vv[i]);
            }
          }
          m = mn;
        }
      }
      asm volatile("" ::: "memory");
    }
    if (mine) {
      const float inv = 1.0f / l;
      T* orow = O + (int64_t)qr * D + h * d;
#pragma unroll
      for (int e = 0; e < HD; ++e)
        if (EXACT || e < d) orow[e] = (T)(acc[e] * inv);
    }
  }
}
}  // namespace
namespace {
// Sum over the LPH consecutive lanes of a head (LPH = 4 or 8): quad
// permutations through DPP, then one exchange with lane ^ 4.
template <int LPH>
__device__ __forceinline__ float head_sum(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, true));  // l ^ 1
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x4E, 0xF, 0xF, true));  // l ^ 2
  if constexpr (LPH == 8) x += __shfl_xor(x, 4, kWave);
  return x;
}

// The same temporal attention for bf16 rows of D = 64 DPL elements and heads
// of 64 dims, LPH = 64 / heads lanes each (D 1024: 16 heads of 4 lanes; D 512:
// 8 heads of 8 lanes): one wave per column, lane l owning dims
// [DPL l, DPL (l + 1)) of every row, so that a row is one coalesced wave load.
// A score is the lanes' DPL-wide partial dot products (bf16 pairs, fp32 sums)
// summed over the head's lanes.  Queries go in chunks of four that share each
// key's loads; fp32 online softmax in base 2 (q is stored scaled by
// log2(e)/sqrt(d)).  Members and key rows are read from the lanes that found
// them (readlane with the wave-uniform frame index).
template <int DPL, int LPH>
__global__ __launch_bounds__(256) void k_attn_temporal_lanes(ReqTable RT, AttnIO io, int D,
                                                             const int32_t* __restrict__ pos, int cached, int ncols) {
  static_assert(DPL == 8 || DPL == 16, "8 or 16 dims per lane");
  constexpr int NV = DPL / 8;  // 16-byte vectors per lane and row
  const int lane = threadIdx.x & 63;
  int c = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  if (c >= ncols) return;  // wave-uniform; the kernel has no barrier
  int r = 0;
  for (;; ++r) {
    const int cols = (RT.h[r] >> 1) * (RT.w[r] >> 1);
    if (c < cols || r + 1 == RT.R) break;
    c -= cols;
  }
  const int F = RT.frames[r];
  const int64_t tpf = (int64_t)(RT.h[r] >> 1) * (RT.w[r] >> 1);
  int p = -1, kr = 0;  // lane f < F: forwarded row of frame f's token, and its key row
  if (lane < F) {
    const int64_t t = RT.tok_off[r] + lane * tpf + c;
    p = pos[t];
    kr = cached ? (int)t : p;
  }
  const uint64_t qmask = __ballot(p >= 0);
  if (qmask == 0) return;
  const uint64_t kmask = cached ? (F >= 64 ? ~0ull : (1ull << F) - 1ull) : qmask;
  const bf16* Q = static_cast<const bf16*>(io.q) + lane * DPL;
  const bf16* K = static_cast<const bf16*>(io.k) + lane * DPL;
  const bf16* V = static_cast<const bf16*>(io.v) + lane * DPL;
  bf16* O = static_cast<bf16*>(io.o) + lane * DPL;
  uint64_t qm = qmask;
  while (qm != 0) {  // chunks of up to four queries
    int qrow[4], nqc = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (qm != 0) {
        qrow[u] = __builtin_amdgcn_readlane(p, __builtin_ctzll(qm));
        qm &= qm - 1;
        nqc = u + 1;
      } else {
        qrow[u] = qrow[0];
      }
    }
    bf16x8 q[4][NV];
    float acc[4][DPL], m[4], l[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int v = 0; v < NV; ++v) q[u][v] = *reinterpret_cast<const bf16x8*>(Q + (int64_t)qrow[u] * io.ldq + 8 * v);
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[u][e] = 0.0f;
      m[u] = -INFINITY;
      l[u] = 0.0f;
    }
    uint64_t km = kmask;
    while (km != 0) {
      const int krow = __builtin_amdgcn_readlane(kr, __builtin_ctzll(km));
      km &= km - 1;
      bf16x8 kv[NV], vv[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        kv[v] = *reinterpret_cast<const bf16x8*>(K + (int64_t)krow * io.ldkv + 8 * v);
        vv[v] = *reinterpret_cast<const bf16x8*>(V + (int64_t)krow * io.ldkv + 8 * v);
      }
      float vf[DPL];
#pragma unroll
      for (int e = 0; e < DPL; ++e) vf[e] = (float)vv[e / 8][e % 8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float sc = 0.0f;
#pragma unroll
        for (int e = 0; e < DPL; e += 2) {
          const bf16x2 a = {q[u][e / 8][e % 8], q[u][e / 8][e % 8 + 1]};
          const bf16x2 b = {kv[e / 8][e % 8], kv[e / 8][e % 8 + 1]};
          sc = __builtin_amdgcn_fdot2_f32_bf16(a, b, sc, false);
        }
        sc = head_sum<LPH>(sc);
        const float mn = fmaxf(m[u], sc);
        const float corr = exp2f(m[u] - mn), pr = exp2f(sc - mn);
        l[u] = fmaf(l[u], corr, pr);
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[u][e] = fmaf(acc[u][e], corr, pr * vf[e]);
        m[u] = mn;
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (u < nqc) {
        const float inv = 1.0f / l[u];
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          bf16x8 o;
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = (bf16)(acc[u][8 * v + e] * inv);
          *reinterpret_cast<bf16x8*>(O + (int64_t)qrow[u] * D + 8 * v) = o;
        }
      }
    }
  }
}
}  // namespace

hipError_t launch_attn_temporal(sphinx_dtype dt, const ReqTable& T, const AttnIO& io, int D, int heads,
                                int head_dim, const int32_t* pos, bool cached, hipStream_t s) {
  int64_t cols = 0;
  for (int r = 0; r < T.R; ++r) cols += (int64_t)(T.h[r] >> 1) * (T.w[r] >> 1);
  const int cf = cached ? 1 : 0;
  // lane-parallel kernel: rows of 64 x 16 or 64 x 8 dims, heads of 64 (of 4 or 8 lanes)
  if (dt == SPHINX_BF16 && head_dim == 64 && (D == 1024 || D == 512)) {
    const unsigned grid = (unsigned)((cols + 3) / 4);
    if (D == 1024)
      k_attn_temporal_lanes<16, 4><<<grid, 256, 0, s>>>(T, io, D, pos, cf, (int)cols);
    else
      k_attn_temporal_lanes<8, 8><<<grid, 256, 0, s>>>(T, io, D, pos, cf, (int)cols);
    return hipGetLastError();
  }
  if (dt == SPHINX_BF16 && head_dim == 64)
    k_attn_temporal<bf16, 64, true><<<(unsigned)cols, 256, 0, s>>>(T, io, D, head_dim, heads, pos, cf);
  else if (dt == SPHINX_BF16)
    k_attn_temporal<bf16, 72, true><<<(unsigned)cols, 256, 0, s>>>(T, io, D, head_dim, heads, pos, cf);
  else
    k_attn_temporal<float, 64, false><<<(unsigned)cols, 256, 0, s>>>(T, io, D, head_dim, heads, pos, cf);
  return hipGetLastError();
}

}  // namespace sphinx
