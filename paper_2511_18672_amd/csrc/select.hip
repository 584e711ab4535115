// Selection mask and stable stream compaction (Alg. 1 opacity mask 1[O < tau_o]
// with u = -O; Sec. 5.3: only positions inside the mask are forwarded).
//
//   mask[t] = active[g(t)] && u[t] > thr[g(t)]        (strict; NaN -> 0)
//   idx     = ascending t with mask[t] = 1
//   cu_sel  = selected count before each request start, cu_sel[R] = n_sel
//
// Reduce-then-scan over chunks of 4096 tokens (256 threads x 4 groups of
// 4 consecutive tokens, float4 loads):
//   1. k_select_count  writes mask (uchar4) and one count per chunk,
//   2. k_select_scan   exclusive scan of the chunk counts (one workgroup),
//   3. k_select_write  ranks each selected token inside its chunk with wave64
//      ballots + mbcnt and writes idx; it also writes cu_sel at request starts.
// The order inside a chunk is (group, wave, lane, element) = token order, so
// idx comes out ascending without any sort and the result is deterministic.
#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int kTPB = 256;
constexpr int kGroups = 4;                      // float4 groups per thread
constexpr int kChunk = kTPB * kGroups * 4;      // 4096 tokens per workgroup

// Global frame of token t and the first token of the next frame.
__device__ __forceinline__ void frame_of(const ReqTable& T, int64_t t, int& g, int64_t& next) {
  const int r = find_request(T, t);
  const uint32_t loc = (uint32_t)(t - T.tok_off[r]);
  const uint32_t tpf = (uint32_t)(T.h[r] >> 1) * (uint32_t)(T.w[r] >> 1);
  const uint32_t f = loc / tpf;
  g = T.frame_off[r] + (int)f;
  next = T.tok_off[r] + (int64_t)(f + 1) * tpf;
}

__global__ __launch_bounds__(kTPB) void k_select_count(ReqTable T, int64_t N, const float* __restrict__ u,
                                                      const float* __restrict__ thr,
                                                      const uint8_t* __restrict__ active, uint8_t* __restrict__ mask,
                                                      int32_t* __restrict__ blk_cnt) {
  __shared__ int s_cnt[kTPB / kWave];
  const int64_t base = (int64_t)blockIdx.x * kChunk;
  int cnt = 0;
#pragma unroll
  for (int gi = 0; gi < kGroups; ++gi) {
    const int64_t t0 = base + ((int64_t)gi * kTPB + threadIdx.x) * 4;
    float v[4];
    if (t0 + 3 < N) {
      const float4 q = *reinterpret_cast<const float4*>(u + t0);
      v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = (t0 + e < N) ? u[t0 + e] : 0.0f;
    }
    // one frame lookup per group of 4 (a second one only when the group
    // straddles a frame boundary)
    uint32_t packed = 0;
    if (t0 < N) {
      int g;
      int64_t next;
      frame_of(T, t0, g, next);
      float th = thr[g];
      bool act = active ? (active[g] != 0) : true;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t t = t0 + e;
        if (t < N) {
          if (t >= next) {
            frame_of(T, t, g, next);
            th = thr[g];
            act = active ? (active[g] != 0) : true;
          }
          const bool m = act && (v[e] > th);
          packed |= (uint32_t)m << (8 * e);
          cnt += m;
        }
      }
    }
    if (t0 + 3 < N) {
      *reinterpret_cast<uint32_t*>(mask + t0) = packed;
    } else {
      for (int e = 0; e < 4; ++e)
        if (t0 + e < N) mask[t0 + e] = (uint8_t)((packed >> (8 * e)) & 1u);
    }
  }
  // block sum
  for (int m = 32; m >= 1; m >>= 1) cnt += __shfl_xor(cnt, m, kWave);
  if (lane_id() == 0) s_cnt[threadIdx.x / kWave] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int tot = 0;
    for (int w = 0; w < kTPB / kWave; ++w) tot += s_cnt[w];
    blk_cnt[blockIdx.x] = tot;
  }
}

// Exclusive scan of nblk chunk counts by one workgroup of 1024 threads.
__global__ __launch_bounds__(1024) void k_select_scan(const int32_t* __restrict__ blk_cnt, int nblk,
                                                     int32_t* __restrict__ blk_off, int32_t* __restrict__ cu_sel,
                                                     int R) {
  __shared__ int s_part[1024 / kWave];
  const int per = (nblk + 1023) / 1024;
  const int b0 = threadIdx.x * per;
  int local = 0;
  for (int i = 0; i < per; ++i)
    if (b0 + i < nblk) local += blk_cnt[b0 + i];
  // inclusive wave scan of `local`
  int incl = local;
  const int lane = lane_id();
  for (int d = 1; d < kWave; d <<= 1) {
    const int y = __shfl_up(incl, d, kWave);
    if (lane >= d) incl += y;
  }
  if (lane == kWave - 1) s_part[threadIdx.x / kWave] = incl;
  __syncthreads();
  int wave_base = 0;
  for (int w = 0; w < (int)(threadIdx.x / kWave); ++w) wave_base += s_part[w];
  int run = wave_base + incl - local;
  for (int i = 0; i < per; ++i) {
    if (b0 + i < nblk) {
      blk_off[b0 + i] = run;
      run += blk_cnt[b0 + i];
    }
  }
  if (threadIdx.x == 1023) {
    int tot = 0;
    for (int w = 0; w < 1024 / kWave; ++w) tot += s_part[w];
    cu_sel[R] = tot;
  }
}

__global__ __launch_bounds__(kTPB) void k_select_write(ReqTable T, int64_t N, const uint8_t* __restrict__ mask,
                                                      const int32_t* __restrict__ blk_off, int32_t* __restrict__ idx,
                                                      int32_t* __restrict__ cu_sel) {
  __shared__ int s_wcnt[kGroups][kTPB / kWave];
  const int64_t base = (int64_t)blockIdx.x * kChunk;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  uint32_t bits[kGroups];
  int lane_prefix[kGroups];
#pragma unroll
  for (int gi = 0; gi < kGroups; ++gi) {
    const int64_t t0 = base + ((int64_t)gi * kTPB + threadIdx.x) * 4;
    uint32_t packed = 0;
    if (t0 + 3 < N) {
      packed = *reinterpret_cast<const uint32_t*>(mask + t0);
    } else {
      for (int e = 0; e < 4; ++e)
        if (t0 + e < N) packed |= (uint32_t)(mask[t0 + e] & 1u) << (8 * e);
    }
    bits[gi] = packed;
    int before = 0, total = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint64_t b = __ballot((packed >> (8 * e)) & 1u);
      before += __popcll(b & ((1ull << lane) - 1ull));
      total += __popcll(b);
    }
    lane_prefix[gi] = before;
    if (lane == 0) s_wcnt[gi][wave] = total;
  }
  __syncthreads();
  int run = blk_off[blockIdx.x];
#pragma unroll
  for (int gi = 0; gi < kGroups; ++gi) {
    int wbase = run;
    for (int w = 0; w < wave; ++w) wbase += s_wcnt[gi][w];
    int gtot = 0;
    for (int w = 0; w < kTPB / kWave; ++w) gtot += s_wcnt[gi][w];
    const int64_t t0 = base + ((int64_t)gi * kTPB + threadIdx.x) * 4;
    int pos = wbase + lane_prefix[gi];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t t = t0 + e;
      if (t < N) {
        for (int r = 0; r < T.R; ++r)
          if (T.tok_off[r] == t) cu_sel[r] = pos;
      }
      if ((bits[gi] >> (8 * e)) & 1u) idx[pos++] = (int32_t)t;
    }
    run += gtot;
  }
}
}  // namespace

size_t select_ws_bytes(int64_t N) {
  const int64_t nblk = (N + kChunk - 1) / kChunk;
  return (size_t)(2 * nblk * sizeof(int32_t) + 256);
}

hipError_t launch_select(const ReqTable& T, int64_t N, const float* u, const float* thr, const uint8_t* active,
                         uint8_t* mask, int32_t* idx, int32_t* cu_sel, void* ws, hipStream_t s) {
  const int nblk = (int)((N + kChunk - 1) / kChunk);
  int32_t* blk_cnt = reinterpret_cast<int32_t*>(ws);
  int32_t* blk_off = blk_cnt + nblk;
  k_select_count<<<nblk, kTPB, 0, s>>>(T, N, u, thr, active, mask, blk_cnt);
  k_select_scan<<<1, 1024, 0, s>>>(blk_cnt, nblk, blk_off, cu_sel, T.R);
  k_select_write<<<nblk, kTPB, 0, s>>>(T, N, mask, blk_off, idx, cu_sel);
  return hipGetLastError();
}

}  // namespace sphinx
