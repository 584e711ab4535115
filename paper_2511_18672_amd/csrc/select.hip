// Selection mask and stable stream compaction (Alg. 1 opacity mask 1[O < tau_o]
// with u = -O; Sec. 5.3: only positions inside the mask are forwarded).
//
//   mask[t] = active[g(t)] && u[t] > thr[g(t)]        (strict; NaN -> 0)
//   idx     = ascending t with mask[t] = 1
//   cu_sel  = selected count before each request start, cu_sel[R] = n_sel
//
// Reduce-then-scan over chunks of 4096 tokens; every thread owns 16
// consecutive tokens (64 contiguous bytes of u, 16 bytes of mask):
//   1. k_select_count  writes the mask and one count per chunk,
//   2. k_select_scan   exclusive scan of the chunk counts (one workgroup),
//   3. k_select_write  ranks the selected tokens of a chunk with a wave64 scan
//      of per-thread counts, stages their indices in LDS and stores them
//      contiguously; it also writes cu_sel at request starts.
// Thread order is token order, so idx comes out ascending without a sort and
// the result is deterministic.  (Non-temporal loads and stores measured slower
// here than ordinary ones, unlike in gather/scatter.)
#include <mutex>

#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int kTPB = 256;
constexpr int kPer = 16;              // consecutive tokens per thread
constexpr int kChunk = kTPB * kPer;   // 4096 tokens per workgroup
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Global frame of token t and the first token of the next frame.
__device__ __forceinline__ void frame_of(const ReqTable& T, int64_t t, int& g, int64_t& next) {
  const int r = find_request(T, t);
  const uint32_t loc = (uint32_t)(t - T.tok_off[r]);
  const uint32_t tpf = (uint32_t)(T.h[r] >> 1) * (uint32_t)(T.w[r] >> 1);
  const uint32_t f = loc / tpf;
  g = T.frame_off[r] + (int)f;
  next = T.tok_off[r] + (int64_t)(f + 1) * tpf;
}

__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
  for (int d = 1; d < kWave; d <<= 1) {
    const int y = __shfl_up(v, d, kWave);
    if (lane >= d) v += y;
  }
  return v;
}

__global__ __launch_bounds__(kTPB) void k_select_count(ReqTable T, int64_t N, const float* __restrict__ u,
                                                      const float* __restrict__ thr,
                                                      const uint8_t* __restrict__ active, uint8_t* __restrict__ mask,
                                                      int32_t* __restrict__ blk_cnt) {
  __shared__ int s_cnt[kTPB / kWave];
  const int64_t t0 = (int64_t)blockIdx.x * kChunk + (int64_t)threadIdx.x * kPer;
  int cnt = 0;
  if (t0 < N) {
    const bool full = t0 + kPer <= N;
    float v[kPer];
    if (full) {
#pragma unroll
      for (int q = 0; q < kPer / 4; ++q) {
        const f32x4 f = reinterpret_cast<const f32x4*>(u + t0)[q];
        v[4 * q] = f[0];
        v[4 * q + 1] = f[1];
        v[4 * q + 2] = f[2];
        v[4 * q + 3] = f[3];
      }
    } else {
#pragma unroll
      for (int e = 0; e < kPer; ++e) v[e] = (t0 + e < N) ? u[t0 + e] : 0.0f;
    }
    // one frame lookup per thread, another only where its tokens cross a frame
    int g;
    int64_t next;
    frame_of(T, t0, g, next);
    float th = thr[g];
    bool act = active ? (active[g] != 0) : true;
    uint32_t w[kPer / 4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      const int64_t t = t0 + e;
      if (t < N) {
        if (t >= next) {
          frame_of(T, t, g, next);
          th = thr[g];
          act = active ? (active[g] != 0) : true;
        }
        const bool m = act && (v[e] > th);
        w[e >> 2] |= (uint32_t)m << (8 * (e & 3));
        cnt += m;
      }
    }
    if (full) {
      *reinterpret_cast<u32x4*>(mask + t0) = u32x4{w[0], w[1], w[2], w[3]};
    } else {
      for (int e = 0; e < kPer; ++e)
        if (t0 + e < N) mask[t0 + e] = (uint8_t)((w[e >> 2] >> (8 * (e & 3))) & 1u);
    }
  }
  for (int m = 32; m >= 1; m >>= 1) cnt += __shfl_xor(cnt, m, kWave);
  if (lane_id() == 0) s_cnt[threadIdx.x / kWave] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int tot = 0;
    for (int w = 0; w < kTPB / kWave; ++w) tot += s_cnt[w];
    blk_cnt[blockIdx.x] = tot;
  }
}

// Exclusive scan of nblk chunk counts by one workgroup of 1024 threads,
// 16384 counts per pass: thread i owns counts 16 i .. 16 i + 15 of the pass
// and moves them with four 16-byte loads and stores (both arrays are 16-byte
// aligned), so no count is staged in LDS; a wave64 scan of the per-thread
// sums and the 16 wave totals (read by every lane of a wave at one address)
// give each thread its base.
constexpr int kScanPer = 16;
constexpr int kScanBlk = 1024 * kScanPer;
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(1024) void k_select_scan(const int32_t* __restrict__ blk_cnt, int nblk,
                                                     int32_t* __restrict__ blk_off, int32_t* __restrict__ cu_sel,
                                                     int R) {
  __shared__ int s_part[1024 / kWave];
  const int tid = (int)threadIdx.x, lane = lane_id(), wave = tid / kWave;
  int carry = 0;  // counts of the passes before this one
  for (int base = 0; base < nblk; base += kScanBlk) {
    const int i0 = base + tid * kScanPer;
    const bool full = i0 + kScanPer <= nblk;
    int v[kScanPer];
    if (full) {
#pragma unroll
      for (int q = 0; q < kScanPer / 4; ++q) {
        const i32x4 x = reinterpret_cast<const i32x4*>(blk_cnt + i0)[q];
        v[4 * q] = x[0];
        v[4 * q + 1] = x[1];
        v[4 * q + 2] = x[2];
        v[4 * q + 3] = x[3];
      }
    } else {
#pragma unroll
      for (int j = 0; j < kScanPer; ++j) v[j] = (i0 + j < nblk) ? blk_cnt[i0 + j] : 0;
    }
    int local = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) local += v[j];
    const int incl = wave_incl_scan(local, lane);
    if (lane == kWave - 1) s_part[wave] = incl;
    __syncthreads();
    int wave_base = 0, total = 0;
    for (int w = 0; w < 1024 / kWave; ++w) {
      const int p = s_part[w];
      if (w < wave) wave_base += p;
      total += p;
    }
    int run = carry + wave_base + incl - local;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
      const int c = v[j];
      v[j] = run;
      run += c;
    }
    if (full) {
#pragma unroll
      for (int q = 0; q < kScanPer / 4; ++q)
        reinterpret_cast<i32x4*>(blk_off + i0)[q] = i32x4{v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
    } else {
#pragma unroll
      for (int j = 0; j < kScanPer; ++j)
        if (i0 + j < nblk) blk_off[i0 + j] = v[j];
    }
    carry += total;
    __syncthreads();  // s_part is rewritten by the next pass
  }
  if (tid == 0) cu_sel[R] = carry;
}

__global__ __launch_bounds__(kTPB) void k_select_write(ReqTable T, int64_t N, const uint8_t* __restrict__ mask,
                                                      const int32_t* __restrict__ blk_off, int32_t* __restrict__ idx,
                                                      int32_t* __restrict__ cu_sel) {
  __shared__ int s_wtot[kTPB / kWave];
  __shared__ int32_t s_idx[kChunk];
  const int64_t t0 = (int64_t)blockIdx.x * kChunk + (int64_t)threadIdx.x * kPer;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  uint32_t w[kPer / 4] = {0u, 0u, 0u, 0u};
  if (t0 + kPer <= N) {
    const u32x4 m4 = *reinterpret_cast<const u32x4*>(mask + t0);
    w[0] = m4[0];
    w[1] = m4[1];
    w[2] = m4[2];
    w[3] = m4[3];
  } else {
    for (int e = 0; e < kPer; ++e)
      if (t0 + e < N) w[e >> 2] |= (uint32_t)(mask[t0 + e] & 1u) << (8 * (e & 3));
  }
  // mask bytes are 0 or 1: fold the 4 bytes of each word into 4 bits
  uint32_t bits = 0;
#pragma unroll
  for (int q = 0; q < kPer / 4; ++q)
    bits |= ((w[q] & 1u) | ((w[q] >> 7) & 2u) | ((w[q] >> 14) & 4u) | ((w[q] >> 21) & 8u)) << (4 * q);
  const int cnt = __popc(bits);
  const int incl = wave_incl_scan(cnt, lane);
  if (lane == kWave - 1) s_wtot[wave] = incl;
  __syncthreads();
  int lpos = incl - cnt;
  for (int i = 0; i < wave; ++i) lpos += s_wtot[i];
  int btot = 0;
  for (int i = 0; i < kTPB / kWave; ++i) btot += s_wtot[i];
  const int boff = blk_off[blockIdx.x];
  for (int r = 0; r < T.R; ++r) {
    const int64_t s = T.tok_off[r];
    if (s >= t0 && s < t0 + kPer && s < N)
      cu_sel[r] = boff + lpos + __popc(bits & ((1u << (uint32_t)(s - t0)) - 1u));
  }
  int p = lpos;
#pragma unroll
  for (int e = 0; e < kPer; ++e)
    if ((bits >> e) & 1u) s_idx[p++] = (int32_t)(t0 + e);
  __syncthreads();
  for (int i = threadIdx.x; i < btot; i += kTPB) idx[boff + i] = s_idx[i];
}
}  // namespace

// Scratch of the allocation-free selection (sphinx_select_mask_static): the
// chunk counts and offsets of up to kStaticChunks chunks, 512 KB, one copy per
// GPU for the life of the process.  Every call fully rewrites the entries it
// reads (counts of all its chunks, then their offsets), so nothing needs
// clearing between calls; calls that overlap on one GPU share the array and
// race.  In host code `scratch` is only a symbol: its device address comes
// from hipGetSymbolAddress, resolved once per device.
constexpr int64_t kStaticChunks = (int64_t)1 << 16;
static __device__ __align__(256) int32_t scratch[2 * kStaticChunks];

static_assert(kStaticChunks * kChunk == SPHINX_SELECT_STATIC_MAX_TOKENS, "the header states the static limit");
static_assert(kStaticChunks % 4 == 0, "the offsets start at a multiple of 4 entries");

int64_t select_static_max_tokens() { return kStaticChunks * kChunk; }

hipError_t select_static_ws(void** ptr) {
  static std::mutex mu;
  static void* dev_ptr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(mu);
  if (dev_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    dev_ptr[dev] = p;
  }
  *ptr = dev_ptr[dev];
  return hipSuccess;
}

// Chunk counts, then their offsets from the next multiple of 4 entries on
// (at most 12 bytes of the 256 spare).
size_t select_ws_bytes(int64_t N) {
  const int64_t nblk = (N + kChunk - 1) / kChunk;
  return (size_t)(2 * nblk * sizeof(int32_t) + 256);
}

hipError_t launch_select(const ReqTable& T, int64_t N, const float* u, const float* thr, const uint8_t* active,
                         uint8_t* mask, int32_t* idx, int32_t* cu_sel, void* ws, hipStream_t s) {
  const int nblk = (int)((N + kChunk - 1) / kChunk);
  int32_t* blk_cnt = reinterpret_cast<int32_t*>(ws);
  int32_t* blk_off = blk_cnt + ((nblk + 3) & ~3);  // 16-byte aligned, like blk_cnt
  k_select_count<<<nblk, kTPB, 0, s>>>(T, N, u, thr, active, mask, blk_cnt);
  k_select_scan<<<1, 1024, 0, s>>>(blk_cnt, nblk, blk_off, cu_sel, T.R);
  k_select_write<<<nblk, kTPB, 0, s>>>(T, N, mask, blk_off, idx, cu_sel);
  return hipGetLastError();
}

}  // namespace sphinx
