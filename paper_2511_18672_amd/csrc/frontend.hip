// Spatial refinement mask from the regression output (Sec. 5.3; Alg. 1
// laplacian_var, otsu(norm(.)), the opacity mask 1[O < tau_o] and their union,
// pooled to latent tokens by the block rule).
//
// Every step is integer-exact:
//   Y   = (77 R + 150 G + 29 B + 128) >> 8                 (luma, 0..255)
//   L   = Y(up) + Y(down) + Y(left) + Y(right) - 4 Y         (4-neighbour Laplacian)
//   V   = 81 sum9x9(L^2) - sum9x9(L)^2                       (81^2 x local variance)
//   Wm  = sum5x5(V)                                          (box smoothing)
//   inv = 255 - floor(255 (Wm - min) / (max - min))          (per-frame min-max, inverted)
//   t   = Otsu threshold of inv over the frame (exact 192-bit comparison)
//   pixel mask = (O < tau_o) | (inv > t); a token (16 x 16 pixels) is selected
//   iff any of its pixels is.
// Every stencil reads its input map with replicated borders.
//
// Kernels (one pass over each input, Wm stored as 8 bytes per pixel and inv
// as 1):
//   k_front_var     per 64x16 tile: the stencil chain in LDS, Wm stored, tile
//                   min/max of Wm;
//   k_front_minmax  per frame: min/max over its tiles; clears the histogram;
//   k_front_quant   per 64x16 tile: inv as bytes from the stored Wm, LDS
//                   histogram merged into the frame's histogram with integer
//                   atomics;
//   k_front_otsu    per frame: Otsu threshold from the 256-bin histogram;
//   k_front_pool    per token: OR over its 16 x 16 pixels of both masks.
#include "kernels.hpp"

namespace sphinx {

namespace {
constexpr int kTX = 64, kTY = 16;  // output tile
constexpr int kRV = 4, kRS = 2;    // 9x9 variance window, 5x5 smoothing
constexpr int kHalo = 1 + kRV + kRS;
// LDS regions (rows x cols), relative to the tile origin
constexpr int kGY = kTY + 2 * kHalo, kGX = kTX + 2 * kHalo;              // luma: halo 7
constexpr int kLY = kTY + 2 * (kHalo - 1), kLX = kTX + 2 * (kHalo - 1);  // Laplacian: halo 6
constexpr int kSY = kLY, kSX = kTX + 2 * kRS;                            // row sums of L, L^2
constexpr int kVY = kTY + 2 * kRS, kVX = kTX + 2 * kRS;                  // V: halo 2
constexpr int kTPB = 256;

// |L| <= 1020 and |sum of 9 L| <= 9180 fit 16 bits; the row sums of V reuse
// the space of the luma .. row-sum regions, which are dead by then.
struct FrontEarly {
  int16_t gray[kGY * kGX];
  int16_t lap[kLY * kLX];
  int16_t s1[kSY * kSX];
  int32_t s2[kSY * kSX];
};
struct FrontSmem {
  union {
    FrontEarly e;
    int64_t r5[kVY * kTX];
  };
  int64_t v[kVY * kVX];
  int64_t red[2 * kTPB / kWave];
};
static_assert(sizeof(int64_t) * kVY * kTX <= sizeof(FrontEarly), "row sums of V must fit the early regions");

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return min(max(v, lo), hi); }

// Tile -> (request, frame, tile origin) for the packed frames of all requests.
struct TileLoc {
  int r, g, y0, x0, H, W;
  int64_t pix0;  // first pixel of the frame
};

__device__ __forceinline__ TileLoc locate_tile(const ReqTable& T, const FrontTiles& F, int tile) {
  int r = 0;
  while (r + 1 < T.R && F.tile_off[r + 1] <= tile) ++r;
  TileLoc L;
  L.r = r;
  L.H = 8 * T.h[r];
  L.W = 8 * T.w[r];
  const int ntx = (L.W + kTX - 1) / kTX, nty = L.H / kTY;
  const int loc = tile - F.tile_off[r];
  const int f = loc / (ntx * nty), rem = loc - f * ntx * nty;
  L.g = T.frame_off[r] + f;
  L.y0 = (rem / ntx) * kTY;
  L.x0 = (rem % ntx) * kTX;
  const int64_t tpf = (int64_t)(T.h[r] >> 1) * (T.w[r] >> 1);
  L.pix0 = 256 * (T.tok_off[r] + (int64_t)f * tpf);
  return L;
}

// The stencil chain of one 64 x 16 tile in LDS: stores Wm at the tile's
// in-image pixels and writes the tile's min and max of Wm to
// part[2 tile .. 2 tile + 1].
__global__ __launch_bounds__(kTPB) void k_front_var(ReqTable T, FrontTiles F, const uint8_t* __restrict__ rgb,
                                                    int64_t* __restrict__ part, int64_t* __restrict__ wm) {
  __shared__ FrontSmem sm;
  const int tid = threadIdx.x;
  const TileLoc L = locate_tile(T, F, blockIdx.x);
  const int H = L.H, W = L.W, y0 = L.y0, x0 = L.x0;
  const uint8_t* img = rgb + 3 * L.pix0;
  // luma at clamped positions
  for (int i = tid; i < kGY * kGX; i += kTPB) {
    const int ry = i / kGX, rx = i - ry * kGX;
    const int y = clampi(y0 - kHalo + ry, 0, H - 1), x = clampi(x0 - kHalo + rx, 0, W - 1);
    const uint8_t* p = img + 3 * ((int64_t)y * W + x);
    sm.e.gray[i] = (int16_t)((77 * (int)p[0] + 150 * (int)p[1] + 29 * (int)p[2] + 128) >> 8);
  }
  __syncthreads();
  // Laplacian at the clamped position of every region pixel
  for (int i = tid; i < kLY * kLX; i += kTPB) {
    const int ry = i / kLX, rx = i - ry * kLX;
    const int y = clampi(y0 - (kHalo - 1) + ry, 0, H - 1) - (y0 - kHalo);  // in luma-region coordinates
    const int x = clampi(x0 - (kHalo - 1) + rx, 0, W - 1) - (x0 - kHalo);
    const int16_t* g = sm.e.gray + y * kGX + x;
    sm.e.lap[i] = (int16_t)(g[-kGX] + g[kGX] + g[-1] + g[1] - 4 * g[0]);
  }
  __syncthreads();
  // horizontal 9-sums of L and L^2 around the clamped column
  for (int i = tid; i < kSY * kSX; i += kTPB) {
    const int ry = i / kSX, rx = i - ry * kSX;
    const int x = clampi(x0 - kRS + rx, 0, W - 1) - (x0 - (kHalo - 1));  // in Laplacian-region columns
    const int16_t* l = sm.e.lap + ry * kLX + x;
    int a = 0, b = 0;
#pragma unroll
    for (int d = -kRV; d <= kRV; ++d) {
      const int v = l[d];
      a += v;
      b += v * v;
    }
    sm.e.s1[i] = (int16_t)a;
    sm.e.s2[i] = b;
  }
  __syncthreads();
  // V = 81 sum(L^2) - (sum L)^2 over the 9x9 window of the clamped position
  for (int i = tid; i < kVY * kVX; i += kTPB) {
    const int ry = i / kVX, rx = i - ry * kVX;
    const int y = clampi(y0 - kRS + ry, 0, H - 1) - (y0 - (kHalo - 1));  // in row-sum-region rows
    int64_t a = 0, b = 0;
#pragma unroll
    for (int d = -kRV; d <= kRV; ++d) {
      a += sm.e.s1[(y + d) * kSX + rx];
      b += sm.e.s2[(y + d) * kSX + rx];
    }
    sm.v[i] = 81 * b - a * a;
  }
  __syncthreads();
  // horizontal 5-sums of V around the clamped column
  for (int i = tid; i < kVY * kTX; i += kTPB) {
    const int ry = i / kTX, rx = i - ry * kTX;
    const int x = clampi(x0 + rx, 0, W - 1) - (x0 - kRS);
    int64_t a = 0;
#pragma unroll
    for (int d = -kRS; d <= kRS; ++d) a += sm.v[ry * kVX + x + d];
    sm.r5[i] = a;
  }
  __syncthreads();
  // Wm at the tile's in-image pixels
  int64_t lo = INT64_MAX, hi = INT64_MIN;
  for (int i = tid; i < kTY * kTX; i += kTPB) {
    const int ry = i / kTX, rx = i - ry * kTX;
    const int y = y0 + ry, x = x0 + rx;
    if (x >= W) continue;
    const int yr = clampi(y, 0, H - 1) - (y0 - kRS);
    int64_t w = 0;
#pragma unroll
    for (int d = -kRS; d <= kRS; ++d) w += sm.r5[(yr + d) * kTX + rx];
    wm[L.pix0 + (int64_t)y * W + x] = w;
    lo = min(lo, w);
    hi = max(hi, w);
  }
  for (int m = 32; m >= 1; m >>= 1) {
    lo = min(lo, (int64_t)__shfl_xor(lo, m, kWave));
    hi = max(hi, (int64_t)__shfl_xor(hi, m, kWave));
  }
  if (lane_id() == 0) {
    sm.red[2 * (tid / kWave)] = lo;
    sm.red[2 * (tid / kWave) + 1] = hi;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kTPB / kWave; ++w) {
      lo = min(lo, sm.red[2 * w]);
      hi = max(hi, sm.red[2 * w + 1]);
    }
    part[2 * blockIdx.x] = lo;
    part[2 * blockIdx.x + 1] = hi;
  }
}

// Quantisation of one 64 x 16 tile's stored Wm with its frame's min/max
// (lohi), four consecutive pixels of a row per thread: inv as bytes, and the
// tile's histogram added to the frame's.
__global__ __launch_bounds__(kTPB) void k_front_quant(ReqTable T, FrontTiles F, const int64_t* __restrict__ wm,
                                                      const int64_t* __restrict__ lohi, uint8_t* __restrict__ inv,
                                                      uint32_t* __restrict__ hist) {
  static_assert(kTX * kTY == 4 * kTPB, "four pixels per thread");
  __shared__ uint32_t sh[256];
  const int tid = threadIdx.x;
  const TileLoc L = locate_tile(T, F, blockIdx.x);
  const int W = L.W;
  sh[tid] = 0;
  const int64_t flo = lohi[2 * L.g], fhi = lohi[2 * L.g + 1];
  const double span = (double)(fhi - flo);
  __syncthreads();
  const int y = L.y0 + tid / (kTX / 4), x = L.x0 + 4 * (tid % (kTX / 4));
  if (x < W) {  // W is a multiple of 8 pixels, so the four are all in the image or all past it
    const int64_t pix = L.pix0 + (int64_t)y * W + x;
    uint32_t packed = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t w = wm[pix + e];
      int q = 0;
      if (fhi > flo) {
        // floor(255 (w - lo) / (hi - lo)): a double quotient corrected to the exact floor
        const int64_t num = 255 * (w - flo), den = fhi - flo;
        int64_t qq = (int64_t)((double)num / span);
        if (qq * den > num) --qq;
        else if ((qq + 1) * den <= num) ++qq;
        q = (int)qq;
      }
      const int iv = 255 - q;
      packed |= (uint32_t)iv << (8 * e);
      atomicAdd(&sh[iv], 1u);
    }
    *reinterpret_cast<uint32_t*>(inv + pix) = packed;
  }
  __syncthreads();
  if (sh[tid] != 0) atomicAdd(&hist[256 * L.g + tid], sh[tid]);
}

// Per frame: min and max of Wm over its tiles; clears the frame's histogram.
__global__ __launch_bounds__(kTPB) void k_front_minmax(ReqTable T, FrontTiles F, const int64_t* __restrict__ part,
                                                       int64_t* __restrict__ lohi, uint32_t* __restrict__ hist) {
  __shared__ int64_t red[2 * kTPB / kWave];
  const int g = blockIdx.x, tid = threadIdx.x;
  int r = 0;
  while (r + 1 < T.R && T.frame_off[r + 1] <= g) ++r;
  const int W = 8 * T.w[r], H = 8 * T.h[r];
  const int per = ((W + kTX - 1) / kTX) * (H / kTY);
  const int t0 = F.tile_off[r] + (g - T.frame_off[r]) * per;
  int64_t lo = INT64_MAX, hi = INT64_MIN;
  for (int i = tid; i < per; i += kTPB) {
    lo = min(lo, part[2 * (t0 + i)]);
    hi = max(hi, part[2 * (t0 + i) + 1]);
  }
  for (int m = 32; m >= 1; m >>= 1) {
    lo = min(lo, (int64_t)__shfl_xor(lo, m, kWave));
    hi = max(hi, (int64_t)__shfl_xor(hi, m, kWave));
  }
  if (lane_id() == 0) {
    red[2 * (tid / kWave)] = lo;
    red[2 * (tid / kWave) + 1] = hi;
  }
  for (int i = tid; i < 256; i += kTPB) hist[256 * g + i] = 0;
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kTPB / kWave; ++w) {
      lo = min(lo, red[2 * w]);
      hi = max(hi, red[2 * w + 1]);
    }
    lohi[2 * g] = min(lo, red[0]);
    lohi[2 * g + 1] = max(hi, red[1]);
  }
}

// 192-bit value of a (128-bit) * b (64-bit), as three 64-bit limbs.
struct U192 {
  uint64_t hi, mid, lo;
};
__device__ __forceinline__ U192 mul128x64(unsigned __int128 a, uint64_t b) {
  const unsigned __int128 p0 = (unsigned __int128)(uint64_t)a * b;
  const unsigned __int128 p1 = (unsigned __int128)(uint64_t)(a >> 64) * b + (uint64_t)(p0 >> 64);
  return U192{(uint64_t)(p1 >> 64), (uint64_t)p1, (uint64_t)p0};
}
__device__ __forceinline__ bool gt192(const U192& x, const U192& y) {
  if (x.hi != y.hi) return x.hi > y.hi;
  if (x.mid != y.mid) return x.mid > y.mid;
  return x.lo > y.lo;
}

struct OtsuCand {
  uint64_t nhi, nlo, d;  // score numerator (128 bits) and denominator
  int t;
};
// a scores above b, or scores equal and has the smaller threshold
__device__ __forceinline__ bool otsu_better(const OtsuCand& a, const OtsuCand& b) {
  const unsigned __int128 na = ((unsigned __int128)a.nhi << 64) | a.nlo;
  const unsigned __int128 nb = ((unsigned __int128)b.nhi << 64) | b.nlo;
  const U192 x = mul128x64(na, b.d), y = mul128x64(nb, a.d);
  if (gt192(x, y)) return true;
  if (gt192(y, x)) return false;
  return a.t < b.t;
}

// Otsu's threshold per frame, one thread per candidate t: the t in 0..254
// maximising (S w0 - W s0)^2 / (w0 w1) (an empty class scores 0), compared
// exactly as cross products; the smallest t among equal maxima.
__global__ __launch_bounds__(256) void k_front_otsu(const uint32_t* __restrict__ hist, int32_t* __restrict__ thr) {
  __shared__ int64_t sw[4], ss[4];
  __shared__ OtsuCand best[4];
  const int g = blockIdx.x, t = threadIdx.x, lane = lane_id(), wave = t >> 6;
  const int64_t h = hist[256 * g + t];
  // inclusive scans of the counts and of t * counts
  int64_t w0 = h, s0 = (int64_t)t * h;
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t a = __shfl_up(w0, d, kWave), b = __shfl_up(s0, d, kWave);
    if (lane >= d) {
      w0 += a;
      s0 += b;
    }
  }
  if (lane == kWave - 1) {
    sw[wave] = w0;
    ss[wave] = s0;
  }
  __syncthreads();
  int64_t Wt = 0, St = 0;
  for (int w = 0; w < 4; ++w) {
    if (w < wave) {
      w0 += sw[w];
      s0 += ss[w];
    }
    Wt += sw[w];
    St += ss[w];
  }
  OtsuCand c{0, 0, 1, t};
  const int64_t w1 = Wt - w0;
  if (t == 255) {
    c.d = 1;  // not a candidate: scores below every real one through the tie rule
  } else if (w0 != 0 && w1 != 0) {
    const __int128 a = (__int128)St * w0 - (__int128)Wt * s0;
    const unsigned __int128 m = (unsigned __int128)(a < 0 ? -a : a);
    const unsigned __int128 n = m * m;
    c.nhi = (uint64_t)(n >> 64);
    c.nlo = (uint64_t)n;
    c.d = (uint64_t)w0 * (uint64_t)w1;
  }
  for (int m = 1; m < kWave; m <<= 1) {
    OtsuCand o;
    o.nhi = __shfl_xor(c.nhi, m, kWave);
    o.nlo = __shfl_xor(c.nlo, m, kWave);
    o.d = __shfl_xor(c.d, m, kWave);
    o.t = __shfl_xor(c.t, m, kWave);
    if (otsu_better(o, c)) c = o;
  }
  if (lane == 0) best[wave] = c;
  __syncthreads();
  if (t == 0) {
    for (int w = 1; w < 4; ++w)
      if (otsu_better(best[w], c)) c = best[w];
    thr[g] = c.t;
  }
}

// Token pooling: lane = 4 * row + k handles pixel row `row` (0..15) of token
// base + k; the 16 rows of a token are OR-reduced across lanes.
__global__ __launch_bounds__(kTPB) void k_front_pool(ReqTable T, const float* __restrict__ opacity, float tau,
                                                     const uint8_t* __restrict__ inv,
                                                     const int32_t* __restrict__ thr, uint8_t* __restrict__ mask,
                                                     float* __restrict__ u) {
  const int64_t N = T.tok_off[T.R];
  const int lane = lane_id(), k = lane & 3, row = lane >> 2;
  const int64_t t = ((int64_t)blockIdx.x * kTPB + threadIdx.x) / kWave * 4 + k;
  bool any = false;
  if (t < N) {
    const TokPos p = decode_token(T, t);
    const int W = 8 * T.w[p.r];
    const int64_t tpf = (int64_t)(T.h[p.r] >> 1) * (T.w[p.r] >> 1);
    const int64_t pix = 256 * (T.tok_off[p.r] + (int64_t)p.f * tpf) + (int64_t)(16 * p.y + row) * W + 16 * p.x;
    const int th = thr[p.g];
    const f32x4* o = reinterpret_cast<const f32x4*>(opacity + pix);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 v = o[q];
      any |= (v[0] < tau) | (v[1] < tau) | (v[2] < tau) | (v[3] < tau);
    }
    const uint4 b = *reinterpret_cast<const uint4*>(inv + pix);
    const uint32_t wv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) any |= (int)((wv[q] >> (8 * e)) & 255u) > th;
  }
  int a = any ? 1 : 0;
  for (int m = 4; m < kWave; m <<= 1) a |= __shfl_xor(a, m, kWave);
  if (t < N && row == 0) {
    mask[t] = (uint8_t)a;
    if (u != nullptr) u[t] = a ? 1.0f : 0.0f;
  }
}
}  // namespace

int front_tiles(const ReqTable& T, FrontTiles* F) {
  int n = 0;
  for (int r = 0; r < T.R; ++r) {
    F->tile_off[r] = n;
    const int W = 8 * T.w[r], H = 8 * T.h[r];
    n += T.frames[r] * ((W + kTX - 1) / kTX) * (H / kTY);
  }
  F->tile_off[T.R] = n;
  return n;
}

size_t front_ws_bytes(const ReqTable& T, int G) {
  FrontTiles F;
  const int tiles = front_tiles(T, &F);
  const int64_t pixels = 256 * T.tok_off[T.R];
  auto a256 = [](size_t b) { return (b + 255) & ~(size_t)255; };
  return a256((size_t)tiles * 16) + a256((size_t)G * 16) + a256((size_t)G * 1024) + a256((size_t)G * 4) +
         a256((size_t)pixels) + a256((size_t)pixels * 8);
}

hipError_t launch_front(const ReqTable& T, int G, const uint8_t* rgb, const float* opacity, float tau,
                        uint8_t* mask, float* u, int32_t* thr_out, void* ws, hipStream_t s) {
  FrontTiles F;
  const int tiles = front_tiles(T, &F);
  auto a256 = [](size_t b) { return (b + 255) & ~(size_t)255; };
  unsigned char* base = static_cast<unsigned char*>(ws);
  int64_t* part = reinterpret_cast<int64_t*>(base);
  base += a256((size_t)tiles * 16);
  int64_t* lohi = reinterpret_cast<int64_t*>(base);
  base += a256((size_t)G * 16);
  uint32_t* hist = reinterpret_cast<uint32_t*>(base);
  base += a256((size_t)G * 1024);
  int32_t* thr = thr_out != nullptr ? thr_out : reinterpret_cast<int32_t*>(base);
  base += a256((size_t)G * 4);
  const int64_t pixels = 256 * T.tok_off[T.R];
  uint8_t* inv = base;
  base += a256((size_t)pixels);
  int64_t* wm = reinterpret_cast<int64_t*>(base);
  k_front_var<<<tiles, kTPB, 0, s>>>(T, F, rgb, part, wm);
  k_front_minmax<<<G, kTPB, 0, s>>>(T, F, part, lohi, hist);
  k_front_quant<<<tiles, kTPB, 0, s>>>(T, F, wm, lohi, inv, hist);
  k_front_otsu<<<G, 256, 0, s>>>(hist, thr);
  const int64_t N = T.tok_off[T.R];
  k_front_pool<<<(unsigned)((N + 15) / 16), kTPB, 0, s>>>(T, opacity, tau, inv, thr, mask, u);
  return hipGetLastError();
}

}  // namespace sphinx
