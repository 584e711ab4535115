// Internal launchers of the gfx950 kernels.  Callers (api.cpp) validate every
// argument and size before calling; the launchers only enqueue work on the
// given stream and return hipGetLastError().
#pragma once

#include "common.hpp"

namespace sphinx {

enum { EPI_BIAS = 0, EPI_GELU = 1, EPI_GATED = 2 };

struct GemmEpi {
  void* out;             // EPI_BIAS/EPI_GELU: activation buffer; EPI_GATED: fp32 residual h
  int ldo;
  const float* gate;     // EPI_GATED: gate rows (conditioning row of each token)
  int ldg;
  const int32_t* crow;   // EPI_GATED: conditioning row of each token
  int qcols;             // EPI_BIAS: columns [0, qcols) are multiplied by qscale before the store
  float qscale;          //   (the queries of the QKV projection, scaled by log2(e)/sqrt(head_dim))
};

// Attention segments (one per request with forwarded tokens): the queries of
// segment i are rows [start, start+len) of q, its keys and values rows
// [kv_start, kv_start+kv_len) of k and v (the same rows without a latent
// cache; all tokens of the request with one).
struct SegTable {
  int nseg;                                  // non-empty segments, most keys first
  int start[SPHINX_MAX_REQUESTS];
  int len[SPHINX_MAX_REQUESTS];
  int kv_start[SPHINX_MAX_REQUESTS];
  int kv_len[SPHINX_MAX_REQUESTS];
  int tile_prefix[SPHINX_MAX_REQUESTS + 1];  // prefix sums of 128-query tiles
};

// Attention operands: q rows with stride ldq, k and v rows with stride ldkv
// (elements), output rows with stride D.
struct AttnIO {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  int ldq;
  int ldkv;
};

// Context tokens of a gather with a latent cache: tokens t with wmask[t] == 0
// take the coefficients a[g], b[g] of this struct instead of the write-set ones.
struct GatherCtx {
  const uint8_t* wmask;  // NULL: every token uses the write-set coefficients
  const float* a;
  const float* b;
};

constexpr int kAttnQueryTile = 128;

// select.hip
size_t select_ws_bytes(int64_t N);
// The library's static selection scratch: the largest N it serves, and its
// device address on the current device (looked up once per device).
constexpr int kMaxDevices = 64;
int64_t select_static_max_tokens();
hipError_t select_static_ws(void** ptr);
hipError_t launch_select(const ReqTable& T, int64_t N, const float* u, const float* thr, const uint8_t* active,
                         uint8_t* mask, int32_t* idx, int32_t* cu_sel, void* ws, hipStream_t s);

// gather_scatter.hip
hipError_t launch_gather(const ReqTable& T, sphinx_layout lay, const void* state, sphinx_dtype sdt, const void* eps,
                         sphinx_dtype edt, const int32_t* idx, int n, const float* a, const float* b,
                         const GatherCtx& ctx, float* x, hipStream_t s);
hipError_t launch_scatter(const ReqTable& T, const float* x, const int32_t* idx, int n, const uint8_t* wmask,
                          void* out, sphinx_dtype odt, sphinx_layout lay, hipStream_t s);
// Latent cache store: cache row idx[j] (2D elements: key then value) <- qkv row j
// columns [D, 3D).
hipError_t launch_kv_store(sphinx_dtype dt, const void* qkv, int n, int D, const int32_t* idx, int64_t N,
                           void* cache, hipStream_t s);
hipError_t launch_convert(const ReqTable& T, const void* in, sphinx_dtype idt, sphinx_layout il, void* out,
                          sphinx_dtype odt, sphinx_layout ol, hipStream_t s);

// frontend.hip: tiles of the mask front-end, per request
struct FrontTiles {
  int tile_off[SPHINX_MAX_REQUESTS + 1];
};
int front_tiles(const ReqTable& T, FrontTiles* F);
size_t front_ws_bytes(const ReqTable& T, int G);
hipError_t launch_front(const ReqTable& T, int G, const uint8_t* rgb, const float* opacity, float tau,
                        uint8_t* mask, float* u, int32_t* thr_out, void* ws, hipStream_t s);

// cond.hip
hipError_t launch_cond_rows(const int32_t* tau, int G, int32_t* fmap, int32_t* utau, int32_t* U, hipStream_t s);
hipError_t launch_temb(const int32_t* utau, const int32_t* U, int Gmax, float* temb, hipStream_t s);
hipError_t launch_rowgemm(const float* X, int ldx, const int32_t* U, int K, const void* W, const void* b,
                          sphinx_dtype wdt, int N, bool silu_out, float* out, int ldo, hipStream_t s);
hipError_t launch_pos_tables(int D, int hp, int wp, int nf, float* Ty, float* Tx, float* Tf, hipStream_t s);
hipError_t launch_token_meta(const ReqTable& T, const int32_t* idx, int n, const int32_t* fmap, int32_t* gframe,
                             int32_t* crow, int32_t* posc, hipStream_t s);

// rowwise.hip
hipError_t launch_embed(const float* x, int n, int D, const void* pe_w, const void* pe_b, sphinx_dtype wdt,
                        const float* Ty, const float* Tx, const float* Tf, const int32_t* posc, float* h,
                        hipStream_t s);
hipError_t launch_ln_mod(const float* h, int n, int D, const float* mod, int ldm, int sh_off, int sc_off,
                         const int32_t* crow, void* out, sphinx_dtype odt, hipStream_t s);
hipError_t launch_final(const float* h, int n, int D, const float* mod, int ldm, int sh_off, int sc_off,
                        const int32_t* crow, const int32_t* gframe, const void* out_w, const void* out_b,
                        sphinx_dtype wdt, const float* c1, const float* c2, float* x, hipStream_t s);

// gemm.hip
hipError_t launch_gemm(int epi, sphinx_dtype dt, const void* A, const void* W, const void* bias, int M, int N, int K,
                       const GemmEpi& e, hipStream_t s);
hipError_t launch_peak_mfma(int iters, bool random, float* out, int blocks, hipStream_t s);

// attention.hip
hipError_t launch_attention(sphinx_dtype dt, const AttnIO& io, int D, int heads, int head_dim, int n,
                            const SegTable& S, hipStream_t s);
// Temporal attention of a factorised denoiser: pos[t] = forwarded row of token t
// or -1; keys are the forwarded tokens of the column (or all of its frames from
// the cache when `cached`).  Frames per request <= 64.
hipError_t launch_attn_temporal(sphinx_dtype dt, const ReqTable& T, const AttnIO& io, int D, int heads,
                                int head_dim, const int32_t* pos, bool cached, hipStream_t s);
// Per-frame counts of the forwarded rows and the token -> row map (rowwise.hip).
hipError_t launch_frame_bounds(const ReqTable& T, const int32_t* idx, int n, int G, int32_t* first, hipStream_t s);
hipError_t launch_pos_map(int64_t N, const int32_t* idx, int n, int32_t* pos, hipStream_t s);

}  // namespace sphinx
