// C ABI of the selective-refinement step (declared in include/sphinx.h).
// Host code only: argument validation (before any HIP call), workspace
// carving, launch sequencing and the host-side step schedule.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <vector>

#include "kernels.hpp"
#include "sphinx_prof.h"

using namespace sphinx;

namespace {

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
constexpr float kLog2e = 1.4426950408889634f;
inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }
inline size_t esize(sphinx_dtype d) { return d == SPHINX_BF16 ? 2 : 4; }
inline bool valid_dtype(sphinx_dtype d) { return d == SPHINX_F32 || d == SPHINX_BF16; }
inline bool valid_layout(sphinx_layout l) { return l == SPHINX_LAYOUT_NCHW || l == SPHINX_LAYOUT_TOKENS; }
inline size_t dtype_bytes(sphinx_dtype d) { return d == SPHINX_F32 ? 4 : 2; }

sphinx_status build_table(const sphinx_request* reqs, int32_t R, ReqTable* T, int64_t* N, int32_t* G) {
  if (reqs == nullptr || R < 1) return SPHINX_E_INVALID;
  if (R > SPHINX_MAX_REQUESTS) return SPHINX_E_UNSUPPORTED;
  std::memset(T, 0, sizeof(*T));
  int64_t tok = 0;
  int64_t fr = 0;
  for (int r = 0; r < R; ++r) {
    const sphinx_request& q = reqs[r];
    if (q.frames < 1 || q.h < 2 || q.w < 2 || (q.h & 1) || (q.w & 1)) return SPHINX_E_INVALID;
    if (q.tok_offset != tok || q.frame_offset != fr) return SPHINX_E_INVALID;
    if (q.h / 2 > 1024 || q.w / 2 > 1024 || q.frames > 2047) return SPHINX_E_UNSUPPORTED;
    T->frames[r] = q.frames;
    T->h[r] = q.h;
    T->w[r] = q.w;
    T->frame_off[r] = (int32_t)fr;
    T->tok_off[r] = tok;
    tok += (int64_t)q.frames * (q.h / 2) * (q.w / 2);
    fr += q.frames;
    if (tok >= (int64_t)INT32_MAX || fr >= (int64_t)INT32_MAX) return SPHINX_E_UNSUPPORTED;
  }
  T->R = R;
  T->tok_off[R] = tok;
  T->frame_off[R] = (int32_t)fr;
  *N = tok;
  *G = (int32_t)fr;
  return SPHINX_OK;
}

sphinx_status check_model(const sphinx_model_desc* m) {
  if (m == nullptr) return SPHINX_E_INVALID;
  if (m->D <= 0 || m->heads <= 0 || m->head_dim <= 0 || m->mlp <= 0 || m->L <= 0) return SPHINX_E_INVALID;
  if ((int64_t)m->heads * m->head_dim != m->D) return SPHINX_E_INVALID;
  if (!valid_dtype(m->dtype)) return SPHINX_E_UNSUPPORTED;
  if (m->attention != SPHINX_ATTN_JOINT && m->attention != SPHINX_ATTN_FACTORISED) return SPHINX_E_UNSUPPORTED;
  if (m->dtype == SPHINX_BF16) {
    if ((m->head_dim != 64 && m->head_dim != 72) || m->D % 128 != 0 || m->mlp % 128 != 0 || m->D > 2048)
      return SPHINX_E_UNSUPPORTED;
  } else {
    if (m->head_dim > 64 || m->D % 64 != 0 || m->mlp % 64 != 0 || m->D > 512) return SPHINX_E_UNSUPPORTED;
  }
  return SPHINX_OK;
}

// Blob layout: walk the tensors in storage order.
struct Tensor {
  sphinx_param p;
  int block;
  size_t count;
};

std::vector<Tensor> blob_order(const sphinx_model_desc& m) {
  const size_t D = m.D, H = m.mlp, L = m.L;
  std::vector<Tensor> t = {{SPHINX_P_PE_W, -1, D * 16}, {SPHINX_P_PE_B, -1, D},
                           {SPHINX_P_T1_W, -1, D * SPHINX_TEMB_DIM}, {SPHINX_P_T1_B, -1, D},
                           {SPHINX_P_T2_W, -1, D * D}, {SPHINX_P_T2_B, -1, D},
                           {SPHINX_P_COND_W, -1, (6 * L + 2) * D * D}, {SPHINX_P_COND_B, -1, (6 * L + 2) * D}};
  for (int l = 0; l < (int)L; ++l) {
    t.push_back({SPHINX_P_QKV_W, l, 3 * D * D});
    t.push_back({SPHINX_P_QKV_B, l, 3 * D});
    t.push_back({SPHINX_P_O_W, l, D * D});
    t.push_back({SPHINX_P_O_B, l, D});
    t.push_back({SPHINX_P_FC1_W, l, H * D});
    t.push_back({SPHINX_P_FC1_B, l, H});
    t.push_back({SPHINX_P_FC2_W, l, D * H});
    t.push_back({SPHINX_P_FC2_B, l, D});
  }
  t.push_back({SPHINX_P_OUT_W, -1, 16 * D});
  t.push_back({SPHINX_P_OUT_B, -1, 16});
  return t;
}

bool per_block(sphinx_param p) { return p >= SPHINX_P_QKV_W && p <= SPHINX_P_FC2_B; }

struct Blob {
  std::vector<size_t> off;  // indexed [p] for globals, [P_COUNT + l*8 + (p - QKV_W)] per block
  size_t total = 0;
  size_t at(sphinx_param p, int l) const {
    return per_block(p) ? off[SPHINX_P_COUNT + (size_t)l * 8 + (p - SPHINX_P_QKV_W)] : off[p];
  }
};

Blob blob_layout(const sphinx_model_desc& m) {
  Blob b;
  b.off.assign(SPHINX_P_COUNT + (size_t)m.L * 8, 0);
  size_t cur = 0;
  for (const Tensor& t : blob_order(m)) {
    cur = align256(cur);
    if (per_block(t.p))
      b.off[SPHINX_P_COUNT + (size_t)t.block * 8 + (t.p - SPHINX_P_QKV_W)] = cur;
    else
      b.off[t.p] = cur;
    cur += t.count * esize(m.dtype);
  }
  b.total = align256(cur);
  return b;
}

struct RefineWs {
  size_t fmap, utau, U, temb, cbuf, sc, mod, Ty, Tx, Tf, gframe, crow, posc, fcnt, pos, h, a, big, total;
  int maxHp, maxWp, maxF;
};

RefineWs refine_layout(const sphinx_model_desc& m, const ReqTable& T, int G, int64_t n) {
  RefineWs w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t D = m.D, act = esize(m.dtype);
  const size_t ldm = (6 * (size_t)m.L + 2) * D;
  w.maxHp = w.maxWp = w.maxF = 1;
  for (int r = 0; r < T.R; ++r) {
    w.maxHp = std::max(w.maxHp, T.h[r] / 2);
    w.maxWp = std::max(w.maxWp, T.w[r] / 2);
    w.maxF = std::max(w.maxF, T.frames[r]);
  }
  w.fmap = take((size_t)G * 4);
  w.utau = take((size_t)G * 4);
  w.U = take(4);
  w.temb = take((size_t)G * SPHINX_TEMB_DIM * 4);
  w.cbuf = take((size_t)G * D * 4);
  w.sc = take((size_t)G * D * 4);
  w.mod = take((size_t)G * ldm * 4);
  w.Ty = take((size_t)w.maxHp * (D / 2) * 4);
  w.Tx = take((size_t)w.maxWp * (D / 2) * 4);
  w.Tf = take((size_t)w.maxF * D * 4);
  w.gframe = take((size_t)n * 4);
  w.crow = take((size_t)n * 4);
  w.posc = take((size_t)n * 4);
  w.fcnt = take((size_t)(G + 1) * 4);     // factorised: first forwarded row of each frame (and n)
  w.pos = take((size_t)T.tok_off[T.R] * 4);  // factorised: token -> forwarded row
  w.h = take((size_t)n * D * 4);
  w.a = take((size_t)n * D * act);
  w.big = take((size_t)n * std::max<size_t>(4 * D, (size_t)m.mlp) * act);
  w.total = off;
  return w;
}

double alpha_bar_at(const std::vector<double>& ab, int t) { return t < 0 ? 1.0 : ab[t]; }

std::vector<double> alpha_bar_table() {
  std::vector<double> ab(SPHINX_TRAIN_STEPS);
  double prod = 1.0;
  for (int i = 0; i < SPHINX_TRAIN_STEPS; ++i) {
    const double beta = 1e-4 + (2e-2 - 1e-4) * (double)i / (double)(SPHINX_TRAIN_STEPS - 1);
    prod *= 1.0 - beta;
    ab[i] = prod;
  }
  return ab;
}

// ---- profiling aid: HIP-event brackets per kernel class ----------------------
struct Timing {
  std::mutex mu;
  uint32_t mask = 0;  // bit k: bracket kernel class k
  struct Pending {
    int cls;
    hipEvent_t a, b;
  };
  std::vector<std::pair<hipEvent_t, hipEvent_t>> spare;
  std::vector<Pending> pending;
  int64_t launches[SPHINX_K_COUNT] = {};
  double ms[SPHINX_K_COUNT] = {};

  void resolve() {  // caller holds mu
    for (const Pending& p : pending) {
      float t = 0.f;
      if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&t, p.a, p.b) == hipSuccess) {
        launches[p.cls] += 1;
        ms[p.cls] += t;
      }
      spare.emplace_back(p.a, p.b);
    }
    pending.clear();
  }
};

Timing& timing() {
  static Timing t;
  return t;
}

// Records an event before the launches of its scope and one after, on `s`.
class Bracket {
 public:
  Bracket(int cls, hipStream_t s) : cls_(cls), s_(s) {
    Timing& T = timing();
    std::lock_guard<std::mutex> g(T.mu);
    if (((T.mask >> cls) & 1u) == 0) return;
    if (T.spare.empty()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess) return;
      if (hipEventCreate(&b) != hipSuccess) {
        (void)hipEventDestroy(a);
        return;
      }
      T.spare.emplace_back(a, b);
    }
    a_ = T.spare.back().first;
    b_ = T.spare.back().second;
    T.spare.pop_back();
    if (hipEventRecord(a_, s_) != hipSuccess) {
      T.spare.emplace_back(a_, b_);
      a_ = nullptr;
    }
  }
  ~Bracket() {
    if (a_ == nullptr) return;
    Timing& T = timing();
    std::lock_guard<std::mutex> g(T.mu);
    if (hipEventRecord(b_, s_) == hipSuccess)
      T.pending.push_back({cls_, a_, b_});
    else
      T.spare.emplace_back(a_, b_);
  }
  Bracket(const Bracket&) = delete;
  Bracket& operator=(const Bracket&) = delete;

 private:
  int cls_;
  hipStream_t s_;
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

inline sphinx_status hip_status(hipError_t e) { return e == hipSuccess ? SPHINX_OK : SPHINX_E_HIP; }

#define SPHINX_TRY(expr)                              \
  do {                                                \
    const hipError_t _e = (expr);                     \
    if (_e != hipSuccess) return SPHINX_E_HIP;        \
  } while (0)

}  // namespace

extern "C" {

const char* sphinx_status_string(sphinx_status s) {
  switch (s) {
    case SPHINX_OK: return "ok";
    case SPHINX_E_INVALID: return "invalid argument";
    case SPHINX_E_UNSUPPORTED: return "unsupported configuration";
    case SPHINX_E_WORKSPACE: return "workspace too small";
    case SPHINX_E_HIP: return "HIP launch or copy failed";
  }
  return "unknown status";
}

sphinx_status sphinx_model_blob_bytes(const sphinx_model_desc* m, size_t* bytes) {
  const sphinx_status st = check_model(m);
  if (st != SPHINX_OK) return st;
  if (bytes == nullptr) return SPHINX_E_INVALID;
  *bytes = blob_layout(*m).total;
  return SPHINX_OK;
}

sphinx_status sphinx_model_param(const sphinx_model_desc* m, sphinx_param p, int32_t block, size_t* offset_bytes,
                                 size_t* count) {
  const sphinx_status st = check_model(m);
  if (st != SPHINX_OK) return st;
  if (offset_bytes == nullptr || count == nullptr || (int)p < 0 || p >= SPHINX_P_COUNT) return SPHINX_E_INVALID;
  if (per_block(p) && (block < 0 || block >= m->L)) return SPHINX_E_INVALID;
  const Blob b = blob_layout(*m);
  for (const Tensor& t : blob_order(*m)) {
    if (t.p == p && (!per_block(p) || t.block == block)) {
      *offset_bytes = b.at(p, block);
      *count = t.count;
      return SPHINX_OK;
    }
  }
  return SPHINX_E_INVALID;
}

sphinx_status sphinx_plan_step_grid(const sphinx_request* reqs, int32_t R, const int32_t* s_start,
                                    const int32_t* nsteps, int32_t step, sphinx_grid grid_kind, uint8_t* active,
                                    uint8_t* newly, int32_t* tau, float* a, float* b, float* c1, float* c2) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (!s_start || !nsteps || !active || !newly || !tau || !a || !b || !c1 || !c2 || step < 0) return SPHINX_E_INVALID;
  if (grid_kind != SPHINX_GRID_SHARED && grid_kind != SPHINX_GRID_PER_FRAME) return SPHINX_E_INVALID;
  for (int g = 0; g < G; ++g)
    if (s_start[g] < 0 || s_start[g] >= SPHINX_TRAIN_STEPS) return SPHINX_E_INVALID;
  for (int r = 0; r < R; ++r)
    if (nsteps[r] < 1) return SPHINX_E_INVALID;
  const std::vector<double> ab = alpha_bar_table();
  auto ddim = [&](int t, int tn, double* o1, double* o2) {
    const double ac = alpha_bar_at(ab, t), an = alpha_bar_at(ab, tn);
    *o1 = std::sqrt(an / ac);
    *o2 = std::sqrt(1.0 - an) - std::sqrt(an * (1.0 - ac) / ac);
  };
  for (int r = 0; r < R; ++r) {
    const int F = T.frames[r], g0 = T.frame_off[r], n = nsteps[r];
    const bool live = step < n;
    if (grid_kind == SPHINX_GRID_PER_FRAME) {
      for (int f = 0; f < F; ++f) {
        const int g = g0 + f, s = s_start[g];
        auto grid = [&](int i) { return (int)(((int64_t)(n - i) * (s + 1)) / n) - 1; };
        const int t = live ? grid(step) : -1;
        double cc1 = 1.0, cc2 = 0.0;
        if (live) ddim(t, grid(step + 1), &cc1, &cc2);
        const bool nw = live && step == 0;
        active[g] = live ? 1 : 0;
        newly[g] = nw ? 1 : 0;
        tau[g] = t;
        a[g] = nw ? (float)std::sqrt(alpha_bar_at(ab, t)) : 1.0f;
        b[g] = nw ? (float)std::sqrt(1.0 - alpha_bar_at(ab, t)) : 0.0f;
        c1[g] = (float)cc1;
        c2[g] = (float)cc2;
      }
      continue;
    }
    int smax = 0;
    for (int f = 0; f < F; ++f) smax = std::max(smax, s_start[g0 + f]);
    auto grid = [&](int i) { return (int)(((int64_t)(n - i) * (smax + 1)) / n) - 1; };
    const int t = live ? grid(step) : -1;
    double cc1 = 1.0, cc2 = 0.0;
    if (live) ddim(t, grid(step + 1), &cc1, &cc2);
    for (int f = 0; f < F; ++f) {
      const int g = g0 + f;
      const bool act = live && t <= s_start[g];
      const bool nw = act && (step == 0 || grid(step - 1) > s_start[g]);
      active[g] = act ? 1 : 0;
      newly[g] = nw ? 1 : 0;
      tau[g] = t;
      a[g] = nw ? (float)std::sqrt(alpha_bar_at(ab, t)) : 1.0f;
      b[g] = nw ? (float)std::sqrt(1.0 - alpha_bar_at(ab, t)) : 0.0f;
      c1[g] = act ? (float)cc1 : 1.0f;
      c2[g] = act ? (float)cc2 : 0.0f;
    }
  }
  return SPHINX_OK;
}

sphinx_status sphinx_plan_step(const sphinx_request* reqs, int32_t R, const int32_t* s_start, const int32_t* nsteps,
                               int32_t step, uint8_t* active, uint8_t* newly, int32_t* tau, float* a, float* b,
                               float* c1, float* c2) {
  return sphinx_plan_step_grid(reqs, R, s_start, nsteps, step, SPHINX_GRID_SHARED, active, newly, tau, a, b, c1,
                               c2);
}

sphinx_status sphinx_plan_cache(const sphinx_request* reqs, int32_t R, const int32_t* s_start, const int32_t* nsteps,
                                int32_t step, int32_t period, sphinx_grid grid_kind, uint8_t* full,
                                uint8_t* forward_all, float* a_ctx, float* b_ctx) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (!s_start || !nsteps || !full || !forward_all || !a_ctx || !b_ctx || step < 0 || period < 1)
    return SPHINX_E_INVALID;
  if (grid_kind != SPHINX_GRID_SHARED && grid_kind != SPHINX_GRID_PER_FRAME) return SPHINX_E_INVALID;
  for (int g = 0; g < G; ++g)
    if (s_start[g] < 0 || s_start[g] >= SPHINX_TRAIN_STEPS) return SPHINX_E_INVALID;
  for (int r = 0; r < R; ++r)
    if (nsteps[r] < 1) return SPHINX_E_INVALID;
  const std::vector<double> ab = alpha_bar_table();
  for (int r = 0; r < R; ++r) {
    const int F = T.frames[r], g0 = T.frame_off[r], n = nsteps[r];
    int smax = 0;
    for (int f = 0; f < F; ++f) smax = std::max(smax, s_start[g0 + f]);
    const bool live = step < n;
    const int t = live ? (int)(((int64_t)(n - step) * (smax + 1)) / n) - 1 : -1;
    full[r] = (live && step % period == 0) ? 1 : 0;
    for (int f = 0; f < F; ++f) {
      const int g = g0 + f;
      // the frame's own timestep on a per-frame grid
      const int tf = (grid_kind == SPHINX_GRID_PER_FRAME && live)
                         ? (int)(((int64_t)(n - step) * (s_start[g] + 1)) / n) - 1
                         : t;
      forward_all[g] = full[r];
      a_ctx[g] = live ? (float)std::sqrt(alpha_bar_at(ab, tf)) : 1.0f;
      b_ctx[g] = live ? (float)std::sqrt(1.0 - alpha_bar_at(ab, tf)) : 0.0f;
    }
  }
  return SPHINX_OK;
}

sphinx_status sphinx_adaptive_start(const sphinx_request* reqs, int32_t R, const float* q_in, const float* q_reg,
                                    float gamma, const sphinx_klogic* tables, int32_t n_tables,
                                    const int32_t* cluster, int32_t S, int32_t* k, int32_t* s_start,
                                    int32_t* nsteps, double* ratio) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (!q_in || !q_reg || !tables || !cluster || !k || !s_start || !nsteps) return SPHINX_E_INVALID;
  if (!(gamma > 0.0f && gamma <= 1.0f) || S < 1 || S > 1000 || n_tables < 1) return SPHINX_E_INVALID;
  for (int c = 0; c < n_tables; ++c) {
    const sphinx_klogic& t = tables[c];
    if (t.n < 0 || t.n > SPHINX_KLOGIC_MAX) return SPHINX_E_INVALID;
    for (int i = 0; i < t.n; ++i)
      if (!std::isfinite(t.ratio[i]) || (i > 0 && !(t.ratio[i] > t.ratio[i - 1]))) return SPHINX_E_INVALID;
    for (int i = 0; i <= t.n; ++i)
      if (t.k[i] < 0 || t.k[i] >= S || (i > 0 && t.k[i] < t.k[i - 1])) return SPHINX_E_INVALID;
  }
  for (int r = 0; r < R; ++r) {
    if (cluster[r] < 0 || cluster[r] >= n_tables) return SPHINX_E_INVALID;
    if (!(q_in[2 * r] > 0.0f) || !(q_in[2 * r + 1] > 0.0f) || !std::isfinite(q_in[2 * r]) ||
        !std::isfinite(q_in[2 * r + 1]))
      return SPHINX_E_INVALID;
  }
  for (int g = 0; g < G; ++g)
    if (!(q_reg[g] >= 0.0f) || !std::isfinite(q_reg[g])) return SPHINX_E_INVALID;
  for (int r = 0; r < R; ++r) {
    const int F = T.frames[r], g0 = T.frame_off[r];
    const double c0 = q_in[2 * r], c1 = q_in[2 * r + 1];
    const sphinx_klogic& tab = tables[cluster[r]];
    int kmin = S;
    for (int f = 0; f < F; ++f) {
      const int g = g0 + f;
      const double t = (double)(f + 1) / (double)(F + 1);
      const double ft = c1 >= c0 ? std::pow(t, (double)gamma) : 1.0 - std::pow(1.0 - t, (double)gamma);
      const double q_ref = c0 + (c1 - c0) * ft;
      const double rat = (double)q_reg[g] / q_ref;
      int i = 0;
      while (i < tab.n && rat >= (double)tab.ratio[i]) ++i;
      k[g] = tab.k[i];
      // round(1000 (S - k) / S) half up, minus 1
      const int64_t num = 1000 * (int64_t)(S - k[g]);
      s_start[g] = (int32_t)((2 * num + S) / (2 * (int64_t)S)) - 1;
      if (ratio != nullptr) ratio[g] = rat;
      kmin = std::min(kmin, k[g]);
    }
    nsteps[r] = S - kmin;
  }
  return SPHINX_OK;
}

sphinx_status sphinx_select_workspace_bytes(int64_t N, size_t* bytes) {
  if (bytes == nullptr || N < 1) return SPHINX_E_INVALID;
  if (N >= (int64_t)INT32_MAX) return SPHINX_E_UNSUPPORTED;
  *bytes = select_ws_bytes(N);
  return SPHINX_OK;
}

sphinx_status sphinx_select_mask(const sphinx_request* reqs, int32_t R, const float* uncert, const float* thr,
                                 const uint8_t* active, uint8_t* mask, int32_t* idx, int32_t* cu_sel,
                                 int32_t* cu_sel_host, void* ws, size_t ws_bytes, void* stream) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (!uncert || !thr || !mask || !idx || !cu_sel || !ws) return SPHINX_E_INVALID;
  if (!aligned(uncert, 16) || !aligned(mask, 16) || !aligned(idx, 16) || !aligned(cu_sel, 16) || !aligned(ws, 16))
    return SPHINX_E_INVALID;
  if (ws_bytes < select_ws_bytes(N)) return SPHINX_E_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  {
    Bracket br(SPHINX_K_SELECT, s);
    SPHINX_TRY(launch_select(T, N, uncert, thr, active, mask, idx, cu_sel, ws, s));
  }
  if (cu_sel_host != nullptr) {
    SPHINX_TRY(hipMemcpyAsync(cu_sel_host, cu_sel, (size_t)(R + 1) * sizeof(int32_t), hipMemcpyDeviceToHost, s));
    SPHINX_TRY(hipStreamSynchronize(s));
  }
  return SPHINX_OK;
}

sphinx_status sphinx_select_mask_static(const sphinx_request* reqs, int32_t R, const float* uncert,
                                        const float* thr, const uint8_t* active, uint8_t* mask, int32_t* idx,
                                        int32_t* cu_sel, int32_t* cu_sel_host, void* stream) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (!uncert || !thr || !mask || !idx || !cu_sel) return SPHINX_E_INVALID;
  if (!aligned(uncert, 16) || !aligned(mask, 16) || !aligned(idx, 16) || !aligned(cu_sel, 16))
    return SPHINX_E_INVALID;
  if (N > select_static_max_tokens()) return SPHINX_E_UNSUPPORTED;
  hipStream_t s = (hipStream_t)stream;
  void* ws = nullptr;
  SPHINX_TRY(select_static_ws(&ws));
  {
    Bracket br(SPHINX_K_SELECT, s);
    SPHINX_TRY(launch_select(T, N, uncert, thr, active, mask, idx, cu_sel, ws, s));
  }
  if (cu_sel_host != nullptr) {
    SPHINX_TRY(hipMemcpyAsync(cu_sel_host, cu_sel, (size_t)(R + 1) * sizeof(int32_t), hipMemcpyDeviceToHost, s));
    SPHINX_TRY(hipStreamSynchronize(s));
  }
  return SPHINX_OK;
}

sphinx_status sphinx_gather(const sphinx_request* reqs, int32_t R, sphinx_layout layout, const void* state,
                            sphinx_dtype state_dtype, const void* eps, sphinx_dtype eps_dtype, const int32_t* idx,
                            int32_t n_sel, const float* a, const float* b, float* x_sel, void* stream) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (n_sel < 0 || n_sel > N) return SPHINX_E_INVALID;
  if (!valid_dtype(state_dtype) || !valid_dtype(eps_dtype) || !valid_layout(layout)) return SPHINX_E_UNSUPPORTED;
  if (n_sel == 0) return SPHINX_OK;
  if (!state || !idx || !a || !b || !x_sel) return SPHINX_E_INVALID;
  if (!aligned(state, 16) || (eps && !aligned(eps, 16)) || !aligned(idx, 16) || !aligned(x_sel, 16))
    return SPHINX_E_INVALID;
  Bracket br(SPHINX_K_GATHER, (hipStream_t)stream);
  return hip_status(launch_gather(T, layout, state, state_dtype, eps, eps_dtype, idx, n_sel, a, b,
                                  GatherCtx{nullptr, nullptr, nullptr}, x_sel, (hipStream_t)stream));
}

sphinx_status sphinx_gather_ctx(const sphinx_request* reqs, int32_t R, sphinx_layout layout, const void* state,
                                sphinx_dtype state_dtype, const void* eps, sphinx_dtype eps_dtype, const int32_t* idx,
                                int32_t n, const uint8_t* wmask, const float* a, const float* b, const float* a_ctx,
                                const float* b_ctx, float* x, void* stream) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (n < 0 || n > N) return SPHINX_E_INVALID;
  if (!valid_dtype(state_dtype) || !valid_dtype(eps_dtype) || !valid_layout(layout)) return SPHINX_E_UNSUPPORTED;
  if (n == 0) return SPHINX_OK;
  if (!state || !idx || !wmask || !a || !b || !a_ctx || !b_ctx || !x) return SPHINX_E_INVALID;
  if (!aligned(state, 16) || (eps && !aligned(eps, 16)) || !aligned(idx, 16) || !aligned(x, 16))
    return SPHINX_E_INVALID;
  Bracket br(SPHINX_K_GATHER, (hipStream_t)stream);
  return hip_status(launch_gather(T, layout, state, state_dtype, eps, eps_dtype, idx, n, a, b,
                                  GatherCtx{wmask, a_ctx, b_ctx}, x, (hipStream_t)stream));
}

sphinx_status sphinx_refine_workspace_bytes(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R,
                                            int64_t max_sel, size_t* bytes) {
  sphinx_status st = check_model(m);
  if (st != SPHINX_OK) return st;
  ReqTable T;
  int64_t N;
  int32_t G;
  st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (bytes == nullptr || max_sel < 0 || max_sel > N) return SPHINX_E_INVALID;
  *bytes = refine_layout(*m, T, G, std::max<int64_t>(max_sel, 1)).total;
  return SPHINX_OK;
}

sphinx_status sphinx_kv_cache_bytes(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R,
                                    size_t* bytes) {
  sphinx_status st = check_model(m);
  if (st != SPHINX_OK) return st;
  ReqTable T;
  int64_t N;
  int32_t G;
  st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (bytes == nullptr) return SPHINX_E_INVALID;
  *bytes = (size_t)m->L * (size_t)N * 2 * (size_t)m->D * esize(m->dtype);
  return SPHINX_OK;
}

namespace {
// One denoiser pass plus the DDIM update over the n forwarded rows; with a
// cache (kv_cache != NULL) every block stores the rows' keys and values and
// attends over all tokens of each request through the cache.
sphinx_status refine_impl(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R, const int32_t* idx,
                          int32_t n_sel, const int32_t* cu_sel_host, const int32_t* tau, const float* c1,
                          const float* c2, float* x_sel, void* kv_cache, void* ws, size_t ws_bytes, void* stream) {
  sphinx_status st = check_model(m);
  if (st != SPHINX_OK) return st;
  ReqTable T;
  int64_t N;
  int32_t G;
  st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (n_sel < 0 || n_sel > N || cu_sel_host == nullptr) return SPHINX_E_INVALID;
  if (cu_sel_host[0] != 0 || cu_sel_host[R] != n_sel) return SPHINX_E_INVALID;
  for (int r = 0; r < R; ++r) {
    const int64_t len = (int64_t)cu_sel_host[r + 1] - cu_sel_host[r];
    if (len < 0 || len > T.tok_off[r + 1] - T.tok_off[r]) return SPHINX_E_INVALID;
  }
  if (n_sel == 0) return SPHINX_OK;
  // GEMM operand tiles are addressed with 32-bit element offsets: the widest
  // activation matrix (n x max(3D, mlp)) must stay below 2^31 elements
  if ((int64_t)n_sel * std::max(3 * (int64_t)m->D, (int64_t)m->mlp) >= ((int64_t)1 << 31))
    return SPHINX_E_UNSUPPORTED;
  if (!idx || !tau || !c1 || !c2 || !x_sel || !ws || m->weights == nullptr) return SPHINX_E_INVALID;
  if (!aligned(idx, 16) || !aligned(x_sel, 16) || !aligned(ws, 256) || !aligned(m->weights, 256))
    return SPHINX_E_INVALID;
  if (kv_cache != nullptr && !aligned(kv_cache, 16)) return SPHINX_E_INVALID;
  const bool factorised = m->attention == SPHINX_ATTN_FACTORISED;
  if (factorised) {
    if (G > SPHINX_MAX_REQUESTS) return SPHINX_E_UNSUPPORTED;
    if (m->dtype == SPHINX_F32 && m->head_dim % 4 != 0) return SPHINX_E_UNSUPPORTED;  // 16-byte head rows
    for (int r = 0; r < R; ++r)
      if (T.frames[r] > 64) return SPHINX_E_UNSUPPORTED;
  }
  const RefineWs W = refine_layout(*m, T, G, n_sel);
  if (ws_bytes < W.total) return SPHINX_E_WORKSPACE;
  const bool cached = kv_cache != nullptr;

  // segments: requests with forwarded tokens, most keys first for the attention schedule
  SegTable S;
  std::memset(&S, 0, sizeof(S));
  std::vector<int> order;
  for (int r = 0; r < R; ++r)
    if (cu_sel_host[r + 1] > cu_sel_host[r]) order.push_back(r);
  auto keys = [&](int r) {
    return cached ? (int64_t)(T.tok_off[r + 1] - T.tok_off[r]) : (int64_t)(cu_sel_host[r + 1] - cu_sel_host[r]);
  };
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return keys(x) > keys(y); });
  S.nseg = (int)order.size();
  S.tile_prefix[0] = 0;
  for (int i = 0; i < S.nseg; ++i) {
    const int r = order[i];
    S.start[i] = cu_sel_host[r];
    S.len[i] = cu_sel_host[r + 1] - cu_sel_host[r];
    S.kv_start[i] = cached ? (int)T.tok_off[r] : S.start[i];
    S.kv_len[i] = (int)keys(r);
    S.tile_prefix[i + 1] = S.tile_prefix[i] + (S.len[i] + kAttnQueryTile - 1) / kAttnQueryTile;
  }

  hipStream_t s = (hipStream_t)stream;
  unsigned char* base = static_cast<unsigned char*>(ws);
  auto I32 = [&](size_t o) { return reinterpret_cast<int32_t*>(base + o); };
  auto F32 = [&](size_t o) { return reinterpret_cast<float*>(base + o); };
  const Blob B = blob_layout(*m);
  const unsigned char* wb = static_cast<const unsigned char*>(m->weights);
  auto P = [&](sphinx_param p, int l) { return static_cast<const void*>(wb + B.at(p, l)); };
  const sphinx_dtype dt = m->dtype;
  const int D = m->D, n = n_sel;
  const int ldm = (6 * m->L + 2) * D;
  int32_t* U = I32(W.U);
  float* mod = F32(W.mod);
  int32_t* crow = I32(W.crow);
  float* h = F32(W.h);
  void* abuf = base + W.a;
  void* qkv = base + W.big;
  void* obuf = base + W.big + (size_t)n * 3 * D * esize(dt);
  void* mbuf = base + W.big;

  // factorised: frame segments (host copy of the per-frame counts: one stream
  // synchronisation) and the token -> row map of the temporal blocks
  SegTable Sf;
  std::memset(&Sf, 0, sizeof(Sf));
  if (factorised) {
    std::vector<int32_t> first(G + 1);
    SPHINX_TRY(launch_frame_bounds(T, idx, n, G, I32(W.fcnt), s));
    SPHINX_TRY(hipMemcpyAsync(first.data(), I32(W.fcnt), (size_t)(G + 1) * 4, hipMemcpyDeviceToHost, s));
    SPHINX_TRY(hipStreamSynchronize(s));
    // an idx outside [0, N) or out of order: rejected before any further launch
    if (first[0] != 0 || first[G] != n) return SPHINX_E_INVALID;
    std::vector<int> frames;
    std::vector<int> fstart(G), cnt(G);
    for (int g = 0; g < G; ++g) {
      if (first[g + 1] < first[g]) return SPHINX_E_INVALID;
      fstart[g] = first[g];
      cnt[g] = first[g + 1] - first[g];
      if (cnt[g] > 0) frames.push_back(g);
    }
    SPHINX_TRY(launch_pos_map(N, idx, n, I32(W.pos), s));
    auto frame_keys = [&](int g) {
      int r = 0;
      while (r + 1 < R && T.frame_off[r + 1] <= g) ++r;
      return cached ? (T.h[r] / 2) * (T.w[r] / 2) : cnt[g];
    };
    std::stable_sort(frames.begin(), frames.end(), [&](int x, int y) { return frame_keys(x) > frame_keys(y); });
    Sf.nseg = (int)frames.size();
    for (int i = 0; i < Sf.nseg; ++i) {
      const int g = frames[i];
      int r = 0;
      while (r + 1 < R && T.frame_off[r + 1] <= g) ++r;
      const int tpf = (T.h[r] / 2) * (T.w[r] / 2);
      Sf.start[i] = fstart[g];
      Sf.len[i] = cnt[g];
      Sf.kv_start[i] = cached ? (int)(T.tok_off[r] + (int64_t)(g - T.frame_off[r]) * tpf) : fstart[g];
      Sf.kv_len[i] = cached ? tpf : cnt[g];
      Sf.tile_prefix[i + 1] = Sf.tile_prefix[i] + (Sf.len[i] + kAttnQueryTile - 1) / kAttnQueryTile;
    }
  }

  // conditioning: one row per run of frames with equal timestep
  {
  Bracket br(SPHINX_K_COND, s);
  SPHINX_TRY(launch_cond_rows(tau, G, I32(W.fmap), I32(W.utau), U, s));
  SPHINX_TRY(launch_temb(I32(W.utau), U, G, F32(W.temb), s));
  SPHINX_TRY(launch_rowgemm(F32(W.temb), SPHINX_TEMB_DIM, U, SPHINX_TEMB_DIM, P(SPHINX_P_T1_W, 0),
                            P(SPHINX_P_T1_B, 0), dt, D, true, F32(W.cbuf), D, s));
  SPHINX_TRY(launch_rowgemm(F32(W.cbuf), D, U, D, P(SPHINX_P_T2_W, 0), P(SPHINX_P_T2_B, 0), dt, D, true,
                            F32(W.sc), D, s));
  SPHINX_TRY(launch_rowgemm(F32(W.sc), D, U, D, P(SPHINX_P_COND_W, 0), P(SPHINX_P_COND_B, 0), dt, ldm, false, mod,
                            ldm, s));
  SPHINX_TRY(launch_pos_tables(D, W.maxHp, W.maxWp, W.maxF, F32(W.Ty), F32(W.Tx), F32(W.Tf), s));
  SPHINX_TRY(launch_token_meta(T, idx, n, I32(W.fmap), I32(W.gframe), crow, I32(W.posc), s));
  }
  {
  Bracket br(SPHINX_K_EMBED, s);
  SPHINX_TRY(launch_embed(x_sel, n, D, P(SPHINX_P_PE_W, 0), P(SPHINX_P_PE_B, 0), dt, F32(W.Ty), F32(W.Tx),
                          F32(W.Tf), I32(W.posc), h, s));
  }
  for (int l = 0; l < m->L; ++l) {
    const int c0 = 6 * D * l;
    {
      Bracket br(SPHINX_K_LN, s);
      SPHINX_TRY(launch_ln_mod(h, n, D, mod, ldm, c0, c0 + D, crow, abuf, dt, s));
    }
    {
      Bracket br(SPHINX_K_GEMM_QKV, s);
      // q leaves the projection scaled by log2(e)/sqrt(head_dim), rounded once:
      // attention scores then come out of q k^T in base-2 units
      GemmEpi e_qkv{qkv, 3 * D, nullptr, 0, nullptr, D, kLog2e / std::sqrt((float)m->head_dim)};
      SPHINX_TRY(launch_gemm(EPI_BIAS, dt, abuf, P(SPHINX_P_QKV_W, l), P(SPHINX_P_QKV_B, l), n, 3 * D, D, e_qkv, s));
    }
    AttnIO io{qkv, static_cast<const unsigned char*>(qkv) + (size_t)D * esize(dt),
              static_cast<const unsigned char*>(qkv) + 2 * (size_t)D * esize(dt), obuf, 3 * D, 3 * D};
    if (cached) {
      unsigned char* cl = static_cast<unsigned char*>(kv_cache) + (size_t)l * (size_t)N * 2 * D * esize(dt);
      Bracket br(SPHINX_K_KV_STORE, s);
      SPHINX_TRY(launch_kv_store(dt, qkv, n, D, idx, N, cl, s));
      io.k = cl;
      io.v = cl + (size_t)D * esize(dt);
      io.ldkv = 2 * D;
    }
    {
      Bracket br(SPHINX_K_ATTENTION, s);
      if (!factorised)
        SPHINX_TRY(launch_attention(dt, io, D, m->heads, m->head_dim, n, S, s));
      else if (l % 2 == 0)  // spatial: within the frame
        SPHINX_TRY(launch_attention(dt, io, D, m->heads, m->head_dim, n, Sf, s));
      else  // temporal: across the request's frames at the same position
        SPHINX_TRY(launch_attn_temporal(dt, T, io, D, m->heads, m->head_dim, I32(W.pos), cached, s));
    }
    {
      Bracket br(SPHINX_K_GEMM_OUT, s);
      GemmEpi e_o{h, D, mod + c0 + 2 * D, ldm, crow};
      SPHINX_TRY(launch_gemm(EPI_GATED, dt, obuf, P(SPHINX_P_O_W, l), P(SPHINX_P_O_B, l), n, D, D, e_o, s));
    }
    {
      Bracket br(SPHINX_K_LN, s);
      SPHINX_TRY(launch_ln_mod(h, n, D, mod, ldm, c0 + 3 * D, c0 + 4 * D, crow, abuf, dt, s));
    }
    {
      Bracket br(SPHINX_K_GEMM_MLP1, s);
      GemmEpi e_1{mbuf, m->mlp, nullptr, 0, nullptr};
      SPHINX_TRY(launch_gemm(EPI_GELU, dt, abuf, P(SPHINX_P_FC1_W, l), P(SPHINX_P_FC1_B, l), n, m->mlp, D, e_1, s));
    }
    {
      Bracket br(SPHINX_K_GEMM_MLP2, s);
      GemmEpi e_2{h, D, mod + c0 + 5 * D, ldm, crow};
      SPHINX_TRY(
          launch_gemm(EPI_GATED, dt, mbuf, P(SPHINX_P_FC2_W, l), P(SPHINX_P_FC2_B, l), n, D, m->mlp, e_2, s));
    }
  }
  const int cf = 6 * D * m->L;
  Bracket br(SPHINX_K_FINAL, s);
  SPHINX_TRY(launch_final(h, n, D, mod, ldm, cf, cf + D, crow, I32(W.gframe), P(SPHINX_P_OUT_W, 0),
                          P(SPHINX_P_OUT_B, 0), dt, c1, c2, x_sel, s));
  return SPHINX_OK;
}
}  // namespace

sphinx_status sphinx_refine_step(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R,
                                 const int32_t* idx, int32_t n_sel, const int32_t* cu_sel_host,
                                 const int32_t* tau, const float* c1, const float* c2, float* x_sel, void* ws,
                                 size_t ws_bytes, void* stream) {
  return refine_impl(m, reqs, R, idx, n_sel, cu_sel_host, tau, c1, c2, x_sel, nullptr, ws, ws_bytes, stream);
}

sphinx_status sphinx_refine_step_cached(const sphinx_model_desc* m, const sphinx_request* reqs, int32_t R,
                                        const int32_t* idx, int32_t n, const int32_t* cu_host, const int32_t* tau,
                                        const float* c1, const float* c2, float* x, void* kv_cache, void* ws,
                                        size_t ws_bytes, void* stream) {
  if (kv_cache == nullptr) return SPHINX_E_INVALID;
  return refine_impl(m, reqs, R, idx, n, cu_host, tau, c1, c2, x, kv_cache, ws, ws_bytes, stream);
}

sphinx_status sphinx_varlen_attention(sphinx_dtype dtype, int32_t heads, int32_t head_dim, const void* q,
                                      int32_t ldq, const void* k, const void* v, int32_t ldkv, void* o,
                                      const int32_t* cu_q, const int32_t* cu_kv, int32_t nseg, void* stream) {
  if (!valid_dtype(dtype)) return SPHINX_E_UNSUPPORTED;
  if (heads < 1 || head_dim < 1 || nseg < 1 || !cu_q || !cu_kv) return SPHINX_E_INVALID;
  if (nseg > SPHINX_MAX_REQUESTS) return SPHINX_E_UNSUPPORTED;
  if (dtype == SPHINX_BF16 ? (head_dim != 64 && head_dim != 72) : head_dim > 64) return SPHINX_E_UNSUPPORTED;
  const int64_t D = (int64_t)heads * head_dim;
  if (D > 4096 || ldq < D || ldkv < D || ldq % 8 != 0 || ldkv % 8 != 0) return SPHINX_E_INVALID;
  if (cu_q[0] != 0 || cu_kv[0] != 0) return SPHINX_E_INVALID;
  for (int i = 0; i < nseg; ++i) {
    if (cu_q[i + 1] < cu_q[i] || cu_kv[i + 1] < cu_kv[i]) return SPHINX_E_INVALID;
    if (cu_q[i + 1] > cu_q[i] && cu_kv[i + 1] == cu_kv[i]) return SPHINX_E_INVALID;
  }
  const int64_t nq = cu_q[nseg], nkv = cu_kv[nseg];
  if (nq == 0) return SPHINX_OK;
  if (!q || !k || !v || !o || !aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16))
    return SPHINX_E_INVALID;
  if (nq * ldq >= ((int64_t)1 << 31) || nkv * ldkv >= ((int64_t)1 << 31) || nq * D >= ((int64_t)1 << 31))
    return SPHINX_E_UNSUPPORTED;
  SegTable S;
  std::memset(&S, 0, sizeof(S));
  std::vector<int> order;
  for (int i = 0; i < nseg; ++i)
    if (cu_q[i + 1] > cu_q[i]) order.push_back(i);
  std::stable_sort(order.begin(), order.end(),
                   [&](int x, int y) { return cu_kv[x + 1] - cu_kv[x] > cu_kv[y + 1] - cu_kv[y]; });
  S.nseg = (int)order.size();
  for (int j = 0; j < S.nseg; ++j) {
    const int i = order[j];
    S.start[j] = cu_q[i];
    S.len[j] = cu_q[i + 1] - cu_q[i];
    S.kv_start[j] = cu_kv[i];
    S.kv_len[j] = cu_kv[i + 1] - cu_kv[i];
    S.tile_prefix[j + 1] = S.tile_prefix[j] + (S.len[j] + kAttnQueryTile - 1) / kAttnQueryTile;
  }
  const AttnIO io{q, k, v, o, ldq, ldkv};
  hipStream_t s = (hipStream_t)stream;
  Bracket br(SPHINX_K_ATTENTION, s);
  return hip_status(launch_attention(dtype, io, (int)D, heads, head_dim, (int)nq, S, s));
}

sphinx_status sphinx_scatter_blend(const sphinx_request* reqs, int32_t R, const float* x_sel, const int32_t* idx,
                                   int32_t n_sel, const void* z_in, sphinx_dtype in_dtype, sphinx_layout in_layout,
                                   void* z_out, sphinx_dtype out_dtype, sphinx_layout out_layout, void* stream) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (!valid_dtype(in_dtype) || !valid_dtype(out_dtype)) return SPHINX_E_UNSUPPORTED;
  if (!valid_layout(in_layout) || !valid_layout(out_layout)) return SPHINX_E_UNSUPPORTED;
  if (n_sel < 0 || n_sel > N || z_in == nullptr || z_out == nullptr) return SPHINX_E_INVALID;
  if (!aligned(z_in, 16) || !aligned(z_out, 16)) return SPHINX_E_INVALID;
  if (n_sel > 0 && (!x_sel || !idx || !aligned(x_sel, 16) || !aligned(idx, 16))) return SPHINX_E_INVALID;
  const bool in_place = (z_in == (const void*)z_out);
  if (in_place && (in_dtype != out_dtype || in_layout != out_layout)) return SPHINX_E_INVALID;
  if (!in_place) {
    const uintptr_t i0 = (uintptr_t)z_in, i1 = i0 + (uintptr_t)(16 * N) * dtype_bytes(in_dtype);
    const uintptr_t o0 = (uintptr_t)z_out, o1 = o0 + (uintptr_t)(16 * N) * dtype_bytes(out_dtype);
    if (i0 < o1 && o0 < i1) return SPHINX_E_INVALID;  // partial overlap
  }
  hipStream_t s = (hipStream_t)stream;
  Bracket br(SPHINX_K_SCATTER, s);
  if (!in_place) SPHINX_TRY(launch_convert(T, z_in, in_dtype, in_layout, z_out, out_dtype, out_layout, s));
  if (n_sel > 0) SPHINX_TRY(launch_scatter(T, x_sel, idx, n_sel, nullptr, z_out, out_dtype, out_layout, s));
  return SPHINX_OK;
}

sphinx_status sphinx_scatter_masked(const sphinx_request* reqs, int32_t R, const float* x, const int32_t* idx,
                                    int32_t n, const uint8_t* wmask, void* z, sphinx_dtype dtype,
                                    sphinx_layout layout, void* stream) {
  ReqTable T;
  int64_t N;
  int32_t G;
  sphinx_status st = build_table(reqs, R, &T, &N, &G);
  if (st != SPHINX_OK) return st;
  if (!valid_dtype(dtype) || !valid_layout(layout)) return SPHINX_E_UNSUPPORTED;
  if (n < 0 || n > N) return SPHINX_E_INVALID;
  if (n == 0) return SPHINX_OK;
  if (!x || !idx || !wmask || !z || !aligned(x, 16) || !aligned(idx, 16) || !aligned(z, 16))
    return SPHINX_E_INVALID;
  hipStream_t s = (hipStream_t)stream;
  Bracket br(SPHINX_K_SCATTER, s);
  return hip_status(launch_scatter(T, x, idx, n, wmask, z, dtype, layout, s));
}

namespace {
sphinx_status front_check(const sphinx_request* reqs, int32_t R, ReqTable* T, int32_t* G) {
  int64_t N;
  sphinx_status st = build_table(reqs, R, T, &N, G);
  if (st != SPHINX_OK) return st;
  for (int r = 0; r < R; ++r)
    if ((int64_t)T->h[r] * T->w[r] > ((int64_t)1 << 20)) return SPHINX_E_UNSUPPORTED;
  return SPHINX_OK;
}
}  // namespace

sphinx_status sphinx_mask_frontend_workspace_bytes(const sphinx_request* reqs, int32_t R, size_t* bytes) {
  ReqTable T;
  int32_t G;
  sphinx_status st = front_check(reqs, R, &T, &G);
  if (st != SPHINX_OK) return st;
  if (bytes == nullptr) return SPHINX_E_INVALID;
  *bytes = front_ws_bytes(T, G);
  return SPHINX_OK;
}

sphinx_status sphinx_mask_frontend(const sphinx_request* reqs, int32_t R, const uint8_t* rgb, const float* opacity,
                                   float tau_o, uint8_t* token_mask, float* uncert, int32_t* otsu_t, void* ws,
                                   size_t ws_bytes, void* stream) {
  ReqTable T;
  int32_t G;
  sphinx_status st = front_check(reqs, R, &T, &G);
  if (st != SPHINX_OK) return st;
  if (!rgb || !opacity || !token_mask || !ws) return SPHINX_E_INVALID;
  if (!aligned(rgb, 16) || !aligned(opacity, 16) || !aligned(token_mask, 16) || !aligned(ws, 256) ||
      (uncert && !aligned(uncert, 16)) || (otsu_t && !aligned(otsu_t, 16)))
    return SPHINX_E_INVALID;
  if (ws_bytes < front_ws_bytes(T, G)) return SPHINX_E_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  Bracket br(SPHINX_K_FRONTEND, s);
  return hip_status(launch_front(T, G, rgb, opacity, tau_o, token_mask, uncert, otsu_t, ws, s));
}

sphinx_status sphinx_timing_enable(int32_t classes) {
  if (classes < 0 || classes >= (1 << SPHINX_K_COUNT)) return SPHINX_E_INVALID;
  Timing& T = timing();
  std::lock_guard<std::mutex> g(T.mu);
  T.resolve();
  if (classes != 0) {
    std::fill(T.launches, T.launches + SPHINX_K_COUNT, 0);
    std::fill(T.ms, T.ms + SPHINX_K_COUNT, 0.0);
  }
  T.mask = (uint32_t)classes;
  return SPHINX_OK;
}

sphinx_status sphinx_timing_read(sphinx_kernel_class k, int64_t* launches, double* total_ms) {
  if ((int)k < 0 || k >= SPHINX_K_COUNT || launches == nullptr || total_ms == nullptr) return SPHINX_E_INVALID;
  Timing& T = timing();
  std::lock_guard<std::mutex> g(T.mu);
  T.resolve();
  *launches = T.launches[k];
  *total_ms = T.ms[k];
  return SPHINX_OK;
}

sphinx_status sphinx_peak_mfma(int32_t iters, int32_t operands, float* out, void* stream) {
  if (iters < 1 || iters > (1 << 24) || out == nullptr || !aligned(out, 16)) return SPHINX_E_INVALID;
  if (operands != SPHINX_PEAK_CONSTANT && operands != SPHINX_PEAK_RANDOM) return SPHINX_E_INVALID;
  return hip_status(launch_peak_mfma(iters, operands == SPHINX_PEAK_RANDOM, out, SPHINX_PEAK_BLOCKS,
                                     (hipStream_t)stream));
}

}  // extern "C"
