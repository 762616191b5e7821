// C interface and host orchestration of Speculative Rejection (section 4.2,
// Algorithm 1) on one MI355X.
//
// The generation loop runs all candidates of one prompt as one batch.  The
// prompt's keys/values are computed once per model and shared by every
// candidate; each candidate owns a tail of its response keys/values in a
// pool whose rows hold `cap` tokens.  At a decision token the reward model
// scores every candidate (prompt prefix + response), the cut keeps the best
// K, completed candidates join the set I, and the survivors' tails are
// packed into the other pool for the next round.  The host synchronises
// with the device once per round (to learn the survivor count).
#include <algorithm>
#include <functional>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "common.h"
#include "kernels.h"

namespace sr {

static thread_local std::string t_err;
void set_error(const std::string& m) { t_err = m; }

static constexpr int64_t kPpm = 1000000;
static constexpr int kMaxN = 4096;

static int64_t alpha_ppm(double alpha) { return (int64_t)std::floor(alpha * 1e6 + 0.5); }
static int keep_of(int b, int64_t appm) { return b - (int)((appm * (int64_t)b) / kPpm); }

struct Dims {
  int nl, d, hq, hkv, hd, ff, V, qkv, dtype, es;
  float theta, eps;
};
static Dims dims_of(const sr_model_config& c) {
  Dims m;
  m.nl = c.n_layers; m.d = c.d_model; m.hq = c.n_heads; m.hkv = c.n_kv_heads; m.hd = c.head_dim;
  m.ff = c.ffn_dim; m.V = c.vocab; m.qkv = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
  m.dtype = c.dtype; m.es = c.dtype == SR_BF16 ? 2 : 4;
  m.theta = c.rope_theta; m.eps = c.rms_eps;
  return m;
}

// ------------------------------------------------------------ validation
static void check_model(const sr_model* m, bool reward, const char* name) {
  std::string n(name);
  SR_REQUIRE(m != nullptr, SR_ERR_INVALID_ARG, n + " is NULL");
  const sr_model_config& c = m->cfg;
  SR_REQUIRE(c.is_reward == (reward ? 1 : 0), SR_ERR_INVALID_ARG,
             n + (reward ? " must be a reward model" : " must be a generator"));
  SR_REQUIRE(c.n_layers >= 1 && c.d_model >= 1 && c.n_heads >= 1 && c.n_kv_heads >= 1 &&
                 c.head_dim >= 1 && c.ffn_dim >= 1 && c.vocab >= 1,
             SR_ERR_INVALID_ARG, n + ": every dimension must be positive");
  SR_REQUIRE(c.dtype == SR_F32 || c.dtype == SR_BF16, SR_ERR_INVALID_ARG, n + ": unknown dtype");
  SR_REQUIRE(c.n_heads % c.n_kv_heads == 0, SR_ERR_INVALID_ARG,
             n + ": n_heads must be a multiple of n_kv_heads");
  SR_REQUIRE(std::isfinite(c.rope_theta) && c.rope_theta > 0.f && std::isfinite(c.rms_eps) &&
                 c.rms_eps >= 0.f,
             SR_ERR_INVALID_ARG, n + ": rope_theta must be > 0 and rms_eps >= 0");
  const int g = c.n_heads / c.n_kv_heads;
  SR_REQUIRE(c.head_dim == 32 || c.head_dim == 64 || c.head_dim == 128, SR_ERR_UNSUPPORTED,
             n + ": head_dim must be 32, 64 or 128");
  SR_REQUIRE(g == 1 || g == 2 || g == 4 || g == 8, SR_ERR_UNSUPPORTED,
             n + ": n_heads / n_kv_heads must be 1, 2, 4 or 8");
  SR_REQUIRE(c.d_model % 64 == 0 && (c.n_heads * c.head_dim) % 64 == 0 && c.ffn_dim % 64 == 0,
             SR_ERR_UNSUPPORTED, n + ": d_model, n_heads*head_dim and ffn_dim must be multiples of 64");
  SR_REQUIRE(c.vocab <= 262144, SR_ERR_UNSUPPORTED, n + ": vocab above 262144");
  const sr_weights& w = m->w;
  SR_REQUIRE(w.embed && w.attn_norm && w.wqkv && w.wo && w.ffn_norm && w.w13 && w.w2 &&
                 w.final_norm && w.head,
             SR_ERR_INVALID_ARG, n + ": a weight pointer is NULL");
}

static void check_pair(const sr_model* gen, const sr_model* rm) {
  check_model(gen, false, "gen");
  check_model(rm, true, "rm");
  SR_REQUIRE(gen->cfg.dtype == rm->cfg.dtype, SR_ERR_INVALID_ARG,
             "gen and rm must have the same dtype");
  SR_REQUIRE(rm->cfg.vocab >= gen->cfg.vocab, SR_ERR_INVALID_ARG,
             "rm vocab must cover the generator's tokens");
}

static void check_params(const sr_params* p, const sr_model* gen) {
  SR_REQUIRE(p != nullptr, SR_ERR_INVALID_ARG, "params is NULL");
  SR_REQUIRE(p->n >= 1 && p->n <= kMaxN, SR_ERR_INVALID_ARG, "n must be in [1, 4096]");
  SR_REQUIRE(p->alpha >= 0.0 && p->alpha < 1.0, SR_ERR_INVALID_ARG, "alpha must be in [0, 1)");
  SR_REQUIRE(p->tau >= 1, SR_ERR_INVALID_ARG, "tau must be >= 1");
  SR_REQUIRE(p->max_new_tokens >= 1, SR_ERR_INVALID_ARG, "max_new_tokens must be >= 1");
  SR_REQUIRE(std::isfinite(p->temperature) && p->temperature >= 0.f, SR_ERR_INVALID_ARG,
             "temperature must be finite and >= 0");
  SR_REQUIRE(p->eos_id >= -1 && p->eos_id < gen->cfg.vocab, SR_ERR_INVALID_ARG,
             "eos_id must be -1 or a token id");
  SR_REQUIRE(p->max_rounds >= 0, SR_ERR_INVALID_ARG, "max_rounds must be >= 0");
  SR_REQUIRE((int64_t)p->n * p->tau <= (int64_t)1 << 31, SR_ERR_INVALID_ARG, "n * tau too large");
  SR_REQUIRE(p->reward_kind == SR_REWARD_MODEL || p->reward_kind == SR_REWARD_LOGPROB, SR_ERR_INVALID_ARG,
             "reward_kind must be SR_REWARD_MODEL or SR_REWARD_LOGPROB");
  SR_REQUIRE(p->reward_recompute == 0 || p->reward_recompute == 1, SR_ERR_INVALID_ARG,
             "reward_recompute must be 0 or 1");
}

// The reward model of a run: `rm`, or (log-probability reward without a
// reward model) a stand-in of the generator's shape that only sizes the
// workspace and is never evaluated.
static const sr_model* reward_model_of(const sr_model* gen, const sr_model* rm, const sr_params* p,
                                       sr_model* stand_in) {
  if (rm != nullptr) return rm;
  SR_REQUIRE(p != nullptr && p->reward_kind == SR_REWARD_LOGPROB && gen != nullptr, SR_ERR_INVALID_ARG,
             "rm is NULL (allowed only with reward_kind = SR_REWARD_LOGPROB)");
  *stand_in = *gen;
  stand_in->cfg.is_reward = 1;
  return stand_in;
}

// ------------------------------------------------------------ planning
struct Plan {
  int N, P, Lmax;
  int64_t appm, B;
  int max_rounds;
  int64_t S[2];  // token-slot capacity of pools A and B
  int Tc;        // tokens per reward-model chunk
  size_t gpart, apart;
  bool rkv;      // the reward model's response K/V is kept across rounds (pools of S[i] slots)
};

// Decision length for a round that starts with b unfinished candidates after
// r cuts (Lmax when nobody can be rejected or the cut budget is spent).
static int decision(const Plan& pl, int b, int r) {
  if (keep_of(b, pl.appm) == b || (pl.max_rounds > 0 && r >= pl.max_rounds)) return pl.Lmax;
  return (int)std::min<int64_t>(pl.Lmax, pl.B / b);
}

static Plan make_plan(const Dims& g, const Dims& rm, int P, const sr_params* p) {
  Plan pl;
  pl.N = p->n; pl.P = P; pl.Lmax = p->max_new_tokens;
  pl.appm = alpha_ppm(p->alpha);
  pl.B = (int64_t)p->n * p->tau;
  pl.max_rounds = p->max_rounds;
  const int D0 = decision(pl, pl.N, 0);
  const bool can_cut = keep_of(pl.N, pl.appm) < pl.N;
  int64_t after = 0;
  if (can_cut) {
    // Rows of a round that runs to Lmax: at most b_skip (no one can be
    // rejected) or the survivors of max_rounds cuts.  Other rounds hold at
    // most floor(B / b) tokens for each of b rows.
    int64_t bskip = pl.appm > 0 ? std::min<int64_t>(pl.N, (kPpm + pl.appm - 1) / pl.appm - 1) : pl.N;
    after = std::max<int64_t>(pl.B, bskip * pl.Lmax);
    if (pl.max_rounds > 0) {
      int b = pl.N;
      for (int r = 0; r < pl.max_rounds; ++r) b = keep_of(b, pl.appm);
      after = std::max<int64_t>(after, (int64_t)b * pl.Lmax);
    }
  }
  pl.S[0] = std::max<int64_t>((int64_t)pl.N * D0, after);
  pl.S[1] = after;
  // A reward-model K/V cache pays off only when some round is scored after
  // an earlier one, i.e. when the first round can end in a cut.
  pl.rkv = p->reward_kind == SR_REWARD_MODEL && !p->reward_recompute && can_cut && D0 < pl.Lmax;
  const int64_t want = std::min<int64_t>((int64_t)pl.N * pl.Lmax, 32768);
  pl.Tc = (int)std::max<int64_t>(std::max<int64_t>(want, pl.Lmax), P);
  // GEMM split-K partials over every shape and row count that can occur.
  const int Mmax = std::max(pl.N, pl.Tc);
  size_t gp = 0;
  for (const Dims* m : {&g, &rm}) {
    if (m->dtype == SR_F32) {
      size_t ncol = std::max({(size_t)m->qkv, (size_t)m->d, (size_t)2 * m->ff, (size_t)m->V});
      gp = std::max(gp, (size_t)Mmax * ncol);
    } else {
      if (m == &g)
        for (int M = 1; M <= pl.N; ++M) {
          gp = std::max(gp, gemm_partial_elems_always(m->dtype, M, m->qkv, m->d));
          gp = std::max(gp, gemm_partial_elems_always(m->dtype, M, m->d, m->hq * m->hd));
          gp = std::max(gp, gemm_partial_elems_always(m->dtype, M, m->d, m->ff));
        }
      for (int M = 1; M <= Mmax; ++M) {
        gp = std::max(gp, gemm_partial_elems(m->dtype, M, m->qkv, m->d, false));
        gp = std::max(gp, gemm_partial_elems(m->dtype, M, m->d, m->hq * m->hd, false));
        gp = std::max(gp, gemm_partial_elems(m->dtype, M, m->ff, m->d, true));
        gp = std::max(gp, gemm_partial_elems(m->dtype, M, m->d, m->ff, false));
        if (m == &g) gp = std::max(gp, gemm_partial_elems(m->dtype, M, m->V, m->d, false));
      }
    }
  }
  pl.gpart = gp;
  size_t ap = 0;
  for (int rows = 1; rows <= pl.N; ++rows) {
    int sp = decode_attn_splits(rows, g.hkv, P + pl.Lmax);
    if (sp > 1) ap = std::max(ap, (size_t)rows * g.hq * sp * (g.hd + 2));
  }
  pl.apart = ap;
  return pl;
}

// ------------------------------------------------------------ workspace
struct Arena {
  char* base;
  size_t off = 0;
  explicit Arena(void* b) : base((char*)b) {}
  template <typename T>
  T* take(size_t n) {
    off = (off + 255) & ~(size_t)255;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += std::max<size_t>(n, 1) * sizeof(T);
    return p;
  }
  void* bytes(size_t n) { return take<char>(n); }
};

struct State {
  int32_t *cand, *len, *done, *tok;
};

struct Layout {
  float2 *rope_g, *rope_r;
  void *gpre, *rpre;        // [nl][2][hkv][P][hd]
  void* pool[2];            // [nl][2][S * hkv * hd]
  void* rpool[2];           // reward model's, same slots (when Plan::rkv)
  int32_t* store;           // [N][Lmax]
  int32_t* cand_len;        // [N]
  State st[3];
  int32_t *i_cand, *i_len, *i_count, *best, *count, *count2;
  float *i_score, *score, *score2;
  float* lp_sum;            // [N] running ln p of each candidate's response (indexed by candidate)
  int32_t *accept, *src_row, *src_row2, *src_tmp;
  float* h; void* xn; float* qkv; float* q; void* o; void* u; float* logits; float* apart;
  int32_t* ctok; int32_t* clen; float* ch; void* cxn; float* cqkv; float* cq; void* ck; void* cv;
  void* co; void* cu;
  float* gpart;
};

static Layout carve(void* base, const Dims& g, const Dims& rm, const Plan& pl, size_t* total) {
  Arena a(base);
  Layout L;
  const int N = pl.N, P = pl.P, Lmax = pl.Lmax;
  L.rope_g = a.take<float2>((size_t)(P + Lmax + 1) * (g.hd / 2));
  L.rope_r = a.take<float2>((size_t)(P + Lmax + 1) * (rm.hd / 2));
  L.gpre = a.bytes((size_t)g.nl * 2 * g.hkv * P * g.hd * g.es);
  L.rpre = a.bytes((size_t)rm.nl * 2 * rm.hkv * P * rm.hd * rm.es);
  for (int i = 0; i < 2; ++i) L.pool[i] = a.bytes((size_t)g.nl * 2 * pl.S[i] * g.hkv * g.hd * g.es);
  for (int i = 0; i < 2; ++i)
    L.rpool[i] = a.bytes(pl.rkv ? (size_t)rm.nl * 2 * pl.S[i] * rm.hkv * rm.hd * rm.es : 0);
  L.store = a.take<int32_t>((size_t)N * Lmax);
  L.cand_len = a.take<int32_t>(N);
  for (int i = 0; i < 3; ++i) {
    L.st[i].cand = a.take<int32_t>(N);
    L.st[i].len = a.take<int32_t>(N);
    L.st[i].done = a.take<int32_t>(N);
    L.st[i].tok = a.take<int32_t>(N);
  }
  L.i_cand = a.take<int32_t>(N); L.i_len = a.take<int32_t>(N); L.i_score = a.take<float>(N);
  L.i_count = a.take<int32_t>(1); L.best = a.take<int32_t>(1);
  L.count = a.take<int32_t>(1); L.count2 = a.take<int32_t>(1);
  L.score = a.take<float>(N); L.score2 = a.take<float>(N);
  L.lp_sum = a.take<float>(N);
  L.accept = a.take<int32_t>(N); L.src_row = a.take<int32_t>(N); L.src_row2 = a.take<int32_t>(N);
  L.src_tmp = a.take<int32_t>(N);
  L.h = a.take<float>((size_t)N * g.d);
  L.xn = a.bytes((size_t)N * std::max(g.d, g.hq * g.hd) * g.es);
  L.qkv = a.take<float>((size_t)N * g.qkv);
  L.q = a.take<float>((size_t)N * g.hq * g.hd);
  L.o = a.bytes((size_t)N * g.hq * g.hd * g.es);
  L.u = a.bytes((size_t)N * g.ff * g.es);
  L.logits = a.take<float>((size_t)N * g.V);
  L.apart = a.take<float>(pl.apart);
  const int Tc = pl.Tc;
  const int cd = std::max(g.d, rm.d), cqkv = std::max(g.qkv, rm.qkv);
  const int chq = std::max(g.hq * g.hd, rm.hq * rm.hd), cff = std::max(g.ff, rm.ff);
  const int ckv = std::max(g.hkv * g.hd, rm.hkv * rm.hd);
  L.ctok = a.take<int32_t>(Tc);
  L.clen = a.take<int32_t>(N);
  L.ch = a.take<float>((size_t)Tc * cd);
  L.cxn = a.bytes((size_t)Tc * std::max(cd, chq) * g.es);
  L.cqkv = a.take<float>((size_t)Tc * cqkv);
  L.cq = a.take<float>((size_t)Tc * chq);
  L.ck = a.bytes((size_t)Tc * ckv * g.es);
  L.cv = a.bytes((size_t)Tc * ckv * g.es);
  L.co = a.bytes((size_t)Tc * chq * g.es);
  L.cu = a.bytes((size_t)Tc * cff * g.es);
  L.gpart = a.take<float>(pl.gpart);
  *total = a.off + 256;
  return L;
}

// ------------------------------------------------------------ model passes
struct Model {
  Dims m;
  const sr_weights* w;
  const char* wb(const void* p, int64_t elems) const { return (const char*)p + elems * m.es; }
  const void* attn_norm(int l) const { return wb(w->attn_norm, (int64_t)l * m.d); }
  const void* ffn_norm(int l) const { return wb(w->ffn_norm, (int64_t)l * m.d); }
  const void* wqkv(int l) const { return wb(w->wqkv, (int64_t)l * m.qkv * m.d); }
  const void* wo(int l) const { return wb(w->wo, (int64_t)l * m.d * m.hq * m.hd); }
  const void* w13(int l) const { return wb(w->w13, (int64_t)l * 2 * m.ff * m.d); }
  const void* w2(int l) const { return wb(w->w2, (int64_t)l * m.d * m.ff); }
};

thread_local LaunchTiming* launch_timing = nullptr;

// Optional per-kernel-class timing with HIP events on the caller's stream,
// stamped by the kernels' own dispatch packets (SR_LAUNCH): a timed call
// spans from its first kernel's start to its last kernel's end.
struct Profiler {
  hipStream_t s = nullptr;
  bool active = false;
  // Launches are recorded in batches that alternate between two event
  // pools: `recs` (pool[cur]) is being recorded, `prev` (pool[cur ^ 1]) is
  // the batch before it.
  std::vector<hipEvent_t> pool[2];
  int cur = 0;
  size_t used = 0;
  struct Rec {
    int cls;
    size_t e0, e1;
    double bytes, flops;
  };
  std::vector<Rec> recs, prev;
  double sec[SR_K_NCLASS] = {}, bytes[SR_K_NCLASS] = {}, flops[SR_K_NCLASS] = {};
  int64_t n[SR_K_NCLASS] = {};
  ~Profiler() {
    for (auto& p : pool)
      for (hipEvent_t e : p) (void)hipEventDestroy(e);
  }
  // the next unused event of the batch being recorded
  size_t slot() {
    std::vector<hipEvent_t>& p = pool[cur];
    if (used == p.size()) {
      hipEvent_t e;
      SR_HIP(hipEventCreate(&e));
      p.push_back(e);
    }
    return used++;
  }
  // Waits for the launches of batch v (events of pool p) and accumulates
  // their durations.
  void drain(std::vector<Rec>& v, std::vector<hipEvent_t>& p) {
    if (v.empty()) return;
    SR_HIP(hipEventSynchronize(p[v.back().e1]));
    for (const Rec& r : v) {
      float ms = 0.f;
      SR_HIP(hipEventElapsedTime(&ms, p[r.e0], p[r.e1]));
      sec[r.cls] += ms * 1e-3;
      bytes[r.cls] += r.bytes;
      flops[r.cls] += r.flops;
      n[r.cls] += 1;
    }
    v.clear();
  }
  // After a profiled decode step: accumulate the batch before it (long
  // complete) and start a new batch, so the stream is not drained for the
  // profiler.
  void rotate() {
    drain(prev, pool[cur ^ 1]);
    prev.swap(recs);
    cur ^= 1;
    used = 0;
  }
  // Waits for every recorded launch and accumulates it.
  void flush() {
    drain(prev, pool[cur ^ 1]);
    drain(recs, pool[cur]);
    used = 0;
  }
};

struct Ctx {
  const Plan* pl;
  Layout* L;
  hipStream_t s;
  Profiler* prof;
};

template <typename F>
static void timed(const Ctx& c, int cls, double bytes, double flops, F&& launch) {
  Profiler* p = c.prof;
  if (!p || !p->active) {
    launch();
    return;
  }
  const size_t a = p->slot(), b = p->slot();
  LaunchTiming lt{p->pool[p->cur][a], p->pool[p->cur][b], false};
  launch_timing = &lt;
  try {
    launch();
  } catch (...) {
    launch_timing = nullptr;
    throw;
  }
  launch_timing = nullptr;
  if (lt.started) p->recs.push_back({cls, a, b, bytes, flops});
}

// Projection launch.  decode: a generator decode projection (classed by
// whether its rows make it MFMA- or weight-bound), else reward/prefill.
static int run_gemm(const Ctx& c, bool decode, int dtype, const void* A, int lda, const void* B, int ldb,
                    int M, int N, int K, int epi, void* out, int ldo, int out_bf16, bool paired = false,
                    int64_t pair_off = 0) {
  GemmArgs g;
  g.dtype = dtype; g.A = A; g.lda = lda; g.B = B; g.ldb = ldb; g.pair_off = pair_off;
  g.paired = paired; g.M = M; g.N = N; g.K = K; g.epi = epi; g.out = out; g.ldo = ldo;
  g.out_bf16 = out_bf16;
  const double es = dtype == SR_BF16 ? 2.0 : 4.0;
  const double nw = paired ? 2.0 * N : (double)N;
  double ob = epi == EPI_RESID ? 8.0 : (epi == EPI_PARTIAL ? 4.0 : (paired || out_bf16 ? es : 4.0));
  const double bytes = es * ((double)M * K + nw * K) + ob * (double)M * N;
  const double flops = 2.0 * M * nw * K;
  const int cls = decode ? (M >= 312 ? SR_K_GEN_GEMM_MFMA : SR_K_GEN_GEMM_HBM) : SR_K_RM_GEMM;
  int splits = 1;
  timed(c, cls, bytes, flops, [&] { splits = gemm(g, c.L->gpart, c.pl->gpart, c.s); });
  return splits;
}

static void run_other(const Ctx& c, double bytes, std::function<void()> f) {
  timed(c, SR_K_OTHER, bytes, 0.0, f);
}

// Feed-forward half of a layer: h += W2 (silu(W1 f) * (W3 f)), f = RMSNorm(h).
static void ffn_block(const Ctx& c, bool decode, const Model& M, int l, float* h, void* xn, void* u,
                      int rows) {
  const Dims& m = M.m;
  const int bf = m.dtype == SR_BF16;
  run_other(c, (double)rows * m.d * (4 + m.es),
            [&] { rmsnorm(m.dtype, h, m.d, M.ffn_norm(l), m.d, m.eps, rows, xn, m.d, c.s); });
  run_gemm(c, decode, m.dtype, xn, m.d, M.w13(l), m.d, rows, m.ff, m.d, EPI_STORE, u, m.ff, bf, true,
           (int64_t)m.ff * m.d);
  run_gemm(c, decode, m.dtype, u, m.ff, M.w2(l), m.ff, rows, m.d, m.ff, EPI_RESID, h, m.d, 0);
}

// Prefill of `rows` sequences of `lr` tokens (device tokens [rows][lr]) at
// positions pos0 + t, attending the shared prefix `pre` (P tokens, may be 0)
// and causally their own tokens.  K/V of layer l are written through
// kv_out(l) as [rows][hkv][cap][hd] at index t0 + t of each row, after t0
// cached tokens of that row which the attention reads too.  Leaves the final
// hidden states in L.ch.
template <typename KvOut>
static void prefill(const Ctx& c, const Model& M, const float2* rope, const int32_t* tokens, int rows,
                    int lr, int pos0, const void* pre, int P, KvOut kv_out, int cap, int t0) {
  const Dims& m = M.m;
  Layout& L = *c.L;
  const int T = rows * lr;
  run_other(c, (double)T * m.d * (4 + m.es), [&] { embed(m.dtype, M.w->embed, m.d, tokens, T, L.ch, c.s); });
  for (int l = 0; l < m.nl; ++l) {
    void *kd, *vd;
    kv_out(l, &kd, &vd);
    run_other(c, (double)T * m.d * (4 + m.es),
              [&] { rmsnorm(m.dtype, L.ch, m.d, M.attn_norm(l), m.d, m.eps, T, L.cxn, m.d, c.s); });
    run_gemm(c, false, m.dtype, L.cxn, m.d, M.wqkv(l), m.d, T, m.qkv, m.d, EPI_STORE, L.cqkv, m.qkv, 0);
    run_other(c, (double)T * (m.qkv * 4.0 + m.hq * m.hd * 4.0 + 2.0 * m.hkv * m.hd * m.es), [&] {
      rope_scatter(m.dtype, L.cqkv, rows, lr, m.hq, m.hkv, m.hd, rope, pos0, L.cq, kd, vd, cap, t0, c.s);
    });
    PrefillAttnArgs a;
    a.dtype = m.dtype; a.hd = m.hd; a.hq = m.hq; a.hkv = m.hkv; a.rows = rows; a.lr = lr;
    a.q = L.cq;
    const size_t lay = (size_t)2 * m.hkv * P * m.hd * m.es;
    a.kpre = pre ? (const char*)pre + l * lay : nullptr;
    a.vpre = pre ? (const char*)pre + l * lay + lay / 2 : nullptr;
    a.P = pre ? P : 0;
    a.kown = kd; a.vown = vd; a.cap = cap; a.t0 = t0; a.out = L.co;
    const double Pp = a.P;
    const double abytes = 2.0 * m.hkv * m.hd * m.es * (Pp + (double)rows * (t0 + lr)) +
                          (double)T * m.hq * m.hd * (4 + m.es);
    const double aflops = 4.0 * m.hq * m.hd * rows * ((Pp + t0) * lr + 0.5 * lr * (lr + 1.0));
    timed(c, SR_K_PREFILL_ATTN, abytes, aflops, [&] { prefill_attn(a, c.s); });
    run_gemm(c, false, m.dtype, L.co, m.hq * m.hd, M.wo(l), m.hq * m.hd, T, m.d, m.hq * m.hd, EPI_RESID,
             L.ch, m.d, 0);
    ffn_block(c, false, M, l, L.ch, L.cxn, L.cu, T);
  }
}

// Prompt prefill of one model into its prefix buffer [nl][2][hkv][P][hd].
static void prompt_prefill(const Ctx& c, const Model& M, const float2* rope, void* pre) {
  const Dims& m = M.m;
  const int P = c.pl->P;
  const size_t lay = (size_t)2 * m.hkv * P * m.hd * m.es;
  prefill(c, M, rope, c.L->ctok, 1, P, 0, nullptr, 0, [&](int l, void** k, void** v) {
    *k = (char*)pre + l * lay;
    *v = (char*)pre + l * lay + lay / 2;
  }, P, 0);
}

// Reward scores of `rows` rows (cand/len arrays of a state) at max length lr.
// Without a cache (pool == nullptr) the whole responses are run through the
// reward model.  With one, row r's K/V of response positions 0..t0-1 are in
// the pool ([nl][2] blocks of pool_block elements, rows of cap positions),
// every row has t0 < len <= lr, and only positions t0..lr-1 are run, their
// K/V appended to the pool.
static void reward_rows(const Ctx& c, const Model& R, const int32_t* cand, const int32_t* len, int rows,
                        int lr, float* score, int t0 = 0, void* pool = nullptr, int64_t pool_block = 0,
                        int cap = 0) {
  const Plan& pl = *c.pl;
  Layout& L = *c.L;
  const Dims& m = R.m;
  SR_REQUIRE(pool || t0 == 0, SR_ERR_INTERNAL, "reward prefix without a cache");
  const int nl = lr - t0;
  const int per = std::max(1, pl.Tc / nl);
  for (int r0 = 0; r0 < rows; r0 += per) {
    const int rc = std::min(per, rows - r0);
    run_other(c, (double)rc * nl * 8,
              [&] { gather_tokens(L.store, pl.Lmax, cand + r0, len + r0, rc, t0, nl, L.ctok, c.s); });
    const size_t row0 = (size_t)r0 * m.hkv * cap * m.hd;
    prefill(c, R, L.rope_r, L.ctok, rc, nl, pl.P + t0, L.rpre, pl.P, [&](int l, void** k, void** v) {
      if (pool) {
        *k = (char*)pool + ((size_t)(2 * l) * pool_block + row0) * m.es;
        *v = (char*)pool + ((size_t)(2 * l + 1) * pool_block + row0) * m.es;
      } else {
        *k = L.ck;
        *v = L.cv;
      }
    }, pool ? cap : nl, t0);
    run_other(c, (double)rc * m.d * 4, [&] {
      score_head(m.dtype, L.ch, m.d, nl, t0, len + r0, rc, R.w->final_norm, R.w->head, m.eps, score + r0, c.s);
    });
  }
}

// One decode step for `rows` rows: feed st.tok (response token t = step-1 at
// position P + step - 1) through the generator, append its K/V to the tail
// pool at index step-1 and leave the logits of the next token in L.logits.
static void decode_step(const Ctx& c, const Model& G, const State& st, int rows, int step, void* pool,
                        int64_t pool_block, int cap) {
  const Dims& m = G.m;
  Layout& L = *c.L;
  const Plan& pl = *c.pl;
  const int bf = m.dtype == SR_BF16;
  run_other(c, (double)rows * m.d * (4 + m.es), [&] {
    embed_norm(m.dtype, G.w->embed, m.d, st.tok, rows, G.attn_norm(0), m.eps, L.h, L.xn, c.s);
  });
  const size_t pre_lay = (size_t)2 * m.hkv * pl.P * m.hd * m.es;
  for (int l = 0; l < m.nl; ++l) {
    char* kpool = (char*)pool + (size_t)(2 * l) * pool_block * m.es;
    char* vpool = (char*)pool + (size_t)(2 * l + 1) * pool_block * m.es;
    int sp = run_gemm(c, true, m.dtype, L.xn, m.d, G.wqkv(l), m.d, rows, m.qkv, m.d, EPI_PARTIAL, nullptr, 0, 0);
    DecodeAttnArgs a;
    a.dtype = m.dtype; a.hd = m.hd; a.hq = m.hq; a.hkv = m.hkv; a.rows = rows; a.q = L.q;
    a.kpre = (const char*)L.gpre + l * pre_lay;
    a.vpre = (const char*)L.gpre + l * pre_lay + pre_lay / 2;
    a.P = pl.P; a.ktail = kpool; a.vtail = vpool; a.cap = cap; a.lt = step; a.out = L.o;
    a.part = L.apart; a.part_cap = pl.apart;
    // the QKV partials are summed, rotated and scattered inside the
    // attention where its streaming form runs, else by their own kernel
    a.qpart = L.gpart; a.qsplits = sp; a.qkv_dim = m.qkv;
    a.rope = L.rope_g + (size_t)(pl.P + step - 1) * (m.hd / 2); a.qout = L.q;
    const double qbytes = (double)rows * (m.qkv * 4.0 * sp + m.hq * m.hd * 4.0 + 2.0 * m.hkv * m.hd * m.es);
    if (!decode_attn_fuses_qkv(a)) {
      a.qpart = nullptr;
      run_other(c, qbytes, [&] {
        qkv_finalize(m.dtype, L.gpart, sp, rows, m.hq, m.hkv, m.hd, L.rope_g, pl.P + step - 1, L.q, kpool, vpool,
                     cap, step - 1, c.s);
      });
    }
    // the method's own attention bytes: the keys and values (the prefix
    // once), the query and the output; the QKV split partials the fused
    // finalize reads are the projection's traffic, not counted here
    const double abytes = 2.0 * m.hkv * m.hd * m.es * ((double)pl.P + (double)rows * step) +
                          (double)rows * m.hq * m.hd * (4 + m.es);
    const double aflops = 4.0 * rows * m.hq * m.hd * ((double)pl.P + step);
    timed(c, SR_K_DECODE_ATTN, abytes, aflops, [&] { decode_attn(a, c.s); });
    sp = run_gemm(c, true, m.dtype, L.o, m.hq * m.hd, G.wo(l), m.hq * m.hd, rows, m.d, m.hq * m.hd, EPI_PARTIAL,
                  nullptr, 0, 0);
    run_other(c, (double)rows * m.d * (4.0 * sp + 8 + m.es), [&] {
      add_norm(m.dtype, L.gpart, sp, rows, m.d, L.h, G.ffn_norm(l), m.eps, L.xn, c.s);
    });
    run_gemm(c, true, m.dtype, L.xn, m.d, G.w13(l), m.d, rows, m.ff, m.d, EPI_STORE, L.u, m.ff, bf, true,
             (int64_t)m.ff * m.d);
    sp = run_gemm(c, true, m.dtype, L.u, m.ff, G.w2(l), m.ff, rows, m.d, m.ff, EPI_PARTIAL, nullptr, 0, 0);
    const void* gnext = l + 1 < m.nl ? G.attn_norm(l + 1) : G.w->final_norm;
    run_other(c, (double)rows * m.d * (4.0 * sp + 8 + m.es), [&] {
      add_norm(m.dtype, L.gpart, sp, rows, m.d, L.h, gnext, m.eps, L.xn, c.s);
    });
  }
  run_gemm(c, true, m.dtype, L.xn, m.d, G.w->head, m.d, rows, m.V, m.d, EPI_STORE, L.logits, m.V, 0);
}

// Logits of the last prompt token into logits row 0 (after prompt_prefill,
// whose hidden states are still in L.ch).
static void prompt_logits(const Ctx& c, const Model& G) {
  const Dims& m = G.m;
  Layout& L = *c.L;
  rmsnorm(m.dtype, L.ch + (size_t)(c.pl->P - 1) * m.d, m.d, G.w->final_norm, m.d, m.eps, 1, L.xn, m.d,
          c.s);
  run_gemm(c, false, m.dtype, L.xn, m.d, G.w->head, m.d, 1, m.V, m.d, EPI_STORE, L.logits, m.V, 0);
}

__global__ void init_state_kernel(int n, int32_t* cand, int32_t* len, int32_t* done, int32_t* cand_len,
                                  int32_t* i_count, float* lp_sum) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    cand[i] = i;
    len[i] = 0;
    done[i] = 0;
    cand_len[i] = 0;
    lp_sum[i] = 0.f;
  }
  if (i == 0) *i_count = 0;
}

__global__ void compose_kernel(const int32_t* outer, const int32_t* inner, const int32_t* count,
                               int32_t* out) {
  int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < *count) out[j] = outer[inner[j]];
}

__global__ void lens_kernel(const int32_t* len, int n, int32_t* cand_len, const int32_t* cand) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) cand_len[cand[i]] = len[i];
}

__global__ void column_kernel(const int32_t* tokens, int ld, int col, int rows, int32_t* out) {
  int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < rows) out[r] = tokens[(int64_t)r * ld + col];
}

struct Timer {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipStream_t s;
  explicit Timer(hipStream_t st) : s(st) {
    SR_HIP(hipEventCreate(&e0));
    SR_HIP(hipEventCreate(&e1));
  }
  ~Timer() {
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
  }
  void start() { SR_HIP(hipEventRecord(e0, s)); }
  double stop() {  // blocking
    SR_HIP(hipEventRecord(e1, s));
    SR_HIP(hipEventSynchronize(e1));
    float ms = 0.f;
    SR_HIP(hipEventElapsedTime(&ms, e0, e1));
    return ms * 1e-3;
  }
};

static void check_prompt(const int32_t* prompt, int P, int V) {
  SR_REQUIRE(P >= 1, SR_ERR_INVALID_ARG, "prompt_len must be >= 1");
  SR_REQUIRE(prompt != nullptr, SR_ERR_INVALID_ARG, "prompt is NULL");
  for (int i = 0; i < P; ++i)
    SR_REQUIRE(prompt[i] >= 0 && prompt[i] < V, SR_ERR_INVALID_ARG, "prompt token out of range");
}

static Layout setup(const sr_model* gen, const sr_model* rm, int P, const sr_params* p, void* ws,
                    size_t ws_bytes, Plan* pl_out, Dims* gd, Dims* rd) {
  *gd = dims_of(gen->cfg);
  *rd = dims_of(rm->cfg);
  *pl_out = make_plan(*gd, *rd, P, p);
  size_t need = 0;
  carve(nullptr, *gd, *rd, *pl_out, &need);
  SR_REQUIRE(ws != nullptr, SR_ERR_INVALID_ARG, "workspace is NULL");
  SR_REQUIRE(((uintptr_t)ws & 255) == 0, SR_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  SR_REQUIRE(ws_bytes >= need, SR_ERR_WORKSPACE_TOO_SMALL,
             "workspace too small: need " + std::to_string(need) + " bytes");
  size_t tot;
  return carve(ws, *gd, *rd, *pl_out, &tot);
}

static void copy_h2d(void* dst, const void* src, size_t n, hipStream_t s) {
  SR_HIP(hipMemcpyAsync(dst, src, n, hipMemcpyHostToDevice, s));
}
static void copy_d2h(void* dst, const void* src, size_t n, hipStream_t s) {
  SR_HIP(hipMemcpyAsync(dst, src, n, hipMemcpyDeviceToHost, s));
  SR_HIP(hipStreamSynchronize(s));
}

static void generate(const sr_model* gen, const sr_model* rm, const int32_t* prompt, int P,
                     const sr_params* p, void* ws, size_t ws_bytes, hipStream_t s, int32_t* out_tokens,
                     sr_result* out, sr_trace* tr) {
  SR_REQUIRE(out_tokens && out, SR_ERR_INVALID_ARG, "out_tokens and out must not be NULL");
  Plan pl;
  Dims gd, rd;
  Layout L = setup(gen, rm, P, p, ws, ws_bytes, &pl, &gd, &rd);
  Profiler prof;
  prof.s = s;
  const int every = p->profile_every;
  Ctx c{&pl, &L, s, every > 0 ? &prof : nullptr};
  const bool lp_mode = p->reward_kind == SR_REWARD_LOGPROB;
  Model G{gd, &gen->w}, R{rd, lp_mode ? nullptr : &rm->w};
  const int N = pl.N, Lmax = pl.Lmax;
  std::memset(out, 0, sizeof(*out));
  // partial rewards of the rows of a round: the reward model, or the mean
  // log-probability accumulated while sampling (section 5.3).  With the
  // reward model's cache, the survivors of the last cut bring their K/V of
  // the first t0 response tokens.
  auto score_rows = [&](const State& st, int b, int D, int cur, int cap, int t0) {
    if (lp_mode) {
      logprob_scores(L.lp_sum, st.cand, st.len, b, L.score, s);
    } else if (pl.rkv) {
      reward_rows(c, R, st.cand, st.len, b, D, L.score, t0, L.rpool[cur], pl.S[cur] * rd.hkv * rd.hd, cap);
    } else {
      reward_rows(c, R, st.cand, st.len, b, D, L.score);
    }
  };
  Timer tall(s), tph(s);
  tall.start();

  // prompt prefill of both models; logits of the first response token
  prof.active = every > 0;
  tph.start();
  rope_table(L.rope_g, P + Lmax + 1, gd.hd, gd.theta, s);
  copy_h2d(L.ctok, prompt, sizeof(int32_t) * P, s);
  if (!lp_mode) {
    rope_table(L.rope_r, P + Lmax + 1, rd.hd, rd.theta, s);
    prompt_prefill(c, R, L.rope_r, L.rpre);
  }
  prompt_prefill(c, G, L.rope_g, L.gpre);
  prompt_logits(c, G);
  SR_LAUNCH(init_state_kernel, dim3((N + 255) / 256), dim3(256), 0, s, N, L.st[0].cand,
                     L.st[0].len, L.st[0].done, L.cand_len, L.i_count, L.lp_sum);
  SR_CHECK_LAUNCH();
  out->sec_prefill = tph.stop();
  prof.flush();

  int cur = 0;  // state/pool index of the running round
  int b = N, r = 0, step = 0;
  int D = decision(pl, b, r);
  int cap = D;
  int t0 = 0;  // response tokens whose reward-model K/V the cache holds
  int64_t generated = 0;
  std::vector<int32_t> h_done, h_i32(N);
  std::vector<float> h_f32(N);
  // watched candidates (trace): their row in the current round, -1 if absent
  const bool watching = tr && tr->n_watch > 0 && tr->watch_cand && tr->watch_logits;
  std::vector<int> watch_row(watching ? tr->n_watch : 0, -1);
  // with an end-of-sequence token, the done flags are read back every
  // kDoneCheck steps so that a round whose rows have all finished ends there
  constexpr int kDoneCheck = 16;
  while (true) {
    // ---- phase 1: generate up to the decision token
    tph.start();
    SR_REQUIRE((int64_t)b * cap <= pl.S[cur], SR_ERR_INTERNAL, "KV pool capacity exceeded");
    if (watching) {
      std::vector<int32_t> rows_cand(b);
      copy_d2h(rows_cand.data(), L.st[cur].cand, sizeof(int32_t) * b, s);
      for (int w = 0; w < tr->n_watch; ++w) {
        watch_row[w] = -1;
        for (int i = 0; i < b; ++i)
          if (rows_cand[i] == tr->watch_cand[w]) watch_row[w] = i;
      }
    }
    for (; step < D; ++step) {
      prof.active = every > 0 && step % every == 0;
      const State& st = L.st[cur];
      if (step > 0) decode_step(c, G, st, b, step, L.pool[cur], pl.S[cur] * gd.hkv * gd.hd, cap);
      for (int w = 0; w < (int)watch_row.size(); ++w)
        if (watch_row[w] >= 0)
          copy_d2h(tr->watch_logits + ((size_t)w * Lmax + step) * gd.V,
                   L.logits + (step == 0 ? 0 : (size_t)watch_row[w] * gd.V), sizeof(float) * gd.V, s);
      SampleArgs sa;
      sa.logits = L.logits; sa.row_stride = step == 0 ? 0 : gd.V; sa.rows = b; sa.vocab = gd.V;
      sa.cand = st.cand; sa.step = step; sa.temperature = p->temperature; sa.seed = p->seed;
      sa.next_tok = st.tok; sa.done = st.done; sa.len = st.len; sa.store = L.store;
      sa.store_ld = Lmax; sa.eos_id = p->eos_id;
      timed(c, SR_K_SAMPLE, (double)b * gd.V * 4, 0.0, [&] { sample(sa, s); });
      if (lp_mode)
        timed(c, SR_K_SAMPLE, (double)b * gd.V * 4, 0.0, [&] {
          logprob_accumulate(L.logits, sa.row_stride, b, gd.V, st.cand, st.tok, st.len, step, L.lp_sum, s);
        });
      if (prof.active) prof.rotate();
      if (p->eos_id >= 0 && (step + 1) % kDoneCheck == 0 && step + 1 < D) {
        h_done.resize(b);
        copy_d2h(h_done.data(), st.done, sizeof(int32_t) * b, s);
        if (std::all_of(h_done.begin(), h_done.end(), [](int32_t v) { return v != 0; })) {
          ++step;
          break;
        }
      }
    }
    prof.active = every > 0;
    out->sec_decode += tph.stop();
    // unfinished rows?
    h_done.resize(b);
    copy_d2h(h_done.data(), L.st[cur].done, sizeof(int32_t) * b, s);
    int unfinished = 0;
    for (int i = 0; i < b; ++i) unfinished += h_done[i] == 0;
    State& st = L.st[cur];
    SR_LAUNCH(lens_kernel, dim3((b + 255) / 256), dim3(256), 0, s, st.len, b, L.cand_len,
                       st.cand);
    SR_CHECK_LAUNCH();
    if (D == Lmax || unfinished == 0) {
      // every candidate of this round is complete (no row is longer than
      // `step`): score all, all join I
      tph.start();
      score_rows(st, b, step, cur, cap, t0);
      out->sec_reward += tph.stop();
      CutArgs ca;
      std::memset(&ca, 0, sizeof(ca));
      ca.score = L.score; ca.cand = st.cand; ca.len = st.len; ca.next_tok = st.tok; ca.b = b;
      ca.keep = b;
      // mark all rows as completed so that they all join I
      SR_HIP(hipMemsetAsync(L.src_tmp, 0xFF, sizeof(int32_t) * b, s));
      ca.done = L.src_tmp; ca.accept = L.accept;
      ca.i_cand = L.i_cand; ca.i_len = L.i_len; ca.i_count = L.i_count; ca.i_score = L.i_score;
      ca.src_row = L.src_row; ca.cand_out = L.st[2].cand; ca.len_out = L.st[2].len;
      ca.tok_out = L.st[2].tok; ca.count = L.count;
      timed(c, SR_K_CUT, (double)b * 24, 0.0, [&] { cut(ca, s); });
      break;
    }
    // ---- phase 2: partial rewards and the cut
    const int K = keep_of(b, pl.appm);
    SR_REQUIRE(K < b, SR_ERR_INTERNAL, "decision point without a possible rejection");
    tph.start();
    score_rows(st, b, D, cur, cap, t0);
    out->sec_reward += tph.stop();
    tph.start();
    const int nxt = 1 - cur;
    State& ns = L.st[nxt];
    CutArgs ca;
    ca.score = L.score; ca.cand = st.cand; ca.len = st.len; ca.done = st.done; ca.next_tok = st.tok;
    ca.b = b; ca.keep = K; ca.accept = L.accept;
    ca.i_cand = L.i_cand; ca.i_len = L.i_len; ca.i_count = L.i_count; ca.i_score = L.i_score;
    ca.src_row = L.src_row; ca.cand_out = ns.cand; ca.len_out = ns.len; ca.tok_out = ns.tok;
    ca.count = L.count;
    timed(c, SR_K_CUT, (double)b * 24, 0.0, [&] { cut(ca, s); });
    // scores of the survivors, for a further cut at the same length
    int cnt = 0;
    copy_d2h(&cnt, L.count, sizeof(int32_t), s);
    if (tr && r < tr->max_rounds_cap) {
      if (tr->round_L) tr->round_L[r] = step;
      if (tr->round_b) tr->round_b[r] = b;
      if (tr->round_keep) tr->round_keep[r] = K;
      if (tr->round_cand) copy_d2h(tr->round_cand + (size_t)r * N, st.cand, sizeof(int32_t) * b, s);
      if (tr->round_scores) copy_d2h(tr->round_scores + (size_t)r * N, L.score, sizeof(float) * b, s);
      if (tr->round_accept) copy_d2h(tr->round_accept + (size_t)r * N, L.accept, sizeof(int32_t) * b, s);
    }
    ++r;
    // survivors' scores (host copy) for cascaded cuts
    std::vector<float> sc_all(b);
    std::vector<int32_t> src(cnt);
    if (cnt > 0) {
      copy_d2h(sc_all.data(), L.score, sizeof(float) * b, s);
      copy_d2h(src.data(), L.src_row, sizeof(int32_t) * cnt, s);
    }
    // ---- phase 3: next round's batch (cut again while memory is still full)
    int nD = Lmax;
    while (cnt > 0) {
      if (keep_of(cnt, pl.appm) == cnt || (pl.max_rounds > 0 && r >= pl.max_rounds)) {
        nD = Lmax;
        break;
      }
      const int Dn = (int)std::min<int64_t>(Lmax, pl.B / cnt);
      if (Dn > step) {
        nD = Dn;
        break;
      }
      const int K2 = keep_of(cnt, pl.appm);
      // scores of the survivors in their packed order
      for (int j = 0; j < cnt; ++j) h_f32[j] = sc_all[src[j]];
      copy_h2d(L.score2, h_f32.data(), sizeof(float) * cnt, s);
      CutArgs c2;
      c2.score = L.score2; c2.cand = ns.cand; c2.len = ns.len; c2.next_tok = ns.tok;
      SR_HIP(hipMemsetAsync(L.src_tmp, 0, sizeof(int32_t) * cnt, s));
      c2.done = L.src_tmp; c2.b = cnt; c2.keep = K2; c2.accept = L.accept;
      c2.i_cand = L.i_cand; c2.i_len = L.i_len; c2.i_count = L.i_count; c2.i_score = L.i_score;
      c2.src_row = L.src_row2; c2.cand_out = L.st[2].cand; c2.len_out = L.st[2].len;
      c2.tok_out = L.st[2].tok; c2.count = L.count2;
      timed(c, SR_K_CUT, (double)cnt * 24, 0.0, [&] { cut(c2, s); });
      int cnt2 = 0;
      copy_d2h(&cnt2, L.count2, sizeof(int32_t), s);
      if (tr && r < tr->max_rounds_cap) {
        if (tr->round_L) tr->round_L[r] = step;
        if (tr->round_b) tr->round_b[r] = cnt;
        if (tr->round_keep) tr->round_keep[r] = K2;
        if (tr->round_cand) copy_d2h(tr->round_cand + (size_t)r * N, ns.cand, sizeof(int32_t) * cnt, s);
        if (tr->round_scores) std::memcpy(tr->round_scores + (size_t)r * N, h_f32.data(), sizeof(float) * cnt);
        if (tr->round_accept) copy_d2h(tr->round_accept + (size_t)r * N, L.accept, sizeof(int32_t) * cnt, s);
      }
      ++r;
      SR_LAUNCH(compose_kernel, dim3((cnt2 + 255) / 256 + 1), dim3(256), 0, s, L.src_row,
                         L.src_row2, L.count2, L.src_tmp);
      SR_CHECK_LAUNCH();
      SR_HIP(hipMemcpyAsync(L.src_row, L.src_tmp, sizeof(int32_t) * std::max(cnt2, 1),
                            hipMemcpyDeviceToDevice, s));
      SR_HIP(hipMemcpyAsync(ns.cand, L.st[2].cand, sizeof(int32_t) * std::max(cnt2, 1),
                            hipMemcpyDeviceToDevice, s));
      SR_HIP(hipMemcpyAsync(ns.len, L.st[2].len, sizeof(int32_t) * std::max(cnt2, 1),
                            hipMemcpyDeviceToDevice, s));
      SR_HIP(hipMemcpyAsync(ns.tok, L.st[2].tok, sizeof(int32_t) * std::max(cnt2, 1),
                            hipMemcpyDeviceToDevice, s));
      SR_HIP(hipMemcpyAsync(L.count, L.count2, sizeof(int32_t), hipMemcpyDeviceToDevice, s));
      std::vector<int32_t> src2(cnt2);
      if (cnt2 > 0) copy_d2h(src2.data(), L.src_row, sizeof(int32_t) * cnt2, s);
      src.swap(src2);
      cnt = cnt2;
    }
    if (cnt == 0) {
      out->sec_cut += tph.stop();
      break;
    }
    // pack the survivors' tails (tokens 0..step-2 hold K/V) into the other pool
    SR_REQUIRE((int64_t)cnt * nD <= pl.S[nxt], SR_ERR_INTERNAL, "KV pool capacity exceeded");
    CompactArgs ka;
    std::memset(&ka, 0, sizeof(ka));
    ka.src = L.pool[cur]; ka.src_block = pl.S[cur] * gd.hkv * gd.hd;
    ka.dst = L.pool[nxt]; ka.dst_block = pl.S[nxt] * gd.hkv * gd.hd;
    ka.src_row = L.src_row; ka.count = L.count; ka.b = b; ka.max_rows = cnt;
    ka.n_layers = gd.nl; ka.hkv = gd.hkv; ka.hd = gd.hd; ka.elem_bytes = gd.es;
    ka.cap_src = cap; ka.cap_dst = nD; ka.len = step - 1;
    timed(c, SR_K_CUT, 4.0 * gd.nl * cnt * (double)(step - 1) * gd.hkv * gd.hd * gd.es, 0.0,
          [&] { compact(ka, s); });
    if (pl.rkv) {
      // the reward model's K/V of all `step` response tokens moves the same way
      CompactArgs kr = ka;
      kr.src = L.rpool[cur]; kr.src_block = pl.S[cur] * rd.hkv * rd.hd;
      kr.dst = L.rpool[nxt]; kr.dst_block = pl.S[nxt] * rd.hkv * rd.hd;
      kr.n_layers = rd.nl; kr.hkv = rd.hkv; kr.hd = rd.hd; kr.elem_bytes = rd.es; kr.len = step;
      timed(c, SR_K_CUT, 4.0 * rd.nl * cnt * (double)step * rd.hkv * rd.hd * rd.es, 0.0,
            [&] { compact(kr, s); });
    }
    SR_HIP(hipMemsetAsync(ns.done, 0, sizeof(int32_t) * cnt, s));
    out->sec_cut += tph.stop();
    prof.flush();
    cur = nxt;
    b = cnt;
    t0 = step;
    D = nD;
    cap = nD;
  }
  // ---- answer: best member of I (eq. output)
  int n_i = 0;
  copy_d2h(&n_i, L.i_count, sizeof(int32_t), s);
  SR_REQUIRE(n_i >= 1 && n_i <= N, SR_ERR_INTERNAL, "set I is empty");
  timed(c, SR_K_CUT, (double)n_i * 8, 0.0, [&] { argmax_best(L.i_score, L.i_cand, L.i_count, N, L.best, s); });
  prof.flush();
  for (int k = 0; k < SR_K_NCLASS; ++k) {
    out->kernel_sec[k] = prof.sec[k];
    out->kernel_launches[k] = prof.n[k];
    out->kernel_bytes[k] = prof.bytes[k];
    out->kernel_flops[k] = prof.flops[k];
  }
  int best = -1;
  copy_d2h(&best, L.best, sizeof(int32_t), s);
  SR_REQUIRE(best >= 0 && best < n_i, SR_ERR_INTERNAL, "arg max failed");
  int bc = 0, bl = 0;
  float bs = 0.f;
  copy_d2h(&bc, L.i_cand + best, sizeof(int32_t), s);
  copy_d2h(&bl, L.i_len + best, sizeof(int32_t), s);
  copy_d2h(&bs, L.i_score + best, sizeof(float), s);
  SR_REQUIRE(bl >= 1 && bl <= Lmax, SR_ERR_INTERNAL, "bad response length");
  copy_d2h(out_tokens, L.store + (size_t)bc * Lmax, sizeof(int32_t) * bl, s);
  std::vector<int32_t> lens(N);
  copy_d2h(lens.data(), L.cand_len, sizeof(int32_t) * N, s);
  for (int i = 0; i < N; ++i) generated += lens[i];
  out->sec_total = tall.stop();
  out->best_index = bc;
  out->best_score = bs;
  out->n_tokens = bl;
  out->rounds = r;
  out->generated_tokens = generated;
  if (tr) {
    if (tr->all_len) std::memcpy(tr->all_len, lens.data(), sizeof(int32_t) * N);
    if (tr->all_tokens) copy_d2h(tr->all_tokens, L.store, sizeof(int32_t) * (size_t)N * Lmax, s);
    if (tr->final_scores) {
      std::vector<int32_t> ic(n_i);
      std::vector<float> is(n_i);
      copy_d2h(ic.data(), L.i_cand, sizeof(int32_t) * n_i, s);
      copy_d2h(is.data(), L.i_score, sizeof(float) * n_i, s);
      for (int i = 0; i < N; ++i) tr->final_scores[i] = NAN;
      for (int i = 0; i < n_i; ++i) tr->final_scores[ic[i]] = is[i];
    }
  }
}

static void teacher_forced(const sr_model* gen, const sr_model* rm, const int32_t* prompt, int P,
                           const sr_params* p, const int32_t* tokens, int rows, int len, float* logits_out,
                           void* ws, size_t ws_bytes, hipStream_t s) {
  Plan pl;
  Dims gd, rd;
  Layout L = setup(gen, rm, P, p, ws, ws_bytes, &pl, &gd, &rd);
  SR_REQUIRE(rows >= 1 && rows <= pl.N && len >= 1 && len <= pl.Lmax, SR_ERR_INVALID_ARG,
             "rows/len exceed the workspace's n/max_new_tokens");
  SR_REQUIRE(tokens && logits_out, SR_ERR_INVALID_ARG, "NULL buffer");
  SR_REQUIRE((int64_t)rows * len <= pl.S[0], SR_ERR_INVALID_ARG, "rows * len exceeds the KV pool");
  {
    std::vector<int32_t> h((size_t)rows * len);
    copy_d2h(h.data(), tokens, h.size() * sizeof(int32_t), s);
    for (int32_t t : h) SR_REQUIRE(t >= 0 && t < gd.V, SR_ERR_INVALID_ARG, "token out of range");
  }
  Ctx c{&pl, &L, s, nullptr};
  Model G{gd, &gen->w};
  rope_table(L.rope_g, P + pl.Lmax + 1, gd.hd, gd.theta, s);
  copy_h2d(L.ctok, prompt, sizeof(int32_t) * P, s);
  prompt_prefill(c, G, L.rope_g, L.gpre);
  prompt_logits(c, G);
  const size_t V = gd.V;
  for (int r = 0; r < rows; ++r)
    SR_HIP(hipMemcpyAsync(logits_out + (size_t)r * len * V, L.logits, V * sizeof(float),
                          hipMemcpyDeviceToDevice, s));
  State st = L.st[0];
  for (int t = 1; t < len; ++t) {
    SR_LAUNCH(column_kernel, dim3((rows + 255) / 256), dim3(256), 0, s, tokens, len, t - 1, rows,
                       st.tok);
    SR_CHECK_LAUNCH();
    decode_step(c, G, st, rows, t, L.pool[0], pl.S[0] * gd.hkv * gd.hd, len);
    SR_HIP(hipMemcpy2DAsync(logits_out + (size_t)t * V, (size_t)len * V * sizeof(float), L.logits,
                            V * sizeof(float), V * sizeof(float), rows, hipMemcpyDeviceToDevice, s));
  }
  SR_HIP(hipStreamSynchronize(s));
}

static void reward_entry(const sr_model* gen, const sr_model* rm, const int32_t* prompt, int P,
                         const sr_params* p, const int32_t* tokens, const int32_t* lens, int rows,
                         int max_len, float* scores, void* ws, size_t ws_bytes, hipStream_t s) {
  Plan pl;
  Dims gd, rd;
  Layout L = setup(gen, rm, P, p, ws, ws_bytes, &pl, &gd, &rd);
  SR_REQUIRE(rows >= 1 && rows <= pl.N && max_len >= 1 && max_len <= pl.Lmax, SR_ERR_INVALID_ARG,
             "rows/max_len exceed the workspace's n/max_new_tokens");
  SR_REQUIRE(tokens && lens && scores, SR_ERR_INVALID_ARG, "NULL buffer");
  {
    std::vector<int32_t> hl(rows), ht((size_t)rows * max_len);
    copy_d2h(hl.data(), lens, hl.size() * sizeof(int32_t), s);
    copy_d2h(ht.data(), tokens, ht.size() * sizeof(int32_t), s);
    for (int r = 0; r < rows; ++r) {
      SR_REQUIRE(hl[r] >= 1 && hl[r] <= max_len, SR_ERR_INVALID_ARG, "lens[r] must be in [1, max_len]");
      for (int t = 0; t < hl[r]; ++t)
        SR_REQUIRE(ht[(size_t)r * max_len + t] >= 0 && ht[(size_t)r * max_len + t] < rd.V,
                   SR_ERR_INVALID_ARG, "token out of range");
    }
  }
  Ctx c{&pl, &L, s, nullptr};
  Model R{rd, &rm->w};
  rope_table(L.rope_r, P + pl.Lmax + 1, rd.hd, rd.theta, s);
  copy_h2d(L.ctok, prompt, sizeof(int32_t) * P, s);
  prompt_prefill(c, R, L.rope_r, L.rpre);
  // the responses become the token store; rows are their own candidates
  SR_HIP(hipMemcpy2DAsync(L.store, (size_t)pl.Lmax * 4, tokens, (size_t)max_len * 4, (size_t)max_len * 4,
                          rows, hipMemcpyDeviceToDevice, s));
  SR_LAUNCH(init_state_kernel, dim3((rows + 255) / 256), dim3(256), 0, s, rows, L.st[0].cand,
                     L.st[0].len, L.st[0].done, L.cand_len, L.i_count, L.lp_sum);
  SR_CHECK_LAUNCH();
  reward_rows(c, R, L.st[0].cand, lens, rows, max_len, scores);
  SR_HIP(hipStreamSynchronize(s));
}

template <typename F>
static sr_status guard(F&& f) {
  try {
    f();
    t_err.clear();
    return SR_OK;
  } catch (const Error& e) {
    t_err = e.msg;
    return (sr_status)e.status;
  } catch (const std::exception& e) {
    t_err = std::string("internal error: ") + e.what();
    return SR_ERR_INTERNAL;
  } catch (...) {
    t_err = "internal error";
    return SR_ERR_INTERNAL;
  }
}

void set_last_error(const char* msg) { t_err = msg; }

}  // namespace sr

using namespace sr;

extern "C" {

const char* sr_last_error(void) { return t_err.c_str(); }

int32_t sr_keep_count(int32_t b, double alpha) {
  if (b < 0 || !(alpha >= 0.0 && alpha < 1.0)) return -1;
  return keep_of(b, alpha_ppm(alpha));
}

sr_status sr_workspace_size(const sr_model* gen, const sr_model* rm, int32_t prompt_len,
                            const sr_params* p, size_t* bytes) {
  return guard([&] {
    sr_model stand_in;
    rm = reward_model_of(gen, rm, p, &stand_in);
    check_pair(gen, rm);
    check_params(p, gen);
    SR_REQUIRE(prompt_len >= 1, SR_ERR_INVALID_ARG, "prompt_len must be >= 1");
    SR_REQUIRE(bytes != nullptr, SR_ERR_INVALID_ARG, "bytes is NULL");
    Dims gd = dims_of(gen->cfg), rd = dims_of(rm->cfg);
    Plan pl = make_plan(gd, rd, prompt_len, p);
    size_t tot = 0;
    carve(nullptr, gd, rd, pl, &tot);
    *bytes = tot;
  });
}

sr_status sr_plan_for_memory(const sr_model* gen, const sr_model* rm, int32_t prompt_len, const sr_params* p,
                             size_t capacity_bytes, sr_params* out) {
  return guard([&] {
    SR_REQUIRE(p != nullptr && out != nullptr, SR_ERR_INVALID_ARG, "params is NULL");
    const bool pick_n = p->n == 0;
    sr_params q = *p;
    if (pick_n) q.n = 1;
    // the largest value of the free field whose workspace fits; the size
    // never decreases as n or tau grows, so a bisection finds it
    auto fits = [&](int v) {
      sr_params t = q;
      (pick_n ? t.n : t.tau) = v;
      size_t need = 0;
      const sr_status st = sr_workspace_size(gen, rm, prompt_len, &t, &need);
      SR_REQUIRE(st == SR_OK, st, t_err);
      return need <= capacity_bytes;
    };
    int lo = 1, hi = pick_n ? kMaxN : std::max(1, p->max_new_tokens);
    SR_REQUIRE(fits(lo), SR_ERR_WORKSPACE_TOO_SMALL,
               std::string("capacity below the workspace of ") + (pick_n ? "n = 1" : "tau = 1"));
    while (lo < hi) {
      const int mid = lo + (hi - lo + 1) / 2;
      if (fits(mid)) lo = mid;
      else hi = mid - 1;
    }
    (pick_n ? q.n : q.tau) = lo;
    *out = q;
  });
}

sr_status sr_generate(const sr_model* gen, const sr_model* rm, const int32_t* prompt, int32_t prompt_len,
                      const sr_params* p, void* workspace, size_t ws_bytes, void* stream,
                      int32_t* out_tokens, sr_result* out, sr_trace* trace) {
  return guard([&] {
    sr_model stand_in;
    rm = reward_model_of(gen, rm, p, &stand_in);
    check_pair(gen, rm);
    check_params(p, gen);
    check_prompt(prompt, prompt_len, gen->cfg.vocab);
    if (trace && trace->n_watch != 0) {
      SR_REQUIRE(trace->n_watch > 0 && trace->watch_cand && trace->watch_logits, SR_ERR_INVALID_ARG,
                 "trace: n_watch must be >= 0 with watch_cand and watch_logits set");
      for (int w = 0; w < trace->n_watch; ++w)
        SR_REQUIRE(trace->watch_cand[w] >= 0 && trace->watch_cand[w] < p->n, SR_ERR_INVALID_ARG,
                   "trace: watch_cand entries must lie in [0, n)");
    }
    generate(gen, rm, prompt, prompt_len, p, workspace, ws_bytes, (hipStream_t)stream, out_tokens, out,
             trace);
  });
}

sr_status sr_philox_fill(uint64_t seed, const uint32_t* ctr, int32_t n, uint32_t* out, void* stream) {
  return guard([&] {
    SR_REQUIRE(n >= 0, SR_ERR_INVALID_ARG, "n must be >= 0");
    SR_REQUIRE(n == 0 || (ctr && out), SR_ERR_INVALID_ARG, "NULL buffer");
    philox_fill(seed, ctr, n, out, (hipStream_t)stream);
  });
}

sr_status sr_sample(const float* logits, int32_t rows, int32_t vocab, const int32_t* cand, int32_t step,
                    float temperature, uint64_t seed, int32_t* tokens, void* stream) {
  return guard([&] {
    SR_REQUIRE(rows >= 0 && vocab >= 1 && step >= 0, SR_ERR_INVALID_ARG, "bad rows/vocab/step");
    SR_REQUIRE(rows == 0 || (logits && cand && tokens), SR_ERR_INVALID_ARG, "NULL buffer");
    SR_REQUIRE(std::isfinite(temperature) && temperature >= 0.f, SR_ERR_INVALID_ARG,
               "temperature must be finite and >= 0");
    SR_REQUIRE(vocab <= 262144, SR_ERR_UNSUPPORTED, "vocab above 262144");
    SampleArgs a;
    std::memset(&a, 0, sizeof(a));
    a.logits = logits; a.row_stride = vocab; a.rows = rows; a.vocab = vocab; a.cand = cand;
    a.step = step; a.temperature = temperature; a.seed = seed; a.next_tok = tokens; a.eos_id = -1;
    sample(a, (hipStream_t)stream);
  });
}

sr_status sr_select(const float* scores, const int32_t* cand, int32_t b, int32_t keep, int32_t* accept,
                    void* stream) {
  return guard([&] {
    SR_REQUIRE(b >= 1 && b <= kMaxN, SR_ERR_INVALID_ARG, "b must be in [1, 4096]");
    SR_REQUIRE(keep >= 1 && keep <= b, SR_ERR_INVALID_ARG, "keep must be in [1, b]");
    SR_REQUIRE(scores && cand && accept, SR_ERR_INVALID_ARG, "NULL buffer");
    select_topk(scores, cand, b, keep, accept, (hipStream_t)stream);
  });
}

sr_status sr_compact(const void* src, int64_t src_block_elems, void* dst, int64_t dst_block_elems,
                     const int32_t* keep_flag, int32_t b, int32_t n_layers, int32_t n_kv_heads,
                     int32_t head_dim, int32_t elem_bytes, int32_t cap_src, int32_t cap_dst, int32_t len,
                     int32_t* src_row, int32_t* new_count, void* stream) {
  return guard([&] {
    SR_REQUIRE(src && dst && keep_flag && src_row && new_count, SR_ERR_INVALID_ARG, "NULL buffer");
    SR_REQUIRE(b >= 1 && b <= kMaxN, SR_ERR_INVALID_ARG, "b must be in [1, 4096]");
    SR_REQUIRE(n_layers >= 1 && n_kv_heads >= 1 && head_dim >= 1, SR_ERR_INVALID_ARG, "bad shape");
    SR_REQUIRE(elem_bytes == 2 || elem_bytes == 4, SR_ERR_INVALID_ARG, "elem_bytes must be 2 or 4");
    SR_REQUIRE((head_dim * elem_bytes) % 16 == 0, SR_ERR_UNSUPPORTED, "KV row must be 16-byte multiple");
    SR_REQUIRE(len >= 0 && cap_src >= 1 && cap_dst >= 1 && len <= cap_src && len <= cap_dst,
               SR_ERR_INVALID_ARG, "len must be <= cap_src and cap_dst");
    SR_REQUIRE((int64_t)b * n_kv_heads * cap_src * head_dim <= src_block_elems &&
                   (int64_t)b * n_kv_heads * cap_dst * head_dim <= dst_block_elems,
               SR_ERR_INVALID_ARG, "pool blocks too small for b rows");
    const char* s0 = (const char*)src;
    const char* s1 = s0 + 2 * (int64_t)n_layers * src_block_elems * elem_bytes;
    const char* d0 = (const char*)dst;
    const char* d1 = d0 + 2 * (int64_t)n_layers * dst_block_elems * elem_bytes;
    SR_REQUIRE(s1 <= d0 || d1 <= s0, SR_ERR_INVALID_ARG, "src and dst overlap");
    CompactArgs a;
    std::memset(&a, 0, sizeof(a));
    a.src = src; a.src_block = src_block_elems; a.dst = dst; a.dst_block = dst_block_elems;
    a.keep_flag = keep_flag; a.b = b; a.max_rows = b; a.n_layers = n_layers; a.hkv = n_kv_heads;
    a.hd = head_dim; a.elem_bytes = elem_bytes; a.cap_src = cap_src; a.cap_dst = cap_dst; a.len = len;
    a.scratch_src_row = src_row;
    a.new_count = new_count;
    compact(a, (hipStream_t)stream);
  });
}

size_t sr_projection_scratch(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t mode) {
  if (M < 0 || N < 0 || K < 0 || mode < 0 || mode > 3) return 0;
  if (dtype == SR_F32) return (size_t)M * (mode == 2 ? 2 * (size_t)N : (size_t)N);
  return gemm_partial_elems(dtype, M, N, K, mode == 2);
}

sr_status sr_projection(int32_t dtype, const void* x, const void* w, int32_t M, int32_t N, int32_t K,
                        int32_t mode, void* out, float* partial, size_t partial_elems, void* stream) {
  return guard([&] {
    SR_REQUIRE(dtype == SR_F32 || dtype == SR_BF16, SR_ERR_INVALID_ARG, "unknown dtype");
    SR_REQUIRE(M >= 0 && N >= 1 && K >= 1, SR_ERR_INVALID_ARG, "bad M/N/K");
    SR_REQUIRE(mode >= 0 && mode <= 3, SR_ERR_INVALID_ARG, "mode must be 0..3");
    SR_REQUIRE(K % 64 == 0, SR_ERR_UNSUPPORTED, "K must be a multiple of 64");
    SR_REQUIRE(M == 0 || (x && w && out), SR_ERR_INVALID_ARG, "NULL buffer");
    const size_t need = sr_projection_scratch(dtype, M, N, K, mode);
    SR_REQUIRE(partial_elems >= need && (need == 0 || partial), SR_ERR_WORKSPACE_TOO_SMALL,
               "partial scratch too small: need " + std::to_string(need) + " floats");
    GemmArgs g;
    g.dtype = dtype; g.A = x; g.lda = K; g.B = w; g.ldb = K; g.paired = mode == 2;
    g.pair_off = (int64_t)N * K; g.M = M; g.N = N; g.K = K;
    g.epi = mode == 1 ? EPI_RESID : EPI_STORE; g.out = out; g.ldo = N;
    g.out_bf16 = (mode == 2 || mode == 3) && dtype == SR_BF16;
    gemm(g, partial, partial_elems, (hipStream_t)stream);
  });
}

size_t sr_decode_attention_scratch(int32_t head_dim, int32_t n_heads, int32_t n_kv_heads, int32_t rows, int32_t P,
                                   int32_t lt) {
  if (head_dim <= 0 || n_heads <= 0 || n_kv_heads <= 0 || rows <= 0 || P < 0 || lt < 0) return 0;
  return (size_t)rows * n_heads * decode_attn_splits(rows, n_kv_heads, P + lt) * (head_dim + 2);
}

// Validated arguments of the kernel-level decode attention entry points
// (rows == 0 leaves a.rows = 0: nothing to launch).
static DecodeAttnArgs decode_attention_args(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                                            int32_t rows, const float* q, const void* kpre, const void* vpre,
                                            int32_t P, const void* ktail, const void* vtail, int32_t cap, int32_t lt,
                                            void* out) {
  SR_REQUIRE(dtype == SR_F32 || dtype == SR_BF16, SR_ERR_INVALID_ARG, "unknown dtype");
  SR_REQUIRE(head_dim == 32 || head_dim == 64 || head_dim == 128, SR_ERR_UNSUPPORTED,
             "head_dim must be 32, 64 or 128");
  SR_REQUIRE(n_heads >= 1 && n_kv_heads >= 1 && n_heads % n_kv_heads == 0, SR_ERR_INVALID_ARG, "bad head counts");
  const int g = n_heads / n_kv_heads;
  SR_REQUIRE(g == 1 || g == 2 || g == 4 || g == 8, SR_ERR_UNSUPPORTED, "query heads per KV head must be 1, 2, 4 or 8");
  SR_REQUIRE(rows >= 0 && P >= 0 && lt >= 0 && lt <= cap && (rows == 0 || P + lt >= 1), SR_ERR_INVALID_ARG,
             "bad rows / P / lt / cap");
  DecodeAttnArgs a;
  a.dtype = dtype; a.hd = head_dim; a.hq = n_heads; a.hkv = n_kv_heads; a.rows = rows; a.q = q;
  a.kpre = kpre; a.vpre = vpre; a.P = P; a.ktail = ktail; a.vtail = vtail; a.cap = cap; a.lt = lt;
  a.out = out; a.part = nullptr; a.part_cap = 0;
  if (rows == 0) return a;
  SR_REQUIRE(q && out && (P == 0 || (kpre && vpre)) && (lt == 0 || (ktail && vtail)), SR_ERR_INVALID_ARG,
             "NULL buffer");
  return a;
}

sr_status sr_decode_attention(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads, int32_t rows,
                              const float* q, const void* kpre, const void* vpre, int32_t P, const void* ktail,
                              const void* vtail, int32_t cap, int32_t lt, void* out, float* scratch,
                              size_t scratch_elems, void* stream) {
  return guard([&] {
    DecodeAttnArgs a = decode_attention_args(dtype, head_dim, n_heads, n_kv_heads, rows, q, kpre, vpre, P, ktail,
                                             vtail, cap, lt, out);
    if (rows == 0) return;
    const size_t need = sr_decode_attention_scratch(head_dim, n_heads, n_kv_heads, rows, P, lt);
    SR_REQUIRE(scratch && scratch_elems >= need, SR_ERR_WORKSPACE_TOO_SMALL,
               "attention scratch too small: need " + std::to_string(need) + " floats");
    a.part = scratch;
    a.part_cap = scratch_elems;
    decode_attn(a, (hipStream_t)stream);
  });
}

sr_status sr_decode_attention_noalloc(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                                      int32_t rows, const float* q, const void* kpre, const void* vpre, int32_t P,
                                      const void* ktail, const void* vtail, int32_t cap, int32_t lt, void* out,
                                      void* stream) {
  return guard([&] {
    DecodeAttnArgs a = decode_attention_args(dtype, head_dim, n_heads, n_kv_heads, rows, q, kpre, vpre, P, ktail,
                                             vtail, cap, lt, out);
    if (rows == 0) return;
    const size_t need = decode_attn_part_floats(a);
    SR_REQUIRE(need <= kStaticScratchFloats, SR_ERR_WORKSPACE_TOO_SMALL,
               "decode attention needs " + std::to_string(need * sizeof(float)) +
                   " bytes of partials, above the static scratch of " +
                   std::to_string(kStaticScratchFloats * sizeof(float)) + " bytes");
    a.part = static_scratch_of_current_device();
    a.part_cap = kStaticScratchFloats;
    decode_attn(a, (hipStream_t)stream);
  });
}

size_t sr_decode_attention_noalloc_limit(void) { return kStaticScratchFloats * sizeof(float); }

sr_status sr_prefill_attention(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads, int32_t rows,
                               int32_t lr, const float* q, const void* kpre, const void* vpre, int32_t P,
                               const void* kown, const void* vown, int32_t cap, int32_t t0, void* out,
                               void* stream) {
  return guard([&] {
    SR_REQUIRE(dtype == SR_F32 || dtype == SR_BF16, SR_ERR_INVALID_ARG, "unknown dtype");
    SR_REQUIRE(head_dim == 32 || head_dim == 64 || head_dim == 128, SR_ERR_UNSUPPORTED,
               "head_dim must be 32, 64 or 128");
    SR_REQUIRE(n_heads >= 1 && n_kv_heads >= 1 && n_heads % n_kv_heads == 0, SR_ERR_INVALID_ARG, "bad head counts");
    const int g = n_heads / n_kv_heads;
    SR_REQUIRE(g == 1 || g == 2 || g == 4 || g == 8, SR_ERR_UNSUPPORTED, "query heads per KV head must be 1, 2, 4 or 8");
    SR_REQUIRE(rows >= 0 && lr >= 0 && P >= 0 && t0 >= 0 && (int64_t)t0 + lr <= cap, SR_ERR_INVALID_ARG,
               "bad rows / lr / P / t0 / cap");
    if (rows == 0 || lr == 0) return;
    SR_REQUIRE(q && out && kown && vown && (P == 0 || (kpre && vpre)), SR_ERR_INVALID_ARG, "NULL buffer");
    PrefillAttnArgs a;
    a.dtype = dtype; a.hd = head_dim; a.hq = n_heads; a.hkv = n_kv_heads; a.rows = rows; a.lr = lr;
    a.q = q; a.kpre = kpre; a.vpre = vpre; a.P = P; a.kown = kown; a.vown = vown; a.cap = cap; a.t0 = t0;
    a.out = out;
    prefill_attn(a, (hipStream_t)stream);
  });
}

sr_status sr_logits_teacher_forced(const sr_model* gen, const sr_model* rm, const int32_t* prompt,
                                   int32_t prompt_len, const sr_params* p, const int32_t* tokens, int32_t rows,
                                   int32_t len, float* logits_out, void* workspace, size_t ws_bytes,
                                   void* stream) {
  return guard([&] {
    check_pair(gen, rm);
    check_params(p, gen);
    check_prompt(prompt, prompt_len, gen->cfg.vocab);
    teacher_forced(gen, rm, prompt, prompt_len, p, tokens, rows, len, logits_out, workspace, ws_bytes,
                   (hipStream_t)stream);
  });
}

sr_status sr_reward_scores(const sr_model* gen, const sr_model* rm, const int32_t* prompt, int32_t prompt_len,
                           const sr_params* p, const int32_t* tokens, const int32_t* lens, int32_t rows,
                           int32_t max_len, float* scores, void* workspace, size_t ws_bytes, void* stream) {
  return guard([&] {
    check_pair(gen, rm);
    check_params(p, gen);
    check_prompt(prompt, prompt_len, rm->cfg.vocab);
    reward_entry(gen, rm, prompt, prompt_len, p, tokens, lens, rows, max_len, scores, workspace, ws_bytes,
                 (hipStream_t)stream);
  });
}

}  // extern "C"
