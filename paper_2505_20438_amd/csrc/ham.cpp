// Host side of libham: configuration checks, buffer layouts, and the launch
// sequences of prefill and of one macro-step.  Every arithmetic step runs in
// the HIP kernels; this file only sequences them on the caller's stream.
#include "../../include/ham.h"
#include "../../include/ham_ops.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "ham_internal.h"
#include "kernels_misc.h"

using namespace ham;

namespace ham {
LaunchTiming& launch_timing() {
  static thread_local LaunchTiming t;
  return t;
}
}  // namespace ham

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(call)                                                                       \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess) return fail(HAM_EHIP, "%s: %s", #call, hipGetErrorString(e_));    \
  } while (0)

size_t al(size_t x) { return (x + 255) & ~size_t(255); }
int rup(int x, int m) { return (x + m - 1) / m * m; }

uint64_t sm64(uint64_t s, uint64_t i) {
  uint64_t z = s + (i + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

constexpr int MAX_GEMM_SPLIT = 16;
constexpr int MAX_ATTN_SPLIT = 64;
constexpr int LOCAL_SLOTS = 64;

size_t attn_part_bytes(int R, int H, int Hk, int hd);
int attn_splits_for(int dtype, int R, int Hk, int kv_max);

struct Layout {
  // dims
  int L, M, d, H, Hk, hd, F, V, G, B, P, steps;
  int QKV, HD, Vpad, S, max_pos, C, Tc, rows_dec, rows_max, Nmax, ctx_l[8];
  size_t es;  // element size of the storage type
  // weights
  size_t E, Pe, Aqkv, Ao, Alin, Wlm, gf, gmf, cos_t, sin_t, w_bytes;
  std::vector<size_t> Wqkv, Wo, Wgu, Wd, g1, g2;
  // state
  size_t Kc, VTc, kv_layer, seq, st_bytes;
  // workspace
  size_t x, x2, xp, xn, qkv, q, ao, act, part, qpart, ssb, nss, tss, gctr, actr, apart, bval, bidx, stopb, ctx, emb_in, emb_o, emb_y,
      rope_cs, Kloc, VTloc, loc_layer, ws_bytes;
};

const char* check_cfg(const ham_config* c) {
  if (!c) return "null config";
  if (c->n_layers < 1 || c->d_model < 32 || c->n_heads < 1 || c->n_kv_heads < 1 || c->ffn_dim < 16 ||
      c->vocab < 2 || c->micro_layers < 1)
    return "dimensions must be positive (micro_layers >= 1)";
  if (c->head_dim != 64 && c->head_dim != 128) return "head_dim must be 64 or 128";
  if (c->n_heads % c->n_kv_heads != 0 || c->n_heads / c->n_kv_heads > 4) return "n_heads must be a multiple (<= 4x) of n_kv_heads";
  if (c->d_model % 32 || (c->n_heads * c->head_dim) % 32 || c->ffn_dim % 32) return "d_model, n_heads*head_dim and ffn_dim must be multiples of 32";
  if (c->d_model > 8192) return "d_model must be <= 8192";
  if (c->max_group < 1 || c->max_group > 4) return "max_group must be in 1..4";
  if (c->embed_layers != 0 && c->embed_layers != 1) return "embed_layers must be 1 (one cross-attention layer)";
  if (c->n_ctx_layers < 0 || c->n_ctx_layers > 8) return "n_ctx_layers must be in 0..8";
  for (int i = 0; i < c->n_ctx_layers; ++i) {
    if (c->ctx_layers[i] < 1 || c->ctx_layers[i] > c->n_layers) return "ctx_layers must lie in 1..n_layers";
    if (i > 0 && c->ctx_layers[i] <= c->ctx_layers[i - 1]) return "ctx_layers must be strictly increasing";
  }
  if (c->stop_mode < 0 || c->stop_mode > 3) return "unknown stop_mode";
  if (c->stop_mode == HAM_STOP_TOKEN && (c->stop_id < 0 || c->stop_id >= c->vocab)) return "stop_id out of range";
  if (!(c->stop_conf >= 0.f && c->stop_conf <= 1.f)) return "stop_conf must be in [0, 1]";
  if (c->dtype != HAM_F32 && c->dtype != HAM_BF16) return "dtype must be HAM_F32 or HAM_BF16";
  if (c->max_batch < 1 || c->max_batch > 64) return "max_batch must be in 1..64";
  if (c->max_prompt < 1 || c->max_steps < 0) return "max_prompt >= 1 and max_steps >= 0 required";
  if ((long long)c->max_prompt + c->max_steps > (1 << 24)) return "capacity too large";
  if (!(c->rope_theta > 1.f) || !(c->norm_eps > 0.f)) return "rope_theta > 1 and norm_eps > 0 required";
  return nullptr;
}

Layout make_layout(const ham_config* c) {
  Layout y;
  y.L = c->n_layers; y.M = c->micro_layers; y.d = c->d_model; y.H = c->n_heads; y.Hk = c->n_kv_heads;
  y.hd = c->head_dim; y.F = c->ffn_dim; y.V = c->vocab; y.G = c->max_group; y.B = c->max_batch;
  y.P = c->max_prompt; y.steps = c->max_steps;
  y.es = c->dtype == HAM_BF16 ? 2 : 4;
  y.HD = y.H * y.hd;
  y.QKV = (y.H + 2 * y.Hk) * y.hd;
  y.Vpad = rup(y.V + 1, 32);
  y.S = rup(y.P + y.steps, 64);
  y.max_pos = y.P + y.G * (y.steps + 1) + 8;
  // context layers of the micro decoder: the configured set, or C = min(4, L)
  // layers at ceil(i * L / C), i = 1..C (evenly spaced, the last one included)
  y.C = c->n_ctx_layers > 0 ? c->n_ctx_layers : std::min(4, y.L);
  for (int i = 0; i < 8; ++i)
    y.ctx_l[i] = i >= y.C ? -1
                 : c->n_ctx_layers > 0 ? c->ctx_layers[i]
                                       : (int)(((long long)(i + 1) * y.L + y.C - 1) / y.C);
  y.Tc = std::min(y.P, 2048);
  y.rows_dec = y.B * (y.C + 1);
  y.rows_max = std::max(y.Tc, std::max(y.rows_dec, 5 * y.B));
  y.Nmax = std::max(std::max(y.QKV, 2 * y.F), std::max(y.d, 3 * y.HD));
  const size_t es = y.es;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t r = o; o += al(bytes); return r; };
  // weights
  y.E = take((size_t)y.V * y.d * es);
  y.Pe = take((size_t)4 * y.d * es);
  y.Aqkv = take((size_t)3 * y.HD * y.d * es);
  y.Ao = take((size_t)y.d * y.HD * es);
  y.Alin = take((size_t)y.d * y.d * es);
  y.Wlm = take((size_t)y.Vpad * y.d * es);
  for (int j = 0; j < y.L + y.M; ++j) {
    y.Wqkv.push_back(take((size_t)y.QKV * y.d * es));
    y.Wo.push_back(take((size_t)y.d * y.HD * es));
    y.Wgu.push_back(take((size_t)2 * y.F * y.d * es));
    y.Wd.push_back(take((size_t)y.d * y.F * es));
    y.g1.push_back(take((size_t)y.d * 4));
    y.g2.push_back(take((size_t)y.d * 4));
  }
  y.gf = take((size_t)y.d * 4);
  y.gmf = take((size_t)y.d * 4);
  y.cos_t = take((size_t)y.max_pos * (y.hd / 2) * 4);
  y.sin_t = take((size_t)y.max_pos * (y.hd / 2) * 4);
  y.w_bytes = o;
  // state: smashed KV cache (K slot-major, V d-major) and per-sequence counters
  o = 0;
  y.kv_layer = al((size_t)y.B * y.Hk * y.S * y.hd * es);
  y.Kc = take(y.kv_layer * y.L);
  y.VTc = take(y.kv_layer * y.L);
  y.seq = take((size_t)y.B * 4 * 32);
  y.st_bytes = o;
  // workspace
  o = 0;
  const size_t R = y.rows_max;
  y.x = take((size_t)y.rows_dec * y.d * 4);
  y.x2 = take((size_t)y.rows_dec * y.d * 4);  // second residual buffer (staged norms write the other one)
  y.xp = take((size_t)y.Tc * y.d * 4);
  // activation operands: 4 bytes per value (fp32, or a bf16 hi/lo pair)
  y.xn = take(R * std::max(y.d, y.HD) * 4);
  y.qkv = take(R * std::max(y.QKV, 3 * y.HD) * 4);
  y.q = take(R * y.HD * 4);
  y.ao = take(R * y.HD * 4);
  y.act = take(R * y.F * 4);
  static_assert(MAX_GEMM_SPLIT * 64 <= PART_ROWS, "partial buffer rows");
  y.part = take((size_t)PART_ROWS * y.Nmax * 4);
  y.qpart = take((size_t)PART_ROWS * y.QKV * 4);  // q/k/v partials (read while part is pending)
  y.ssb = take((size_t)MAX_GEMM_SPLIT * 64 * 4);
  y.nss = take((size_t)y.rows_max * ((y.d + 255) / 256) * 4);  // two-phase RMSNorm chunk sums
  y.tss = take((size_t)NORM_OUT_MAX_TILES * NORM_OUT_MAX_ROWS * 4);  // NormOut tile sums of squares
  y.gctr = take((size_t)(y.Vpad / 32 + y.Nmax / 32 + 64) * 4);
  y.actr = take((size_t)y.rows_dec * y.Hk * 4);
  y.apart = take(attn_part_bytes(y.rows_dec, y.H, y.Hk, y.hd));
  y.bval = take((size_t)(y.Vpad / 16) * 64 * 4);
  y.bidx = take((size_t)(y.Vpad / 16) * 64 * 4);
  y.stopb = take(64 * 4);
  y.ctx = take((size_t)y.B * y.C * y.d * 4);
  y.emb_in = take((size_t)5 * y.B * y.d * 4);
  y.emb_o = take((size_t)y.B * y.HD * 4);
  y.emb_y = take((size_t)y.B * y.d * 4);
  y.rope_cs = take((size_t)y.B * y.hd * 4);
  y.loc_layer = al((size_t)y.B * y.Hk * LOCAL_SLOTS * y.hd * es);
  y.Kloc = take(y.loc_layer * y.M);
  y.VTloc = take(y.loc_layer * y.M);
  y.ws_bytes = o;
  return y;
}

}  // namespace

struct ham_model {
  ham_config cfg;
  Layout y;
  char* w;
  char* st;
  char* ws;
  hipStream_t s;
  SeqPtrs sp;
  int batch = 0, prompt_len = 0, steps_done = -1, has_teacher = 0, kv_visible = 0;
  // host-side fields of the last ham_state_save (saved_steps < 0: none)
  int saved_batch = 0, saved_prompt = 0, saved_steps = -1, saved_teacher = 0;
  float tau;
  float* dbg = nullptr;
  // optional per-class event timing
  struct Rec { int kind; hipEvent_t a, b; double bytes; };
  bool prof_on = false;
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  size_t pool_used = 0;
  hipEvent_t ev() {
    if (pool_used == pool.size()) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return nullptr;
      pool.push_back(e);
    }
    return pool[pool_used++];
  }
  int prof_kind = -1;
  double prof_bytes = 0;
  hipEvent_t prof_a = nullptr;
  // The launches of a macro-step after k_macro_begin, captured once as a HIP
  // graph and replayed (a dependent launch costs ~0.6 us less from a graph).
  // Everything they depend on is fixed until the key changes.
  struct GraphKey {
    int batch = -1, prompt_len = -1, has_teacher = -1;
    const void* out_tokens = nullptr;
    const void* out_lens = nullptr;
    const void* dbg = nullptr;
    bool operator==(const GraphKey& o) const {
      return batch == o.batch && prompt_len == o.prompt_len && has_teacher == o.has_teacher &&
             out_tokens == o.out_tokens && out_lens == o.out_lens && dbg == o.dbg;
    }
  };
  bool use_graph = true;
  hipStream_t cap_stream = nullptr;  // private stream the graph is captured on (launched on s)
  hipGraph_t graph = nullptr;
  hipGraphExec_t gexec = nullptr;
  GraphKey gkey;
  void drop_graph() {
    if (gexec) hipGraphExecDestroy(gexec);
    if (graph) hipGraphDestroy(graph);
    gexec = nullptr;
    graph = nullptr;
    gkey = GraphKey{};
  }
  // the next kernel launched is timed by events attached to its dispatch
  void pbegin(int kind, double bytes) {
    if (!prof_on || kind < 0) return;
    prof_kind = kind;
    prof_bytes = bytes;
    prof_a = ev();
    hipEvent_t b = ev();
    if (prof_a && b) launch_timing() = LaunchTiming{prof_a, b};
  }
  void pend() {
    if (!prof_on || !prof_a) return;
    LaunchTiming& t = launch_timing();
    if (!t.start) recs.push_back(Rec{prof_kind, prof_a, pool[pool_used - 1], prof_bytes});
    t = LaunchTiming{};  // nothing was launched: disarm
    prof_a = nullptr;
  }
  ~ham_model() {
    drop_graph();
    if (cap_stream) hipStreamDestroy(cap_stream);
    for (hipEvent_t e : pool) hipEventDestroy(e);
  }
  // typed views
  template <typename P> P* W(size_t off) const { return (P*)(w + off); }
  template <typename P> P* WS(size_t off) const { return (P*)(ws + off); }
};

namespace {

SeqPtrs seq_ptrs(char* st, const Layout& y) {
  int* base = (int*)(st + y.seq);
  const int B = y.B;
  SeqPtrs p;
  int* q = base;
  auto next = [&](int n) { int* r = q; q += (size_t)n * B; return r; };
  p.kv_len = next(1); p.pos_last = next(1); p.cur_pos = next(1); p.cur_slot = next(1);
  p.emitted = next(1); p.budget = next(1); p.done = next(1); p.groups = next(1);
  p.hist = next(5); p.step_on = next(1); p.fused = next(1); p.active = next(1);
  p.grp_n = next(1); p.grp_tok = next(4); p.forced = next(1); p.teacher = next(4); p.err = next(1);
  return p;
}

int dtype_of(const ham_model* m) { return m->cfg.dtype; }

// algorithmic bytes of one weight GEMM: weights once, activation rows in (4 B per
// value), fp32 results out
double gemm_bytes(const Layout& y, int N, int K, int M) {
  return (double)N * K * y.es + (double)M * K * 4 + (double)M * N * 4;
}

// A split-K GEMM result still held as partials (the next RMSNorm adds it to x),
// or (tss set) the first half of the next RMSNorm already done by a NormOut
// epilogue: x is up to date, the operand buffer holds g * x of the next norm
// and tss the per-tile sums of squares of x (tss_n tiles).  A full RMSNorm
// may still run on such rows: it reads x and ignores the rest.
struct Pending {
  const float* part = nullptr;
  int nsplit = 0, M = 0;
  const float* tss = nullptr;
  int tss_n = 0;
};

int gemm_p(ham_model* m, int epi, const GemmArgs& a, int max_split, int kind, int* nsplit) {
  m->pbegin(kind, gemm_bytes(m->y, a.N, a.K, a.M));
  const bool base = kind >= HAM_PROF_QKV && kind <= HAM_PROF_DOWN;
  const int rc = launch_gemm(dtype_of(m), epi, a, max_split, m->s, base ? 0 : 1, nsplit);
  m->pend();
  return rc;
}

// RMSNorm of R rows of x (row r reads x row r*stride + off) into the operand buffer,
// after adding a pending split-K result to those rows and copying them to ctx
int norm_rows(ham_model* m, float* x, int R, int stride, int off, const float* g, Pending& pend, float* ctx,
               int ldctx, float* hid, const int* gate, int gate_n) {
  const Layout& y = m->y;
  NormArgs na{};
  na.x = x; na.ldx = y.d; na.row_stride = stride; na.row_off = off; na.g = g; na.d = y.d; na.R = R;
  na.eps = m->cfg.norm_eps; na.out = m->WS<char>(y.xn); na.ldo = y.d; na.hid = hid; na.ldh = y.d;
  na.part = pend.part; na.nsplit = pend.nsplit; na.pM = pend.M; na.ctx = ctx; na.ldctx = ldctx;
  na.gate = gate; na.gate_n = gate_n; na.ss = m->WS<float>(y.nss);
  pend = Pending{};
  m->pbegin(HAM_PROF_NORM, (double)R * y.d * 4 * (na.nsplit + 3));
  const int rc = launch_rmsnorm(dtype_of(m), na, m->s);
  m->pend();
  return rc ? fail(HAM_EINVAL, "rmsnorm shape") : HAM_OK;
}

// The RMSNorm feeding GEMM `ga` (rows x, gain g): where the batched GEMM can
// build the normed operand itself (XS_NORMW), only the norm's first phase
// launches; otherwise the whole norm writes the operand buffer (XS_ACT).
int norm_into_gemm(ham_model* m, GemmArgs& ga, int epi, float* x, int R, const float* g, Pending& pend,
                   float* ctx, int ldctx, const int* gate, int gate_n) {
  const Layout& y = m->y;
  GemmArgs gw = ga;
  gw.xsrc = XS_NORMW;
  gw.xs.x = x; gw.xs.ldx = y.d; gw.xs.g = g; gw.xs.eps = m->cfg.norm_eps;
  gw.xs.ssw = m->WS<float>(y.nss); gw.xs.nchw = (y.d + 255) / 256;
  if (gemm_stage_fits(dtype_of(m), epi, gw, MAX_GEMM_SPLIT)) {
    NormArgs na{};
    na.x = x; na.ldx = y.d; na.row_stride = 1; na.row_off = 0; na.g = g; na.d = y.d; na.R = R;
    na.eps = m->cfg.norm_eps; na.part = pend.part; na.nsplit = pend.nsplit; na.pM = pend.M;
    na.ctx = ctx; na.ldctx = ldctx; na.gate = gate; na.gate_n = gate_n; na.ss = m->WS<float>(y.nss);
    m->pbegin(HAM_PROF_NORM, (double)R * y.d * 4 * (na.nsplit + 3));
    const int nrc = launch_norm_reduce(na, m->s);
    m->pend();
    if (nrc == 0) {
      pend = Pending{};
      ga = gw;
      return HAM_OK;
    }
  }
  if (norm_rows(m, x, R, 1, 0, g, pend, ctx, ldctx, nullptr, gate, gate_n)) return HAM_EINVAL;
  ga.xsrc = XS_ACT; ga.X = m->WS<char>(y.xn); ga.ldx = y.d;
  return HAM_OK;
}

// The rest of a layer after attention: o-projection into the residual, second
// norm, gate/up with the SwiGLU epilogue, down-projection into the residual.
template <typename GK>
int layer_tail(ham_model* m, int j, int R, float* x, int split, const int* gate, int gate_n, Pending& pend,
               const GK& gk) {
  const Layout& y = m->y;
  int ns = 1;
  GemmArgs ga{};
  ga.part = m->WS<float>(y.part); ga.gate = gate; ga.gate_n = gate_n; ga.M = R;
  ga.W = m->W<char>(y.Wo[j]); ga.N = y.d; ga.K = y.HD; ga.X = m->WS<char>(y.ao); ga.ldx = y.HD;
  ga.out = x; ga.ldo = y.d;
  if (gemm_p(m, EPI_RESID, ga, split, gk(HAM_PROF_O), &ns)) return fail(HAM_EINVAL, "o-proj gemm shape");
  if (ns > 1) pend = Pending{m->WS<float>(y.part), ns, R};

  ga.W = m->W<char>(y.Wgu[j]); ga.N = 2 * y.F; ga.K = y.d;
  ga.out = m->WS<char>(y.act); ga.ldo = y.F;
  if (norm_into_gemm(m, ga, EPI_SWIGLU, x, R, m->W<float>(y.g2[j]), pend, nullptr, 0, gate, gate_n))
    return HAM_EINVAL;
  if (gemm_p(m, EPI_SWIGLU, ga, 1, gk(HAM_PROF_GU), &ns)) return fail(HAM_EINVAL, "gate/up gemm shape");

  ga.xsrc = XS_ACT;
  ga.W = m->W<char>(y.Wd[j]); ga.N = y.d; ga.K = y.F; ga.X = m->WS<char>(y.act); ga.ldx = y.F;
  ga.out = x; ga.ldo = y.d;
  if (gemm_p(m, EPI_RESID, ga, split, gk(HAM_PROF_DOWN), &ns)) return fail(HAM_EINVAL, "down gemm shape");
  if (ns > 1) pend = Pending{m->WS<float>(y.part), ns, R};
  return HAM_OK;
}

// Fused decode step of a layer (rows of mode DECODE or MICROK): where the RoPE
// factors of each row are, and the bound on the cached slots of every row.
struct StepAttn {
  const float* cos_p;
  const float* sin_p;
  long long cs_stride;
  int kv_cap;
};

// slot splits of the fused step.  A workgroup streams its share of the cache at
// about the rate of one compute unit and holds one CU (its register use allows
// one per CU), so the (row, kv head) pairs are split until about 256
// workgroups run, keeping at least two key blocks per split; long contexts
// then loop over chunks inside each wave rather than adding workgroups.
int attn_step_splits(int dtype, int R, int Hk, int hd, int kv_cap) {
  (void)hd;
  const int kb = dtype == HAM_BF16 ? 32 : 16;
  const int blocks = (kv_cap + kb - 1) / kb;
  const int for_width = std::min((256 + R * Hk - 1) / (R * Hk), (blocks + 1) / 2);
  return std::max(1, std::min(MAX_ATTN_SPLIT, for_width));
}

// splits of the base layers' fused step in a macro-step over B sequences: at
// most 16 at up to 8 rows (each split adds records to merge: the
// o-projection's prologue merges them where it fits, else k_attn_combine;
// 8 or 4 splits measured slower)
int macro_attn_splits(int dtype, int B, int Hk, int hd, int kv_cap) {
  const int n = attn_step_splits(dtype, B, Hk, hd, kv_cap);
  return B <= 8 ? std::min(16, n) : n;
}

// one transformer layer (base layer j < L, micro layer j >= L) over R rows.
// On entry `pend` may hold the previous layer's down-projection partials (folded
// into x by the first norm, which also copies the updated rows to ctx_prev); on
// exit it holds this layer's, if split.
// The fused decode path of one layer (rows of mode DECODE or MICROK): the first
// RMSNorm folded into the q/k/v projection, the fused attention step, the
// merge of the attention splits folded into the o-projection, the second
// RMSNorm folded into gate/up.  Where a staged prologue does not fit, the
// separate kernels run instead.  A folded norm writes the updated residual to
// the other row buffer: `x` names the current one on entry and on exit.
//
// Rows 1..8 of a model wide enough to give every CU a 16-column tile (d >=
// 4096), and at narrower widths rows 2..8 whose q/k/v prologue does not fit
// (it would hold the rows' whole k-range of X in LDS), take the NormOut form
// instead: the o-projection and the down projection run unsplit, one
// workgroup per column tile, and their epilogue finishes the residual, writes
// g * x of the next norm (gain g2, or `g_next`: the next layer's g1, null after
// the last layer) and per-tile sums of squares; the fused attention step and
// the gate/up epilogue apply 1/rms.  Only a layer whose input rows come from
// elsewhere (pend without tss) normalises them itself (the staged prologue, or
// an RMSNorm launch).  The down projection then also copies its output rows to
// `ctx_out` (where the next norm would have).
int run_layer_step(ham_model* m, int j, int R, const RowMap& rm, float*& x, void* Kc, void* VTc, long long sb,
                   long long sh, int S, int attn_split, const int* gate, int gate_n, Pending& pend,
                   float* ctx_prev, int ldctx, int kv_visible, const StepAttn& step, bool base,
                   const float* g_next, float* ctx_out) {
  const Layout& y = m->y;
  const int dt = dtype_of(m);
  const auto gk = [&](int kind) { return base ? kind : HAM_PROF_MICRO; };
  float* xa = m->WS<float>(y.x);
  float* xb = m->WS<float>(y.x2);
  const auto other = [&](float* p) { return p == xa ? xb : xa; };
  const int split = MAX_GEMM_SPLIT;
  const float eps = m->cfg.norm_eps;
  int ns = 1;

  // q/k/v projection, first norm folded in; its partials go to qpart
  GemmArgs ga{};
  ga.gate = gate; ga.gate_n = gate_n; ga.M = R;
  ga.W = m->W<char>(y.Wqkv[j]); ga.N = y.QKV; ga.K = y.d; ga.out = m->WS<float>(y.qkv); ga.ldo = y.QKV;
  ga.part = m->WS<float>(y.qpart);
  ga.xsrc = XS_NORM;
  ga.xs.x = x; ga.xs.ldx = y.d; ga.xs.part = pend.part; ga.xs.nsplit = pend.nsplit; ga.xs.pM = pend.M;
  ga.xs.g = m->W<float>(y.g1[j]); ga.xs.eps = eps; ga.xs.x_out = other(x); ga.xs.ctx = ctx_prev;
  ga.xs.ldctx = ldctx; ga.xs.ss_out = m->WS<float>(y.ssb);
  const int qkv_split = std::min(split, attn_step_max_qkv_split());
  // NormOut form: decided on the q/k/v prologue without pending partials, so
  // that every layer of a batch takes the same form
  GemmArgs probe = ga;
  probe.xs.part = nullptr; probe.xs.nsplit = 0; probe.xs.pM = 0;
  const int ntiles_no = gemm_norm_out_tiles(y.d);
  // Taken at any row count once the unsplit launches give every CU a tile
  // (d >= 4096: 8B shape at batch 1, 480 -> 500 tok/s); narrower models only
  // where the staged q/k/v prologue does not fit (at d = 2048 the 128 unsplit
  // workgroups leave half the CUs idle: batch 1 of the 1B shape 9% slower).
  const bool fuse = R >= 1 && R <= NORM_OUT_MAX_ROWS && gemm_norm_out_fits(R, y.d, y.HD) &&
                    gemm_norm_out_fits(R, y.d, y.F) &&
                    (ntiles_no >= NORM_OUT_FILL_TILES || (R >= 2 && !gemm_stage_fits(dt, EPI_F32, probe, qkv_split)));
  const float* ss_in = nullptr;  // tile sums for the attention step's 1/rms
  int ss_in_n = 0;
  bool q_staged = false;
  if (pend.tss) {
    // the previous layer's NormOut epilogue wrote g1 * x and its tile sums
    // (and copied x to ctx_prev if that was asked)
    ga.xsrc = XS_ACT; ga.X = m->WS<char>(y.xn); ga.ldx = y.d;
    ss_in = pend.tss; ss_in_n = pend.tss_n;
    pend = Pending{};
  } else {
    q_staged = gemm_stage_fits(dt, EPI_F32, ga, qkv_split);
    if (!q_staged) {
      ga.xsrc = XS_ACT;
      if (norm_into_gemm(m, ga, EPI_F32, x, R, m->W<float>(y.g1[j]), pend, ctx_prev, ldctx, gate, gate_n))
        return HAM_EINVAL;
    }
  }
  if (gemm_p(m, EPI_F32, ga, qkv_split, gk(HAM_PROF_QKV), &ns)) return fail(HAM_EINVAL, "qkv gemm shape");
  if (q_staged) {
    x = other(x);
    pend = Pending{};
  }

  // the o-projection takes the attention splits directly when its prologue fits
  GemmArgs go{};
  go.gate = gate; go.gate_n = gate_n; go.M = R; go.part = m->WS<float>(y.part);
  go.W = m->W<char>(y.Wo[j]); go.N = y.d; go.K = y.HD; go.out = x; go.ldo = y.d;
  go.xsrc = XS_ATTN;
  go.xs.rec_o = m->WS<float>(y.apart);
  go.xs.rec_ml = m->WS<float>(y.apart) + (size_t)R * y.Hk * attn_split * (y.H / y.Hk) * y.hd;
  go.xs.ans = attn_split; go.xs.Hkv = y.Hk; go.xs.grp = y.H / y.Hk; go.xs.hd = y.hd;
  const bool o_staged = !fuse && attn_split > 1 && gemm_stage_fits(dt, EPI_RESID, go, split);

  AttnStepArgs sa{};
  sa.qkv = m->WS<float>(y.qkv); sa.part = ns > 1 ? m->WS<float>(y.qpart) : nullptr; sa.nsplit_qkv = ns;
  sa.pM = R; sa.ldqkv = y.QKV;
  sa.cos_p = step.cos_p; sa.sin_p = step.sin_p; sa.cs_stride = step.cs_stride;
  sa.K = Kc; sa.VT = VTc; sa.sb = sb; sa.sh = sh; sa.S = S;
  sa.H = y.H; sa.Hkv = y.Hk; sa.hd = y.hd; sa.R = R; sa.nsplit = attn_split; sa.kv_cap = step.kv_cap;
  sa.o = m->WS<char>(y.ao); sa.ldo = y.HD; sa.part_out = m->WS<float>(y.apart); sa.rm = rm;
  sa.combine = !o_staged;
  sa.gate = gate; sa.gate_n = gate_n;
  sa.ss = (q_staged && ns > 1) ? m->WS<float>(y.ssb) : nullptr; sa.ss_n = ns; sa.d = y.d; sa.eps = eps;
  if (ss_in) {
    sa.ss = ss_in; sa.ss_n = ss_in_n;
  }
  m->pbegin(base ? HAM_PROF_ATTN : -1, (double)kv_visible * y.Hk * y.hd * 2 * y.es);
  const int arc = launch_attn_step(dt, sa, m->s);
  m->pend();
  if (arc != 0) return fail(HAM_EINVAL, "attention step shape");

  if (!o_staged) {
    go.xsrc = XS_ACT; go.X = m->WS<char>(y.ao); go.ldx = y.HD;
  }
  if (fuse) {
    go.no.g = m->W<float>(y.g2[j]); go.no.act = m->WS<char>(y.xn); go.no.lda = y.d; go.no.ss = m->WS<float>(y.tss);
  }
  if (gemm_p(m, EPI_RESID, go, split, gk(HAM_PROF_O), &ns)) return fail(HAM_EINVAL, "o-proj gemm shape");
  if (fuse) {
    // gate/up on g2 * x, rows scaled by 1/rms before SwiGLU; then the down
    // projection's NormOut epilogue
    GemmArgs gu{};
    gu.gate = gate; gu.gate_n = gate_n; gu.M = R;
    gu.W = m->W<char>(y.Wgu[j]); gu.N = 2 * y.F; gu.K = y.d; gu.out = m->WS<char>(y.act); gu.ldo = y.F;
    gu.xsrc = XS_ACT; gu.X = m->WS<char>(y.xn); gu.ldx = y.d;
    gu.rs.ss = m->WS<float>(y.tss); gu.rs.n = ntiles_no; gu.rs.d = y.d; gu.rs.eps = eps;
    if (gemm_p(m, EPI_SWIGLU, gu, 1, gk(HAM_PROF_GU), &ns)) return fail(HAM_EINVAL, "gate/up gemm shape");
    GemmArgs gd{};
    gd.gate = gate; gd.gate_n = gate_n; gd.M = R;
    gd.W = m->W<char>(y.Wd[j]); gd.N = y.d; gd.K = y.F; gd.X = m->WS<char>(y.act); gd.ldx = y.F;
    gd.out = x; gd.ldo = y.d; gd.ctx = ctx_out; gd.ldctx = ldctx;
    gd.no.g = g_next; gd.no.act = m->WS<char>(y.xn); gd.no.lda = y.d; gd.no.ss = m->WS<float>(y.tss);
    if (gemm_p(m, EPI_RESID, gd, 1, gk(HAM_PROF_DOWN), &ns)) return fail(HAM_EINVAL, "down gemm shape");
    pend = g_next ? Pending{nullptr, 0, 0, m->WS<float>(y.tss), ntiles_no} : Pending{};
    return HAM_OK;
  }
  if (ns > 1) pend = Pending{m->WS<float>(y.part), ns, R};

  // gate/up, second norm folded in
  GemmArgs gu{};
  gu.gate = gate; gu.gate_n = gate_n; gu.M = R; gu.part = m->WS<float>(y.part);  // free again once x is normed
  gu.W = m->W<char>(y.Wgu[j]); gu.N = 2 * y.F; gu.K = y.d; gu.out = m->WS<char>(y.act); gu.ldo = y.F;
  gu.xsrc = XS_NORM;
  gu.xs.x = x; gu.xs.ldx = y.d; gu.xs.part = pend.part; gu.xs.nsplit = pend.nsplit; gu.xs.pM = pend.M;
  gu.xs.g = m->W<float>(y.g2[j]); gu.xs.eps = eps; gu.xs.x_out = other(x);
  const bool u_staged = gemm_stage_fits(dt, EPI_SWIGLU, gu, 1);
  if (!u_staged) {
    gu.xsrc = XS_ACT;
    if (norm_into_gemm(m, gu, EPI_SWIGLU, x, R, m->W<float>(y.g2[j]), pend, nullptr, 0, gate, gate_n))
      return HAM_EINVAL;
  }
  if (gemm_p(m, EPI_SWIGLU, gu, 1, gk(HAM_PROF_GU), &ns)) return fail(HAM_EINVAL, "gate/up gemm shape");
  if (u_staged) {
    x = other(x);
    pend = Pending{};
  }

  GemmArgs gd{};
  gd.gate = gate; gd.gate_n = gate_n; gd.M = R; gd.part = m->WS<float>(y.part);
  gd.W = m->W<char>(y.Wd[j]); gd.N = y.d; gd.K = y.F; gd.X = m->WS<char>(y.act); gd.ldx = y.F;
  gd.out = x; gd.ldo = y.d;
  if (gemm_p(m, EPI_RESID, gd, split, gk(HAM_PROF_DOWN), &ns)) return fail(HAM_EINVAL, "down gemm shape");
  if (ns > 1) pend = Pending{m->WS<float>(y.part), ns, R};
  return HAM_OK;
}

// Rows of micro step 1 above which its last micro layer runs attention and
// tail on each sequence's last row only (below, the batched GEMMs cost the
// same for fewer rows: they stream the weights either way)
constexpr int LAST_ROWS_MIN = 64;

int run_layer(ham_model* m, int j, int R, const RowMap& rm, float*& x, bool prefill, void* Kc, void* VTc,
              long long sb, long long sh, int S, int attn_split, const int* gate, int gate_n, Pending& pend,
              float* ctx_prev, int ldctx, int kv_visible, const StepAttn* step, const float* g_next = nullptr,
              float* ctx_out = nullptr, bool last_rows = false, bool kv_only = false, bool last_row = false) {
  const Layout& y = m->y;
  const int dt = dtype_of(m);
  hipStream_t s = m->s;
  const bool base = !prefill && j < y.L;
  const auto gk = [&](int kind) { return prefill ? -1 : (base ? kind : HAM_PROF_MICRO); };
  // Base layers run for every sequence of the batch (finished rows compute values that
  // nothing reads; their KV append and decisions are skipped per row), so they carry no
  // gate: a gate costs a dependent memory round trip before any other load.
  if (base) {
    gate = nullptr;
    gate_n = 0;
  }
  if (step)
    return run_layer_step(m, j, R, rm, x, Kc, VTc, sb, sh, S, attn_split, gate, gate_n, pend, ctx_prev, ldctx,
                          kv_visible, *step, base, g_next, ctx_out);
  const int split = prefill ? 1 : MAX_GEMM_SPLIT;
  int ns = 1;
  GemmArgs ga{};
  ga.part = m->WS<float>(y.part); ga.gate = gate; ga.gate_n = gate_n;
  ga.W = m->W<char>(y.Wqkv[j]); ga.N = y.QKV; ga.K = y.d; ga.M = R;
  ga.out = m->WS<float>(y.qkv); ga.ldo = y.QKV;
  if (prefill) {
    if (norm_rows(m, x, R, 1, 0, m->W<float>(y.g1[j]), pend, ctx_prev, ldctx, nullptr, gate, gate_n))
      return HAM_EINVAL;
    ga.X = m->WS<char>(y.xn); ga.ldx = y.d;
  } else if (norm_into_gemm(m, ga, EPI_F32, x, R, m->W<float>(y.g1[j]), pend, ctx_prev, ldctx, gate, gate_n)) {
    return HAM_EINVAL;
  }
  if (gemm_p(m, EPI_F32, ga, split, gk(HAM_PROF_QKV), &ns)) return fail(HAM_EINVAL, "qkv gemm shape");

  RopeArgs ra{};
  ra.qkv = m->WS<float>(y.qkv); ra.ldqkv = y.QKV; ra.R = R; ra.q = m->WS<char>(y.q); ra.ldq = y.HD;
  ra.part = ns > 1 ? m->WS<float>(y.part) : nullptr; ra.nsplit = ns;
  ra.K = Kc; ra.VT = VTc; ra.sb = sb; ra.sh = sh; ra.S = S; ra.H = y.H; ra.Hkv = y.Hk; ra.hd = y.hd;
  ra.cos_t = m->W<float>(y.cos_t); ra.sin_t = m->W<float>(y.sin_t); ra.max_pos = y.max_pos; ra.rm = rm;
  ra.gate = gate; ra.gate_n = gate_n;
  launch_rope_append(dt, ra, s);
  if (kv_only) return HAM_OK;  // only this layer's K and V of these rows are read later

  AttnArgs aa{};
  aa.q = m->WS<char>(y.q); aa.ldq = y.HD; aa.K = Kc; aa.VT = VTc; aa.sb = sb; aa.sh = sh; aa.S = S;
  aa.H = y.H; aa.Hkv = y.Hk; aa.hd = y.hd; aa.R = R; aa.nsplit = attn_split; aa.o = m->WS<char>(y.ao);
  aa.ldo = y.HD; aa.part = m->WS<float>(y.apart); aa.rm = rm;  // rows gate themselves (row map)
  if (last_rows) {
    // The last micro layer of micro step 1: every row's K and V are in the
    // local cache now (the later micro steps attend over them), but only each
    // sequence's last row (its first token, local position C) goes on to the
    // decision, so attention and tail run on those B rows.  Their residual rows
    // are copied to the second residual buffer, which x then names; their q
    // rows are read in place (pitch C + 1 rows).
    if (prefill || rm.mode != ROWS_MICRO1 || R % (y.C + 1) != 0) return fail(HAM_EINVAL, "last-row micro layer");
    const int B = R / (y.C + 1);
    float* xc = m->WS<float>(y.x2);
    if (launch_copy_rows(x + (size_t)y.C * y.d, (long long)(y.C + 1) * y.d, xc, y.d, B, y.d, s))
      return fail(HAM_EINVAL, "row copy shape");
    RowMap r1 = rm;
    r1.mode = ROWS_MICROK;
    r1.k = 1;  // local position C + k - 1 = C, slots 0..C
    aa.q = m->WS<char>(y.q) + (size_t)y.C * y.HD * 4;  // 4 bytes per activation value
    aa.q_pitch = (y.C + 1) * y.HD;
    aa.R = B;
    aa.rm = r1;
    R = B;
    x = xc;
  }
  if (last_row) {
    // The prompt's last chunk at the last base layer: every row's K and V are
    // appended, but the outputs are read only at the last row (the first
    // decision and the context rows), so attention (split over that row's
    // slots) and tail run on it alone
    if (!prefill || rm.mode != ROWS_PREFILL) return fail(HAM_EINVAL, "last-row prefill layer");
    RowMap r1 = rm;
    r1.t0 = rm.t0 + R - 1;
    aa.q = m->WS<char>(y.q) + (size_t)(R - 1) * y.HD * 4;  // 4 bytes per activation value
    aa.R = 1;
    aa.rm = r1;
    aa.nsplit = attn_splits_for(dt, 1, y.Hk, r1.t0 + 1);
    if (launch_attn_decode(dt, aa, s) != 0) return fail(HAM_EINVAL, "attention shape");
    return layer_tail(m, j, 1, x + (size_t)(R - 1) * y.d, split, gate, gate_n, pend, gk);
  }
  m->pbegin(base ? HAM_PROF_ATTN : -1, (double)kv_visible * y.Hk * y.hd * 2 * y.es);
  const int arc = prefill ? launch_attn_prefill(dt, aa, s) : launch_attn_decode(dt, aa, s);
  m->pend();
  if (arc != 0) return fail(HAM_EINVAL, "attention shape");
  return layer_tail(m, j, R, x, split, gate, gate_n, pend, gk);
}

// final norm of one row per sequence (folding in pending partials, capturing the
// last context row) + LM head with per-tile argmax and stop logit, then the
// decision and stop test (decision k)
int run_decision(ham_model* m, int k, float* x, int row_stride, int row_off, const float* g, Pending& pend,
                 float* ctx_last, int* out_tokens, int* out_lens) {
  const Layout& y = m->y;
  const int B = m->batch;
  float* hid = m->dbg ? m->dbg + (size_t)4 * y.B * y.V + ((size_t)k * y.B) * y.d : nullptr;
  if (norm_rows(m, x, B, row_stride, row_off, g, pend, ctx_last, y.C * y.d, hid, m->sp.active, B)) return HAM_EINVAL;

  GemmArgs ga{};
  ga.W = m->W<char>(y.Wlm); ga.N = y.Vpad; ga.K = y.d; ga.X = m->WS<char>(y.xn); ga.ldx = y.d; ga.M = B;
  ga.gate = m->sp.active; ga.gate_n = B;
  DecideArgs& d = ga.dec;
  d.st = m->sp; d.B = B; d.k = k; d.mode = m->cfg.stop_mode; d.stop_id = m->cfg.stop_id; d.G = y.G; d.V = y.V;
  d.tau = m->tau; d.out_tokens = out_tokens; d.out_lens = out_lens; d.has_teacher = m->has_teacher;
  d.dbg_logits = m->dbg ? m->dbg + (size_t)k * y.B * y.V : nullptr;
  d.dbg_stop = m->dbg ? m->dbg + (size_t)4 * y.B * y.V + (size_t)4 * y.B * y.d + (size_t)k * y.B : nullptr;
  d.stop_buf = m->WS<float>(y.stopb); d.best_val = m->WS<float>(y.bval); d.best_idx = m->WS<int>(y.bidx);
  d.ntiles = skinny_tiles(y.Vpad);
  // the next micro step's input rows, written by the same launch (the micro
  // decoder's rows start in the first residual buffer)
  d.prep_k = k + 1 < y.G ? k + 1 : 0; d.C = y.C; d.d = y.d;
  d.ctx = m->WS<float>(y.ctx); d.E = m->W<char>(y.E); d.x = m->WS<float>(y.x);
  int ns = 1;
  if (gemm_p(m, EPI_ARGMAX, ga, 1, k == 0 ? HAM_PROF_HEAD0 : HAM_PROF_HEADK, &ns))
    return fail(HAM_EINVAL, "lm head shape");
  if (launch_decide(dtype_of(m), d, skinny_tiles(y.Vpad), B, m->s)) return fail(HAM_EINVAL, "decision shape");
  return HAM_OK;
}

// decision k = 0 from the base model, then the micro steps (all gated on device)
int decode_tail(ham_model* m, Pending& pend, float* ctx_last, float* xres, int* out_tokens, int* out_lens) {
  const Layout& y = m->y;
  const int dt = dtype_of(m);
  const int B = m->batch;
  int rc = run_decision(m, 0, xres, 1, 0, m->W<float>(y.gf), pend, ctx_last, out_tokens, out_lens);
  if (rc) return rc;
  const long long lsb = (long long)y.Hk * LOCAL_SLOTS * y.hd, lsh = (long long)LOCAL_SLOTS * y.hd;
  for (int k = 1; k < y.G; ++k) {
    float* x = m->WS<float>(y.x);  // written by decision k - 1
    RowMap rm{};
    rm.mode = k == 1 ? ROWS_MICRO1 : ROWS_MICROK; rm.C = y.C; rm.k = k; rm.st = m->sp;
    const int R = k == 1 ? B * (y.C + 1) : B;
    Pending mp_pend;
    // micro step k >= 2: one new local slot per sequence at local position C + k - 1
    const int lpos = y.C + k - 1, half = y.hd / 2;
    const StepAttn lstep{m->W<float>(y.cos_t) + (size_t)lpos * half, m->W<float>(y.sin_t) + (size_t)lpos * half, 0,
                         lpos};
    const bool last_rows = k == 1 && R > LAST_ROWS_MIN;
    for (int mj = 0; mj < y.M; ++mj) {
      const float* g_next = mj + 1 < y.M ? m->W<float>(y.g1[y.L + mj + 1]) : nullptr;
      rc = run_layer(m, y.L + mj, R, rm, x, false, m->WS<char>(y.Kloc + mj * y.loc_layer),
                     m->WS<char>(y.VTloc + mj * y.loc_layer), lsb, lsh, LOCAL_SLOTS, 1, m->sp.active, B, mp_pend,
                     nullptr, 0, k == 1 ? B * (y.C + 1) * (y.C + 2) / 2 : B * (y.C + k), k == 1 ? nullptr : &lstep,
                     g_next, nullptr, last_rows && mj == y.M - 1);
      if (rc) return rc;
    }
    // micro step 1 leaves C + 1 rows per sequence (the last is the decision's),
    // or only that row where its last layer ran on it alone
    const bool all_rows = k == 1 && !last_rows;
    rc = run_decision(m, k, x, all_rows ? y.C + 1 : 1, all_rows ? y.C : 0, m->W<float>(y.gmf), mp_pend, nullptr,
                      out_tokens, out_lens);
    if (rc) return rc;
  }
  return HAM_OK;
}

// slot splits across workgroups: none while every wave of a workgroup gets at
// most a few key blocks; otherwise enough to give about 4096 waves in total
int attn_splits_for(int dtype, int R, int Hk, int kv_max) {
  const int kb = dtype == HAM_BF16 ? 32 : 16;
  const int blocks = (kv_max + kb - 1) / kb;
  if (blocks <= 8 * 8) return 1;  // 8 waves x at most 8 blocks each
  const int wgs = R * Hk;
  int want = (4096 / 8 + wgs - 1) / wgs;
  const int most = std::max(1, blocks / (8 * 2));  // at least 2 blocks per wave
  return std::max(1, std::min(std::min(want, most), MAX_ATTN_SPLIT));
}

size_t attn_part_bytes(int R, int H, int Hk, int hd) {
  return (size_t)R * Hk * MAX_ATTN_SPLIT * (H / Hk) * (hd + 2) * 4;
}

}  // namespace

// ============================================================================ C ABI
extern "C" {

const char* ham_last_error(void) { return g_err.c_str(); }

size_t ham_weights_bytes(const ham_config* c) { return check_cfg(c) ? 0 : make_layout(c).w_bytes; }
size_t ham_state_bytes(const ham_config* c) { return check_cfg(c) ? 0 : make_layout(c).st_bytes; }
size_t ham_workspace_bytes(const ham_config* c) { return check_cfg(c) ? 0 : make_layout(c).ws_bytes; }

int ham_state_info(const ham_config* c, int32_t layer, size_t* k_offset, size_t* v_offset, int32_t* slots) {
  if (!k_offset || !v_offset || !slots) return fail(HAM_EINVAL, "null output");
  if (const char* e = check_cfg(c)) return fail(HAM_EINVAL, "%s", e);
  const Layout y = make_layout(c);
  if (layer < 0 || layer >= y.L) return fail(HAM_EINVAL, "layer %d out of range", layer);
  *k_offset = y.Kc + (size_t)layer * y.kv_layer;
  *v_offset = y.VTc + (size_t)layer * y.kv_layer;
  *slots = y.S;
  return HAM_OK;
}

int ham_tensor_info(const ham_config* c, int32_t id, size_t* offset, int32_t* rows, int32_t* cols,
                    int32_t* row_off, int32_t* mat_rows, int32_t* interleave, int32_t* tiled) {
  if (const char* e = check_cfg(c)) return fail(HAM_EINVAL, "%s", e);
  if (!offset || !rows || !cols || !row_off || !mat_rows || !interleave || !tiled)
    return fail(HAM_EINVAL, "null output pointer");
  const Layout y = make_layout(c);
  *interleave = 0;
  *row_off = 0;
  *tiled = 1;
  auto set = [&](size_t off, int r, int cl, int roff, int mrows) {
    *offset = off; *rows = r; *cols = cl; *row_off = roff; *mat_rows = mrows;
  };
  switch (id) {
    case 0: set(y.E, y.V, y.d, 0, y.V); *tiled = 0; return HAM_OK;
    case 1: set(y.Pe, 4, y.d, 0, 4); *tiled = 0; return HAM_OK;
    case 2: case 3: case 4: set(y.Aqkv, y.HD, y.d, (id - 2) * y.HD, 3 * y.HD); return HAM_OK;
    case 5: set(y.Ao, y.d, y.HD, 0, y.d); return HAM_OK;
    case 6: set(y.Alin, y.d, y.d, 0, y.d); return HAM_OK;
    case 7: set(y.Wlm, y.V, y.d, 0, y.Vpad); return HAM_OK;
    case 8: set(y.Wlm, 1, y.d, y.V, y.Vpad); return HAM_OK;
    default: break;
  }
  if (id < 16) return fail(HAM_EINVAL, "unknown tensor id %d", id);
  const int j = (id - 16) / 8, t = (id - 16) % 8;
  if (j >= y.L + y.M || t > 6) return fail(HAM_EINVAL, "unknown tensor id %d", id);
  const int kvd = y.Hk * y.hd;
  switch (t) {
    case 0: set(y.Wqkv[j], y.HD, y.d, 0, y.QKV); break;
    case 1: set(y.Wqkv[j], kvd, y.d, y.HD, y.QKV); break;
    case 2: set(y.Wqkv[j], kvd, y.d, y.HD + kvd, y.QKV); break;
    case 3: set(y.Wo[j], y.d, y.HD, 0, y.d); break;
    case 4: set(y.Wgu[j], y.F, y.d, 0, 2 * y.F); *interleave = 1; break;
    case 5: set(y.Wgu[j], y.F, y.d, 0, 2 * y.F); *interleave = 2; break;
    case 6: set(y.Wd[j], y.d, y.F, 0, y.d); break;
  }
  return HAM_OK;
}

int ham_init_weights(const ham_config* c, uint64_t seed, void* d_weights, size_t weights_bytes, void* d_state,
                     size_t state_bytes, void* d_workspace, size_t workspace_bytes, void* hip_stream,
                     ham_model** out) {
  if (!out) return fail(HAM_EINVAL, "null output handle");
  *out = nullptr;
  if (const char* e = check_cfg(c)) return fail(HAM_EINVAL, "%s", e);
  if (!d_weights || !d_state || !d_workspace) return fail(HAM_EINVAL, "null buffer");
  const Layout y = make_layout(c);
  if (weights_bytes < y.w_bytes || state_bytes < y.st_bytes || workspace_bytes < y.ws_bytes)
    return fail(HAM_ENOMEM, "buffers too small (need %zu / %zu / %zu bytes)", y.w_bytes, y.st_bytes, y.ws_bytes);
  if (((uintptr_t)d_weights | (uintptr_t)d_state | (uintptr_t)d_workspace) & 255)
    return fail(HAM_EINVAL, "buffers must be 256-byte aligned");
  ham_model* m = new ham_model();
  m->cfg = *c;
  m->y = y;
  m->w = (char*)d_weights;
  m->st = (char*)d_state;
  m->ws = (char*)d_workspace;
  m->s = (hipStream_t)hip_stream;
  m->sp = seq_ptrs(m->st, y);
  const double cf = c->stop_conf;
  m->tau = cf <= 0.0 ? INFINITY : (cf >= 1.0 ? -INFINITY : (float)std::log((1.0 - cf) / cf));
  const int dt = c->dtype;
  hipStream_t s = m->s;
  auto bad = [&](int rc) { delete m; return rc; };
#define INIT_TRY(call)                                                                      \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess) return bad(fail(HAM_EHIP, "%s: %s", #call, hipGetErrorString(e_))); \
  } while (0)
  INIT_TRY(hipMemsetAsync(d_weights, 0, y.w_bytes, s));
  INIT_TRY(hipMemsetAsync(d_state, 0, y.st_bytes, s));
  INIT_TRY(hipMemsetAsync(d_workspace, 0, y.ws_bytes, s));
  // every GEMM weight matrix is stored fragment-tiled; E and P (row gathers) row-major
  auto gen = [&](size_t off, int rows, int cols, long long row_off, int inter, int tid, int tiled = 1) {
    GenArgs g{};
    g.dst = m->w + off; g.rows = rows; g.cols = cols; g.row_off = row_off; g.interleave = inter;
    g.tiled = tiled; g.key = sm64(seed, (uint64_t)tid);
    launch_gen_normal(dt, g, s);
  };
  gen(y.E, y.V, y.d, 0, 0, 0, 0);
  gen(y.Pe, 4, y.d, 0, 0, 1, 0);
  for (int i = 0; i < 3; ++i) gen(y.Aqkv, y.HD, y.d, (long long)i * y.HD, 0, 2 + i);
  gen(y.Ao, y.d, y.HD, 0, 0, 5);
  gen(y.Alin, y.d, y.d, 0, 0, 6);
  gen(y.Wlm, y.V, y.d, 0, 0, 7);
  gen(y.Wlm, 1, y.d, y.V, 0, 8);
  for (int j = 0; j < y.L + y.M; ++j) {
    const int base = 16 + 8 * j;
    gen(y.Wqkv[j], y.HD, y.d, 0, 0, base + 0);
    gen(y.Wqkv[j], y.Hk * y.hd, y.d, y.HD, 0, base + 1);
    gen(y.Wqkv[j], y.Hk * y.hd, y.d, y.HD + y.Hk * y.hd, 0, base + 2);
    gen(y.Wo[j], y.d, y.HD, 0, 0, base + 3);
    gen(y.Wgu[j], y.F, y.d, 0, 1, base + 4);
    gen(y.Wgu[j], y.F, y.d, 0, 2, base + 5);
    gen(y.Wd[j], y.d, y.F, 0, 0, base + 6);
    launch_fill_f32(m->W<float>(y.g1[j]), y.d, 1.0f, s);
    launch_fill_f32(m->W<float>(y.g2[j]), y.d, 1.0f, s);
  }
  launch_fill_f32(m->W<float>(y.gf), y.d, 1.0f, s);
  launch_fill_f32(m->W<float>(y.gmf), y.d, 1.0f, s);
  INIT_TRY(hipGetLastError());
  // RoPE tables: angle p * theta^(-2i/hd) in float64, cos/sin rounded to fp32
  const int half = y.hd / 2;
  std::vector<float> ct((size_t)y.max_pos * half), stt((size_t)y.max_pos * half);
  for (int i = 0; i < half; ++i) {
    const double inv = std::pow((double)c->rope_theta, -2.0 * i / (double)y.hd);
    for (int p = 0; p < y.max_pos; ++p) {
      const double a = (double)p * inv;
      ct[(size_t)p * half + i] = (float)std::cos(a);
      stt[(size_t)p * half + i] = (float)std::sin(a);
    }
  }
  INIT_TRY(hipMemcpyAsync(m->w + y.cos_t, ct.data(), ct.size() * 4, hipMemcpyHostToDevice, s));
  INIT_TRY(hipMemcpyAsync(m->w + y.sin_t, stt.data(), stt.size() * 4, hipMemcpyHostToDevice, s));
  INIT_TRY(hipStreamSynchronize(s));
#undef INIT_TRY
  *out = m;
  return HAM_OK;
}

}  // extern "C"

namespace {

// Prefill of `batch` sequences of T base inputs each: prompt token ids (gathered
// from E, positions 0..T-1), or caller-given fp32 input vectors at caller-given
// positions.  One KV slot per input, then the first decision and micro loop.
int prefill_common(ham_model* m, int32_t batch, int32_t T, const int32_t* d_prompt, const float* d_embeds,
                   const int32_t* d_positions, const int32_t* h_max_new, const int32_t* d_forced_lens,
                   const int32_t* d_teacher, int32_t* d_out_tokens, int32_t* d_out_lens) {
  const Layout& y = m->y;
  const bool forced_mode = m->cfg.stop_mode == HAM_STOP_FORCED || m->cfg.stop_mode == HAM_STOP_FORCED_TOKEN;
  if (forced_mode && !d_forced_lens) return fail(HAM_EINVAL, "FORCED mode needs forced lengths");
  if (d_teacher && !forced_mode) return fail(HAM_EINVAL, "teacher forcing needs FORCED mode");
  for (int b = 0; b < batch; ++b)
    if (h_max_new[b] < 0) return fail(HAM_EINVAL, "negative budget");
  const int dt = dtype_of(m);
  hipStream_t s = m->s;
  m->batch = batch;
  m->prompt_len = T;
  m->steps_done = -1;
  m->has_teacher = d_teacher != nullptr;
  // budgets are read by kernels of earlier calls: let those finish, then copy synchronously
  HIP_TRY(hipStreamSynchronize(s));
  HIP_TRY(hipMemcpy(m->sp.budget, h_max_new, sizeof(int32_t) * batch, hipMemcpyHostToDevice));
  PrefillArgs pa{};
  pa.st = m->sp; pa.B = batch; pa.P = T; pa.G = y.G; pa.forced_in = d_forced_lens;
  pa.pos_in = d_positions; pa.ldpos = T;
  pa.teacher_in = d_teacher; pa.out_tokens = d_out_tokens; pa.out_lens = d_out_lens;
  launch_prefill_begin(pa, s);
  float* xp = m->WS<float>(y.xp);
  float* x = m->WS<float>(y.x);
  float* ctx = m->WS<float>(y.ctx);
  const long long sb = (long long)y.Hk * y.S * y.hd, sh = (long long)y.S * y.hd;
  for (int b = 0; b < batch; ++b) {
    for (int t0 = 0; t0 < T; t0 += y.Tc) {
      const int R = std::min(y.Tc, T - t0);
      const bool last = t0 + R == T;
      GatherArgs g{};
      if (d_embeds) g.rows = d_embeds + ((size_t)b * T + t0) * y.d;
      else g.ids = d_prompt + (size_t)b * T + t0;
      g.R = R; g.E = m->W<char>(y.E); g.d = y.d; g.V = y.V;
      g.x = xp; g.ldx = y.d; g.err = m->sp.err + b;
      launch_gather_rows(dt, g, s);
      RowMap rm{};
      rm.mode = ROWS_PREFILL; rm.b = b; rm.t0 = t0; rm.pos = d_positions; rm.ldpos = T; rm.st = m->sp;
      for (int l = 0; l < y.L; ++l) {
        Pending none;
        // the last layer's outputs are read only at the prompt's last row (the
        // decision and the context rows): earlier chunks append its K and V
        // only, the last chunk runs attention and tail on that row alone
        const bool kv_only = !last && l == y.L - 1;
        const bool last_row = last && l == y.L - 1 && R > 1;
        int rc = run_layer(m, l, R, rm, xp, true, m->st + y.Kc + l * y.kv_layer, m->st + y.VTc + l * y.kv_layer,
                           sb, sh, y.S, 1, nullptr, 0, none, nullptr, 0, 0, nullptr, nullptr, nullptr, false, kv_only,
                           last_row);
        if (rc) return rc;
        if (last)
          for (int c = 0; c < y.C; ++c)
            if (y.ctx_l[c] == l + 1)
              launch_copy_row(xp + (size_t)(R - 1) * y.d, ctx + ((size_t)b * y.C + c) * y.d, y.d, s);
      }
      if (last) launch_copy_row(xp + (size_t)(R - 1) * y.d, x + (size_t)b * y.d, y.d, s);
    }
  }
  Pending none;
  int rc = decode_tail(m, none, nullptr, x, d_out_tokens, d_out_lens);
  if (rc) return rc;
  HIP_TRY(hipGetLastError());
  m->steps_done = 0;
  return HAM_OK;
}

}  // namespace

extern "C" {

int ham_prefill(ham_model* m, int32_t batch, const int32_t* d_prompt, int32_t prompt_len, const int32_t* h_max_new,
                const int32_t* d_forced_lens, const int32_t* d_teacher, int32_t* d_out_tokens, int32_t* d_out_lens) {
  if (!m) return fail(HAM_EINVAL, "null model");
  const Layout& y = m->y;
  if (batch < 1 || prompt_len < 1 || !d_prompt || !h_max_new || !d_out_tokens || !d_out_lens)
    return fail(HAM_EINVAL, "bad prefill arguments");
  if (batch > y.B || prompt_len > y.P)
    return fail(HAM_ECAP, "batch %d / prompt %d exceed capacity %d / %d", batch, prompt_len, y.B, y.P);
  return prefill_common(m, batch, prompt_len, d_prompt, nullptr, nullptr, h_max_new, d_forced_lens, d_teacher,
                        d_out_tokens, d_out_lens);
}

int ham_prefill_embeds(ham_model* m, int32_t batch, const float* d_embeds, const int32_t* d_positions,
                       int32_t n_inputs, const int32_t* h_max_new, const int32_t* d_forced_lens,
                       const int32_t* d_teacher, int32_t* d_out_tokens, int32_t* d_out_lens) {
  if (!m) return fail(HAM_EINVAL, "null model");
  const Layout& y = m->y;
  if (batch < 1 || n_inputs < 1 || !d_embeds || !d_positions || !h_max_new || !d_out_tokens || !d_out_lens)
    return fail(HAM_EINVAL, "bad prefill arguments");
  if (batch > y.B || n_inputs > y.P + y.steps)
    return fail(HAM_ECAP, "batch %d / inputs %d exceed capacity %d / %d", batch, n_inputs, y.B, y.P + y.steps);
  return prefill_common(m, batch, n_inputs, nullptr, d_embeds, d_positions, h_max_new, d_forced_lens, d_teacher,
                        d_out_tokens, d_out_lens);
}

}  // extern "C"

namespace {

// Everything of a macro-step after k_macro_begin: the embedder, the base
// forward writing one KV slot per running sequence, the decisions and the
// micro loop.  Launch arguments depend only on the batch, the prompt length,
// the output pointers, the debug buffer and teacher forcing.
int macro_step_body(ham_model* m, int32_t* d_out_tokens, int32_t* d_out_lens) {
  const Layout& y = m->y;
  const int dt = dtype_of(m);
  hipStream_t s = m->s;
  const int B = m->batch;
  float* x = m->WS<float>(y.x);
  // compositional embedder (Sec. 3.2), skipped on device unless some group has > 1 token
  GemmArgs ga{};
  ga.part = m->WS<float>(y.part); ga.gate = m->sp.fused; ga.gate_n = B;
  ga.W = m->W<char>(y.Aqkv); ga.N = 3 * y.HD; ga.K = y.d; ga.X = m->WS<char>(y.emb_in); ga.ldx = y.d;
  ga.M = 5 * B; ga.out = m->WS<float>(y.qkv); ga.ldo = 3 * y.HD;
  int ns = 1;
  if (gemm_p(m, EPI_F32, ga, MAX_GEMM_SPLIT, HAM_PROF_EMBED, &ns)) return fail(HAM_EINVAL, "embedder gemm shape");
  EmbedAttnArgs ea{};
  ea.proj = m->WS<float>(y.qkv); ea.fused = m->sp.fused; ea.B = B; ea.H = y.H; ea.d = y.d; ea.hd = y.hd;
  ea.part = ns > 1 ? m->WS<float>(y.part) : nullptr; ea.nsplit = ns;
  ea.out = m->WS<char>(y.emb_o);
  launch_embed_attn(dt, ea, s);
  // the embedder's two output projections run unsplit: a split would need a
  // reduce launch, which costs about as much as the slower GEMM even when no
  // group is fused and the whole chain is gated off
  ga.W = m->W<char>(y.Ao); ga.N = y.d; ga.K = y.HD; ga.X = m->WS<char>(y.emb_o); ga.ldx = y.HD; ga.M = B;
  ga.out = m->WS<char>(y.emb_y); ga.ldo = y.d;
  if (gemm_p(m, EPI_OP, ga, 1, HAM_PROF_EMBED, &ns)) return fail(HAM_EINVAL, "embedder gemm shape");
  if (ns > 1) {
    ga.nsplit = ns;
    if (launch_split_reduce(dt, EPI_OP, ga, s)) return fail(HAM_EINVAL, "split reduce shape");
  }
  ga.W = m->W<char>(y.Alin); ga.N = y.d; ga.K = y.d; ga.X = m->WS<char>(y.emb_y); ga.ldx = y.d;
  ga.out = x; ga.ldo = y.d; ga.rowmask = m->sp.fused;
  if (gemm_p(m, EPI_XMASK, ga, 1, HAM_PROF_EMBED, &ns)) return fail(HAM_EINVAL, "embedder gemm shape");
  if (ns > 1) {
    ga.nsplit = ns;
    if (launch_split_reduce(dt, EPI_XMASK, ga, s)) return fail(HAM_EINVAL, "split reduce shape");
  }

  // base forward: one new KV slot per running sequence
  RowMap rm{};
  rm.mode = ROWS_DECODE; rm.st = m->sp;
  const long long sb = (long long)y.Hk * y.S * y.hd, sh = (long long)y.S * y.hd;
  // the attention launch is sized for the most slots any step of this generation
  // can hold, so every macro-step launches the same kernels with the same
  // arguments (graph replay); each row attends over its own device-side length
  const int kv_cap = std::min(m->prompt_len + y.steps - 1, y.S - 1);
  const int nsplit = macro_attn_splits(dt, B, y.Hk, y.hd, kv_cap);
  const StepAttn bstep{m->WS<float>(y.rope_cs), m->WS<float>(y.rope_cs) + y.hd / 2, y.hd, kv_cap};
  float* ctx = m->WS<float>(y.ctx);
  Pending pend;
  float* ctx_prev = nullptr;  // context slot of the previous layer's output, captured by the next norm
  for (int l = 0; l < y.L; ++l) {
    float* ctx_out = nullptr;  // context slot of this layer's output
    for (int c = 0; c < y.C; ++c)
      if (y.ctx_l[c] == l + 1) ctx_out = ctx + (size_t)c * y.d;
    const float* g_next = l + 1 < y.L ? m->W<float>(y.g1[l + 1]) : nullptr;
    int rc = run_layer(m, l, B, rm, x, false, m->st + y.Kc + l * y.kv_layer, m->st + y.VTc + l * y.kv_layer, sb,
                       sh, y.S, nsplit, m->sp.step_on, B, pend, ctx_prev, y.C * y.d, m->kv_visible, &bstep, g_next,
                       ctx_out);
    if (rc) return rc;
    ctx_prev = ctx_out;
  }
  int rc = decode_tail(m, pend, ctx_prev, x, d_out_tokens, d_out_lens);
  if (rc) return rc;
  HIP_TRY(hipGetLastError());
  return HAM_OK;
}

}  // namespace

extern "C" {

int ham_macro_step(ham_model* m, const int32_t* d_forced_lens, const int32_t* d_teacher, int32_t* d_out_tokens,
                   int32_t* d_out_lens) {
  if (!m) return fail(HAM_EINVAL, "null model");
  if (m->steps_done < 0) return fail(HAM_ESTATE, "ham_macro_step before ham_prefill");
  if (!d_out_tokens || !d_out_lens) return fail(HAM_EINVAL, "null output");
  const Layout& y = m->y;
  if (m->steps_done >= y.steps) return fail(HAM_ECAP, "max_steps (%d) reached", y.steps);
  if (m->prompt_len + m->steps_done + 1 > y.S)
    return fail(HAM_ECAP, "KV slot capacity (%d) reached", y.S);
  const bool forced_mode = m->cfg.stop_mode == HAM_STOP_FORCED || m->cfg.stop_mode == HAM_STOP_FORCED_TOKEN;
  if (forced_mode && !d_forced_lens) return fail(HAM_EINVAL, "FORCED mode needs forced lengths");
  if (d_teacher && !forced_mode) return fail(HAM_EINVAL, "teacher forcing needs FORCED mode");
  const int dt = dtype_of(m);
  hipStream_t s = m->s;
  const int B = m->batch;
  m->has_teacher = d_teacher != nullptr;
  float* x = m->WS<float>(y.x);
  MacroArgs ma{};
  ma.st = m->sp; ma.B = B; ma.d = y.d; ma.G = y.G; ma.E = m->W<char>(y.E); ma.P = m->W<char>(y.Pe); ma.x = x;
  ma.ldx = y.d; ma.emb_in = m->WS<char>(y.emb_in); ma.forced_in = d_forced_lens; ma.teacher_in = d_teacher;
  ma.out_tokens = d_out_tokens; ma.out_lens = d_out_lens;
  ma.cos_t = m->W<float>(y.cos_t); ma.sin_t = m->W<float>(y.sin_t); ma.max_pos = y.max_pos; ma.hd = y.hd;
  ma.rope_cs = m->WS<float>(y.rope_cs);
  launch_macro_begin(dt, ma, s);
  m->kv_visible = B * (m->prompt_len + m->steps_done + 1);  // slots attended this step (profiling bytes)

  if (m->use_graph && !m->prof_on) {
    const ham_model::GraphKey key{B, m->prompt_len, m->has_teacher, d_out_tokens, d_out_lens, m->dbg};
    if (!(m->gexec && m->gkey == key)) {
      m->drop_graph();
      hipGraph_t g = nullptr;
      // captured on a private stream (the caller's may be the legacy default
      // stream, which cannot be captured), launched on the caller's stream
      if (!m->cap_stream && hipStreamCreateWithFlags(&m->cap_stream, hipStreamNonBlocking) != hipSuccess)
        m->cap_stream = nullptr;
      if (m->cap_stream && hipStreamBeginCapture(m->cap_stream, hipStreamCaptureModeThreadLocal) == hipSuccess) {
        m->s = m->cap_stream;
        const int rc = macro_step_body(m, d_out_tokens, d_out_lens);
        m->s = s;
        const hipError_t ec = hipStreamEndCapture(m->cap_stream, &g);
        if (rc) {
          if (g) hipGraphDestroy(g);
          return rc;
        }
        if (ec == hipSuccess && g && hipGraphInstantiate(&m->gexec, g, nullptr, nullptr, 0) == hipSuccess) {
          m->graph = g;
          m->gkey = key;
        } else {
          if (g) hipGraphDestroy(g);
          m->gexec = nullptr;
          m->use_graph = false;  // capture unavailable: launch on the stream from now on
          (void)hipGetLastError();
        }
      } else {
        m->use_graph = false;
        (void)hipGetLastError();
      }
    }
    if (m->gexec) {
      HIP_TRY(hipGraphLaunch(m->gexec, s));
      m->steps_done += 1;
      return HAM_OK;
    }
  }
  const int rc = macro_step_body(m, d_out_tokens, d_out_lens);
  if (rc) return rc;
  m->steps_done += 1;
  return HAM_OK;
}

int ham_kv_stats(ham_model* m, ham_kv_stats_t* h_out) {
  if (!m || !h_out) return fail(HAM_EINVAL, "null argument");
  if (m->steps_done < 0) return fail(HAM_ESTATE, "ham_kv_stats before ham_prefill");
  HIP_TRY(hipStreamSynchronize(m->s));
  const int B = m->batch;
  std::vector<int> kv(B), em(B), gr(B), dn(B), hist(5 * B), err(B);
  HIP_TRY(hipMemcpy(kv.data(), m->sp.kv_len, 4 * B, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(em.data(), m->sp.emitted, 4 * B, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(gr.data(), m->sp.groups, 4 * B, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(dn.data(), m->sp.done, 4 * B, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(hist.data(), m->sp.hist, 20 * B, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(err.data(), m->sp.err, 4 * B, hipMemcpyDeviceToHost));
  for (int b = 0; b < B; ++b) {
    ham_kv_stats_t& o = h_out[b];
    o.kv_len = kv[b];
    o.prompt_slots = m->prompt_len;
    o.gen_slots = kv[b] - m->prompt_len;
    o.tokens = em[b];
    o.groups = gr[b];
    o.done = dn[b];
    for (int j = 0; j < 5; ++j) o.len_hist[j] = hist[5 * b + j];
    o.device_error = err[b];
  }
  return HAM_OK;
}

int ham_set_debug(ham_model* m, void* d_buf, size_t bytes) {
  if (!m) return fail(HAM_EINVAL, "null model");
  const Layout& y = m->y;
  if (d_buf && bytes < (size_t)4 * y.B * (y.V + y.d + 1) * 4) return fail(HAM_ENOMEM, "debug buffer too small");
  m->dbg = (float*)d_buf;
  return HAM_OK;
}

int ham_steps_done(const ham_model* m) { return m ? m->steps_done : -1; }

int ham_state_save(ham_model* m, void* d_dst, size_t bytes) {
  if (!m || !d_dst) return fail(HAM_EINVAL, "null argument");
  if (m->steps_done < 0) return fail(HAM_ESTATE, "ham_state_save before ham_prefill");
  if (bytes < m->y.st_bytes) return fail(HAM_ENOMEM, "state copy needs %zu bytes", m->y.st_bytes);
  HIP_TRY(hipMemcpyAsync(d_dst, m->st, m->y.st_bytes, hipMemcpyDeviceToDevice, m->s));
  m->saved_batch = m->batch;
  m->saved_prompt = m->prompt_len;
  m->saved_steps = m->steps_done;
  m->saved_teacher = m->has_teacher;
  return HAM_OK;
}

int ham_state_restore(ham_model* m, const void* d_src, size_t bytes) {
  if (!m || !d_src) return fail(HAM_EINVAL, "null argument");
  if (m->saved_steps < 0) return fail(HAM_ESTATE, "ham_state_restore before ham_state_save");
  if (bytes < m->y.st_bytes) return fail(HAM_ENOMEM, "state copy needs %zu bytes", m->y.st_bytes);
  HIP_TRY(hipMemcpyAsync(m->st, d_src, m->y.st_bytes, hipMemcpyDeviceToDevice, m->s));
  m->batch = m->saved_batch;
  m->prompt_len = m->saved_prompt;
  m->steps_done = m->saved_steps;
  m->has_teacher = m->saved_teacher;
  return HAM_OK;
}

int ham_set_graph(ham_model* m, int enable) {
  if (!m) return fail(HAM_EINVAL, "null model");
  m->drop_graph();
  m->use_graph = enable != 0;
  return HAM_OK;
}

int ham_profile(ham_model* m, int enable) {
  if (!m) return fail(HAM_EINVAL, "null model");
  if (enable) {
    m->recs.clear();
    m->pool_used = 0;
  }
  m->prof_on = enable != 0;
  return HAM_OK;
}

int ham_profile_read(ham_model* m, ham_prof_t* out, int n) {
  if (!m || !out || n < 0) return fail(HAM_EINVAL, "bad arguments");
  HIP_TRY(hipStreamSynchronize(m->s));
  for (int k = 0; k < n; ++k) out[k] = ham_prof_t{0, 0.0, 0.0};
  for (const auto& r : m->recs) {
    if (r.kind < 0 || r.kind >= n) continue;
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, r.a, r.b));
    out[r.kind].launches += 1;
    out[r.kind].ms += ms;
    out[r.kind].bytes += r.bytes;
  }
  return HAM_OK;
}

void ham_destroy(ham_model* m) { delete m; }

size_t ham_op_attention_workspace_bytes(int32_t rows, int32_t H, int32_t Hk, int32_t hd) {
  if (rows < 1 || H < 1 || Hk < 1 || H % Hk) return 0;
  return al(attn_part_bytes(rows, H, Hk, hd));
}

int ham_op_decode_attention(int32_t dtype, int32_t rows, int32_t H, int32_t Hk, int32_t hd, int32_t S,
                            const void* d_q, const void* d_k, const void* d_vt, const int32_t* d_kv_len,
                            const int32_t* d_enable, int32_t kv_max, void* d_out, void* d_ws, size_t ws_bytes,
                            void* stream) {
  if (dtype != HAM_F32 && dtype != HAM_BF16) return fail(HAM_EINVAL, "bad dtype");
  if (rows < 1 || H < 1 || Hk < 1 || H % Hk || H / Hk > 4 || (hd != 64 && hd != 128) || S < 64 || S % 64)
    return fail(HAM_EINVAL, "bad attention shape");
  if (kv_max < 0 || kv_max > S) return fail(HAM_EINVAL, "kv_max out of range");
  if (!d_q || !d_k || !d_vt || !d_kv_len || !d_enable || !d_out || !d_ws) return fail(HAM_EINVAL, "null pointer");
  if (ws_bytes < attn_part_bytes(rows, H, Hk, hd)) return fail(HAM_ENOMEM, "workspace too small");
  SeqPtrs sp{};
  sp.kv_len = const_cast<int*>(d_kv_len);
  sp.step_on = const_cast<int*>(d_enable);
  sp.cur_slot = sp.kv_len;  // read by the row map, unused by attention
  sp.cur_pos = sp.kv_len;
  AttnArgs aa{};
  aa.q = d_q; aa.ldq = H * hd; aa.K = d_k; aa.VT = d_vt; aa.sb = (long long)Hk * S * hd;
  aa.sh = (long long)S * hd; aa.S = S; aa.H = H; aa.Hkv = Hk; aa.hd = hd; aa.R = rows;
  aa.nsplit = attn_splits_for(dtype, rows, Hk, std::max(kv_max, 1));
  aa.o = d_out; aa.ldo = H * hd; aa.part = (float*)d_ws;
  aa.rm.mode = ROWS_DECODE; aa.rm.st = sp;
  if (launch_attn_decode(dtype, aa, (hipStream_t)stream)) return fail(HAM_EINVAL, "attention shape");
  HIP_TRY(hipGetLastError());
  return HAM_OK;
}

}  // extern "C"

namespace {

// Scratch of ham_op_attention_step_noalloc: the split records of the attention
// step, at most NOALLOC_SCRATCH bytes, one copy per GPU for the life of the
// process.  Host code reaches it only through the device address that
// hipGetSymbolAddress returns for the current device (noalloc_scratch).
constexpr size_t NOALLOC_SCRATCH = size_t(4) << 20;
__device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH];

std::mutex g_scratch_mu;
constexpr int MAX_DEVICES = 64;
void* g_scratch_dev[MAX_DEVICES] = {};

int noalloc_scratch(void** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(HAM_EINVAL, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(HAM_EHIP, "no device address for the scratch array");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return HAM_OK;
}

// split-record bytes of one fused attention step launch (nothing when unsplit)
size_t attn_step_record_bytes(int rows, int H, int Hk, int hd, int nsplit) {
  return nsplit > 1 ? (size_t)rows * Hk * nsplit * (H / Hk) * (hd + 2) * 4 : 0;
}

int attention_step_common(int32_t dtype, int32_t rows, int32_t H, int32_t Hk, int32_t hd, int32_t S,
                          const float* d_qkv, const float* d_cos, const float* d_sin, void* d_k, void* d_vt,
                          const int32_t* d_kv_len, const int32_t* d_new_slot, const int32_t* d_enable,
                          int32_t kv_cap, int32_t* d_err, void* d_out, void* d_ws, size_t ws_bytes, bool noalloc,
                          void* stream) {
  if (dtype != HAM_F32 && dtype != HAM_BF16) return fail(HAM_EINVAL, "bad dtype");
  if (rows < 1 || rows > 64 || H < 1 || Hk < 1 || H % Hk || H / Hk > 4 || (hd != 64 && hd != 128) || S < 64 ||
      S % 64)
    return fail(HAM_EINVAL, "bad attention shape");
  if (kv_cap < 0 || kv_cap >= S) return fail(HAM_EINVAL, "kv_cap out of range");
  if (!d_qkv || !d_cos || !d_sin || !d_k || !d_vt || !d_kv_len || !d_new_slot || !d_enable || !d_err || !d_out ||
      (!noalloc && !d_ws))
    return fail(HAM_EINVAL, "null pointer");
  const int nsplit = macro_attn_splits(dtype, rows, Hk, hd, kv_cap);
  if (noalloc) {
    const size_t need = attn_step_record_bytes(rows, H, Hk, hd, nsplit);
    if (need > NOALLOC_SCRATCH)
      return fail(HAM_ENOMEM, "split records need %zu bytes, above the %zu-byte scratch of the allocation-free entry",
                  need, NOALLOC_SCRATCH);
    if (int rc = noalloc_scratch(&d_ws)) return rc;
  } else if (ws_bytes < attn_part_bytes(rows, H, Hk, hd)) {
    return fail(HAM_ENOMEM, "workspace too small");
  }
  SeqPtrs sp{};
  sp.kv_len = const_cast<int*>(d_kv_len);
  sp.cur_slot = const_cast<int*>(d_new_slot);
  sp.cur_pos = sp.cur_slot;  // read by the row map, unused by attention (RoPE factors are given)
  sp.step_on = const_cast<int*>(d_enable);
  sp.err = d_err;
  AttnStepArgs sa{};
  sa.qkv = d_qkv; sa.part = nullptr; sa.nsplit_qkv = 1; sa.pM = rows; sa.ldqkv = (H + 2 * Hk) * hd;
  sa.cos_p = d_cos; sa.sin_p = d_sin; sa.cs_stride = hd / 2;
  sa.K = d_k; sa.VT = d_vt; sa.sb = (long long)Hk * S * hd; sa.sh = (long long)S * hd; sa.S = S;
  sa.H = H; sa.Hkv = Hk; sa.hd = hd; sa.R = rows; sa.kv_cap = kv_cap;
  sa.nsplit = nsplit;
  sa.o = d_out; sa.ldo = H * hd; sa.part_out = (float*)d_ws; sa.combine = true;
  sa.ss = nullptr; sa.ss_n = 0; sa.d = 1; sa.eps = 0.f;
  sa.rm.mode = ROWS_DECODE; sa.rm.st = sp;
  if (launch_attn_step(dtype, sa, (hipStream_t)stream)) return fail(HAM_EINVAL, "attention step shape");
  HIP_TRY(hipGetLastError());
  return HAM_OK;
}

}  // namespace

extern "C" {

int ham_op_attention_step(int32_t dtype, int32_t rows, int32_t H, int32_t Hk, int32_t hd, int32_t S,
                          const float* d_qkv, const float* d_cos, const float* d_sin, void* d_k, void* d_vt,
                          const int32_t* d_kv_len, const int32_t* d_new_slot, const int32_t* d_enable,
                          int32_t kv_cap, int32_t* d_err, void* d_out, void* d_ws, size_t ws_bytes, void* stream) {
  return attention_step_common(dtype, rows, H, Hk, hd, S, d_qkv, d_cos, d_sin, d_k, d_vt, d_kv_len, d_new_slot,
                               d_enable, kv_cap, d_err, d_out, d_ws, ws_bytes, false, stream);
}

int ham_op_attention_step_noalloc(int32_t dtype, int32_t rows, int32_t H, int32_t Hk, int32_t hd, int32_t S,
                                  const float* d_qkv, const float* d_cos, const float* d_sin, void* d_k, void* d_vt,
                                  const int32_t* d_kv_len, const int32_t* d_new_slot, const int32_t* d_enable,
                                  int32_t kv_cap, int32_t* d_err, void* d_out, void* stream) {
  return attention_step_common(dtype, rows, H, Hk, hd, S, d_qkv, d_cos, d_sin, d_k, d_vt, d_kv_len, d_new_slot,
                               d_enable, kv_cap, d_err, d_out, nullptr, 0, true, stream);
}

size_t ham_op_attention_step_noalloc_max_bytes(void) { return NOALLOC_SCRATCH; }

int ham_op_attention_step_splits(int32_t dtype, int32_t rows, int32_t Hk, int32_t hd, int32_t kv_cap) {
  if ((dtype != HAM_F32 && dtype != HAM_BF16) || rows < 1 || Hk < 1 || kv_cap < 0) return 0;
  return macro_attn_splits(dtype, rows, Hk, hd, kv_cap);
}

}  // extern "C"
