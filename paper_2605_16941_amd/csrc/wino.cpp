// Host side of the WINO library: argument validation, workspace, kernel
// sequencing of one step, the block loop and the semi-autoregressive decode.
#include "wino.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"

using namespace wino;

// Scratch of wino_epilogue_noalloc: the partial statistics live in this
// file-scope device array (one copy per GPU, held until the process ends)
// instead of a caller workspace.  In host code its name is only a host-side
// stand-in, never a device address: host code uses the per-device address
// from hipGetSymbolAddress (noalloc_scratch).
constexpr size_t kNoAllocScratchBytes = WINO_EPILOGUE_NOALLOC_MAX_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

enum KClass {
  K_EMBED_NORM = 0, K_RMSNORM, K_GEMM_QKV, K_ATTENTION, K_GEMM_O, K_GEMM_GATEUP, K_GEMM_DOWN,
  K_SELECT_NORM, K_LM_HEAD, K_DECIDE, K_EPI_STATS, K_GEMM_DEBUG, K_GEMM_LAST
};
const char* kClassNames[WINO_N_KERNEL_CLASSES] = {
    "embed_norm", "rmsnorm", "gemm_qkv_rope", "attention", "gemm_o_residual", "gemm_gateup_swiglu",
    "gemm_down_residual", "select_norm", "lm_head_stats", "decide", "epilogue_stats", "gemm_logits",
    "gemm_last_layer_rows"};

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
constexpr int kMaxSplits = 8;
int round64(int v) { return (v + 63) / 64 * 64; }

struct Layout {
  size_t x, h, q, k, vt, att, u, hf, hf_lo, xc, part, target, rope_tab, pm, ps, pb, pi, pt, pz, misc,
      total;
  size_t rows;  // rows the LM-head partials hold
  int max_part;
  size_t part_elems;  // split-K partial buffer (fp32 elements)
};

Layout make_layout(const wino_model_config& c, int max_batch, int max_seq) {
  Layout L{};
  const size_t d = c.d_model, F = c.d_ff, hd = c.head_dim, H = c.n_heads;
  const size_t M = (size_t)max_batch * max_seq;
  const size_t Tp = round64(max_seq);
  const size_t R = (size_t)max_batch * (max_seq / 2 + 1);  // decision rows: B * Lb
  L.max_part = (c.vocab + 127) / 128;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
  L.x = take(M * d * 4);
  L.h = take(M * d * 2);
  L.q = take((size_t)max_batch * H * Tp * hd * 2);
  L.k = take((size_t)max_batch * H * Tp * hd * 2);
  L.vt = take((size_t)max_batch * H * Tp * hd * 2);
  L.att = take(M * d * 2);
  L.u = take(M * F * 2);
  L.hf = take(2 * R * d * 2);    // selected rows (hi, lo) for the LM head: up to
  L.hf_lo = take(2 * R * d * 2); // 2 * Lb per sequence (the test entry point)
  L.xc = take(2 * R * d * 4);    // last layer's current-block and shadow rows
  L.part_elems = (size_t)kMaxSplits * std::min<size_t>(M, 1024) * d;
  L.part = take(L.part_elems * 4);
  L.target = take(M * 4);
  L.rope_tab = take((size_t)max_seq * hd * 4);
  const size_t P = R * L.max_part;
  L.pm = take(P * 4);
  L.ps = take(P * 4);
  L.pb = take(P * 4);
  L.pi = take(P * 4);
  L.pt = take(P * 4);
  L.pz = take(P * 4);
  L.rows = R;
  L.misc = take((size_t)max_batch * 4 * 4);
  L.total = off;
  return L;
}

}  // namespace

struct wino_ctx {
  wino_model_config cfg{};
  int device = 0;
  int max_batch = 0, max_seq = 0;
  const uint16_t* tok_emb = nullptr;
  std::vector<const uint16_t*> attn_norm, w_qkv, w_o, ffn_norm, w_gu, w_down;
  const uint16_t* final_norm = nullptr;
  const uint16_t* lm_head = nullptr;
  const float* lm_bias = nullptr;
  int f16 = 0;                  // activations and GEMM weights in fp16
  uint16_t* wcopy = nullptr;    // fp16 copies of the GEMM and LM-head weights (f16)
  Layout L{};
  char* ws = nullptr;
  int32_t* h_pinned = nullptr;  // 4 * max_batch ints (block starts, step counts, next_verify)
  std::string err;
  // profiling
  uint32_t prof_mask = 0;
  struct Ev { int cls; hipEvent_t a, b; double flops, bytes; };
  std::vector<Ev> pending;
  std::vector<hipEvent_t> pool;
  int64_t launches[WINO_N_KERNEL_CLASSES] = {};
  double ms[WINO_N_KERNEL_CLASSES] = {}, flops[WINO_N_KERNEL_CLASSES] = {},
         bytes[WINO_N_KERNEL_CLASSES] = {};

  template <class T> T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
  float* x() const { return at<float>(L.x); }
  float* xc() const { return at<float>(L.xc); }
  uint16_t* h() const { return at<uint16_t>(L.h); }
  uint16_t* q() const { return at<uint16_t>(L.q); }
  uint16_t* k() const { return at<uint16_t>(L.k); }
  uint16_t* vt() const { return at<uint16_t>(L.vt); }
  uint16_t* att() const { return at<uint16_t>(L.att); }
  uint16_t* u() const { return at<uint16_t>(L.u); }
  uint16_t* hf() const { return at<uint16_t>(L.hf); }
  uint16_t* hf_lo() const { return at<uint16_t>(L.hf_lo); }
  float* part() const { return at<float>(L.part); }
  int32_t* target() const { return at<int32_t>(L.target); }
  float* rope_tab() const { return at<float>(L.rope_tab); }
  int32_t* block_steps() const { return at<int32_t>(L.misc); }
  int32_t* seq_steps() const { return at<int32_t>(L.misc) + max_batch; }
  int32_t* n_masked() const { return at<int32_t>(L.misc) + 2 * max_batch; }
  int32_t* next_verify() const { return at<int32_t>(L.misc) + 3 * max_batch; }

  hipEvent_t get_event() {
    if (!pool.empty()) { hipEvent_t e = pool.back(); pool.pop_back(); return e; }
    hipEvent_t e = nullptr;
    hipEventCreate(&e);
    return e;
  }
};

namespace {

wino_status hip_fail(wino_ctx* c, hipError_t e, const char* what) {
  if (c) {
    c->err = std::string(what) + ": " + hipGetErrorString(e);
  }
  return WINO_ERR_HIP;
}

#define HIP_TRY(ctx, expr)                                   \
  do {                                                       \
    hipError_t _e = (expr);                                  \
    if (_e != hipSuccess) return hip_fail(ctx, _e, #expr);   \
  } while (0)

// RAII-free launch bracket: records events around a launch when profiling.
struct Bracket {
  wino_ctx* c; int cls; hipStream_t st; hipEvent_t a = nullptr;
  Bracket(wino_ctx* c_, int cls_, hipStream_t st_) : c(c_), cls(cls_), st(st_) {
    if (c->prof_mask & (1u << cls)) { a = c->get_event(); hipEventRecord(a, st); }
  }
  void done(double flops, double bytes) {
    if (!a) return;
    hipEvent_t b = c->get_event();
    hipEventRecord(b, st);
    c->pending.push_back({cls, a, b, flops, bytes});
  }
};

bool shape_supported(const wino_model_config& c) {
  return c.n_layers >= 1 && c.d_model > 0 && c.n_heads > 0 && (c.head_dim == 64 || c.head_dim == 128) &&
         c.d_model == c.n_heads * c.head_dim && c.d_model % 64 == 0 && c.d_model <= 4096 &&
         c.d_ff % 64 == 0 && c.d_ff > 0 && c.vocab % 256 == 0 && c.vocab > 0 &&
         std::isfinite(c.rope_theta) && c.rope_theta > 0 && std::isfinite(c.rms_eps) && c.rms_eps > 0 &&
         (c.act_precision == WINO_ACT_BF16 || c.act_precision == WINO_ACT_FP16);
}

wino_status validate_params(wino_ctx* ctx, const wino_params* p) {
  if (!p) return WINO_ERR_INVALID_ARG;
  if (!std::isfinite(p->tau1) || !std::isfinite(p->tau2)) return WINO_ERR_INVALID_ARG;
  if (p->max_steps < 0 || p->tokens_per_step < 0) return WINO_ERR_INVALID_ARG;
  if (p->batch < 1 || p->prompt_len < 0 || p->gen_len < 1 || p->block_len < 1) return WINO_ERR_SHAPE;
  if (p->block_len > p->gen_len || p->gen_len % p->block_len) return WINO_ERR_SHAPE;
  if (p->block_len > 4096) return WINO_ERR_SHAPE;
  if (ctx) {
    if (p->mask_id < 0 || p->mask_id >= ctx->cfg.vocab) return WINO_ERR_INVALID_ARG;
    if (p->batch > ctx->max_batch) return WINO_ERR_SHAPE;
    if ((long)p->prompt_len + p->gen_len + p->block_len > ctx->max_seq) return WINO_ERR_SHAPE;
  }
  return WINO_OK;
}

StepGeom make_geom(const wino_ctx* c, const wino_params* p, const int32_t* block_start,
                   bool shadow = true) {
  StepGeom g{};
  g.f16 = c->f16;
  g.B = p->batch; g.P = p->prompt_len; g.G = p->gen_len; g.Lb = p->block_len;
  g.Ls = shadow ? g.Lb : 0;
  g.S = g.P + g.G; g.T = g.S + g.Ls; g.Tp = round64(g.T);
  g.mask_id = p->mask_id;
  g.block_start = block_start;
  return g;
}

// Split-K partials of a residual GEMM not yet added to x: n splits of the
// rows from row0 on.
struct Pending {
  int n = 0, row0 = 0;
};

// Residual-add GEMM.  When the planner splits the trailing row tiles over K,
// their fp32 partials land in the workspace and the caller adds them to x
// (fused into the next RMSNorm).
Pending residual_gemm(wino_ctx* c, GemmCall g, hipStream_t st, hipError_t* err) {
  g.part = c->part();
  plan_residual_gemm(g, c->L.part_elems);
  *err = launch_gemm(g, st);
  Pending p;
  if (g.splits > 1) { p.n = g.splits; p.row0 = g.split_row0; }
  return p;
}

// Bytes an RMSNorm moves: x read (and written back when partials are added),
// h written, partials read.
double norm_bytes(int M, int d, const Pending& p) {
  const double rows = p.n ? M - p.row0 : 0;
  return (double)M * d * 6 + rows * d * 4 + 4.0 * rows * d * p.n;
}

// Embedding and the first n_sub sublayers (attention and FFN halves of each
// layer, in order); leaves the residual stream in x.
// With compact, the last layer's attention queries, O projection and FFN run
// only on each sequence's current-block and shadow rows (the only rows the
// decision reads; keys and values still come from every row), gathered into
// xc = [B * (Lb + Ls), d]; the caller then reads the final rows from xc.
wino_status run_forward(wino_ctx* c, const StepGeom& g, const int32_t* tokens, int n_sub,
                        hipStream_t st, bool compact = false) {
  const wino_model_config& m = c->cfg;
  const int d = m.d_model, F = m.d_ff, H = m.n_heads, hd = m.head_dim;
  const int M = g.B * g.T;
  compact = compact && n_sub >= 2 * m.n_layers;
  Pending pend;  // split-K partials not yet added to x
  float* xr = c->x();  // residual stream of the rows being computed
  int Mr = M;
  {
    Bracket br(c, K_EMBED_NORM, st);
    launch_embed_norm(g, tokens, c->tok_emb, m.vocab, c->attn_norm[0], m.rms_eps, d, c->x(), c->h(), st);
    HIP_TRY(c, hipGetLastError());
    br.done(0, (double)M * d * (2 + 4 + 2));
  }
  for (int l = 0; l < m.n_layers && 2 * l < n_sub; ++l) {
    GemmCall qc{};
    qc.f16 = c->f16;
    qc.A = c->h(); qc.lda = d; qc.W = c->w_qkv[l]; qc.ldw = d;
    qc.M = M; qc.N = 3 * d; qc.K = d; qc.epi = EPI_QKV_ROPE;
    qc.rope = RopeOut{c->q(), c->k(), c->vt(), c->rope_tab(), H, hd};
    qc.geom = g;
    {
      Bracket br(c, K_GEMM_QKV, st);
      HIP_TRY(c, launch_gemm(qc, st));
      br.done(2.0 * M * 3.0 * d * d, 2.0 * ((double)M * d + 3.0 * d * d + 3.0 * M * d));
    }
    const bool last_compact = compact && l == m.n_layers - 1;
    {
      Bracket br(c, K_ATTENTION, st);
      HIP_TRY(c, launch_attention(g, c->q(), c->k(), c->vt(), H, hd, c->att(), st, last_compact));
      const double pairs = last_compact
                               ? (double)g.Lb * g.S + (double)g.Ls * (g.T - 1)
                               : (double)g.S * g.S + (double)g.Ls * (g.T - 1);
      br.done(4.0 * hd * H * g.B * pairs, 2.0 * 4.0 * M * d);
    }
    if (last_compact) {
      Bracket br(c, K_RMSNORM, st);
      launch_gather_block_rows(g, c->x(), d, c->xc(), st);
      HIP_TRY(c, hipGetLastError());
      xr = c->xc();
      Mr = g.B * (g.Lb + g.Ls);
      br.done(0, 8.0 * Mr * d);
    }
    GemmCall oc{};
    oc.f16 = c->f16;
    oc.A = c->att(); oc.lda = d; oc.W = c->w_o[l]; oc.ldw = d;
    oc.M = Mr; oc.N = d; oc.K = d; oc.epi = EPI_RESIDUAL; oc.outf = xr; oc.ldc = d;
    {
      Bracket br(c, xr == c->x() ? K_GEMM_O : K_GEMM_LAST, st);
      hipError_t e;
      pend = residual_gemm(c, oc, st, &e);
      HIP_TRY(c, e);
      br.done(2.0 * Mr * d * d, 2.0 * ((double)Mr * d + (double)d * d) + 8.0 * Mr * d);
    }
    if (2 * l + 1 >= n_sub) break;
    {
      Bracket br(c, K_RMSNORM, st);
      launch_rmsnorm(xr, c->ffn_norm[l], m.rms_eps, Mr, d, c->h(), c->part(), pend.n, pend.row0, st,
                     c->f16);
      HIP_TRY(c, hipGetLastError());
      br.done(0, norm_bytes(Mr, d, pend));
      pend = Pending{};
    }
    GemmCall gc{};
    gc.f16 = c->f16;
    gc.A = c->h(); gc.lda = d; gc.W = c->w_gu[l]; gc.ldw = d;
    gc.M = Mr; gc.N = 2 * F; gc.K = d; gc.epi = EPI_SWIGLU; gc.outh = c->u(); gc.ldc = F; gc.F = F;
    {
      Bracket br(c, xr == c->x() ? K_GEMM_GATEUP : K_GEMM_LAST, st);
      HIP_TRY(c, launch_gemm(gc, st));
      br.done(2.0 * Mr * 2.0 * F * d, 2.0 * ((double)Mr * d + 2.0 * F * d + (double)Mr * F));
    }
    GemmCall dc{};
    dc.f16 = c->f16;
    dc.A = c->u(); dc.lda = F; dc.W = c->w_down[l]; dc.ldw = F;
    dc.M = Mr; dc.N = d; dc.K = F; dc.epi = EPI_RESIDUAL; dc.outf = xr; dc.ldc = d;
    {
      Bracket br(c, xr == c->x() ? K_GEMM_DOWN : K_GEMM_LAST, st);
      hipError_t e;
      pend = residual_gemm(c, dc, st, &e);
      HIP_TRY(c, e);
      br.done(2.0 * Mr * (double)F * d, 2.0 * ((double)Mr * F + (double)F * d) + 8.0 * Mr * d);
    }
    if (l + 1 < m.n_layers && 2 * (l + 1) < n_sub) {
      Bracket br(c, K_RMSNORM, st);
      launch_rmsnorm(c->x(), c->attn_norm[l + 1], m.rms_eps, M, d, c->h(), c->part(), pend.n,
                     pend.row0, st, c->f16);
      HIP_TRY(c, hipGetLastError());
      br.done(0, norm_bytes(M, d, pend));
      pend = Pending{};
    }
  }
  if (pend.n) {
    Bracket br(c, K_RMSNORM, st);
    launch_residual_reduce(xr, c->part(), pend.n, pend.row0, Mr, d, st);
    HIP_TRY(c, hipGetLastError());
    const double rows = Mr - pend.row0;
    br.done(0, rows * d * 8 + 4.0 * rows * d * pend.n);
  }
  return WINO_OK;
}

// One fused WINO step.  shadow = false drops the shadow block for a step in
// which no position can be verified (tau2 <= 0, or every active sequence's
// Y_cur is all masks): the other rows never see it and Eq. 4 reads only
// current rows then, so the result is unchanged.
wino_status step_impl(wino_ctx* c, const wino_params* p, int32_t* tokens, int32_t* block_start,
                      int32_t* block_steps, uint8_t* flags, int32_t* n_masked, void* stats,
                      int advance, int32_t* seq_steps, bool shadow, hipStream_t st,
                      int32_t* final_step = nullptr) {
  const wino_model_config& m = c->cfg;
  shadow = shadow && p->tokens_per_step == 0;  // the baselines never verify
  const StepGeom g = make_geom(c, p, block_start, shadow);
  wino_status s = run_forward(c, g, tokens, 2 * m.n_layers, st, true);
  if (s != WINO_OK) return s;
  const int R = g.B * g.Lb;
  {
    Bracket br(c, K_SELECT_NORM, st);
    launch_select_norm(g, 0, tokens, c->xc(), c->final_norm, m.rms_eps, m.d_model, c->hf(), c->hf_lo(),
                       c->target(), st, 0, 0, nullptr, true);
    HIP_TRY(c, hipGetLastError());
    br.done(0, (double)R * m.d_model * 6);
  }
  GemmCall lc{};
  lc.f16 = c->f16;
  lc.A = c->hf(); lc.A2 = c->hf_lo(); lc.lda = m.d_model; lc.W = c->lm_head; lc.ldw = m.d_model;
  lc.M = R; lc.N = m.vocab; lc.K = m.d_model; lc.epi = EPI_LMSTATS;
  const int bn = gemm_tile_n(lc);
  if (bn == 0) { c->err = "no LM-head tile for this shape"; return WINO_ERR_UNSUPPORTED; }
  const int n_part = m.vocab / bn;
  lc.lm = LmStatsOut{c->lm_bias, c->target(), p->mask_id, n_part, c->at<float>(c->L.pm),
                     c->at<float>(c->L.ps), c->at<float>(c->L.pb), c->at<int32_t>(c->L.pi),
                     c->at<float>(c->L.pt)};
  {
    Bracket br(c, K_LM_HEAD, st);
    HIP_TRY(c, launch_gemm(lc, st));
    br.done(2.0 * R * (double)m.vocab * m.d_model,
            2.0 * ((double)R * m.d_model + (double)m.vocab * m.d_model) + 20.0 * R * n_part);
  }
  DecideArgs da{};
  da.pm = lc.lm.pm; da.ps = lc.lm.ps; da.pb = lc.lm.pb; da.pi = lc.lm.pi; da.pt = lc.lm.pt;
  da.n_part = n_part;
  da.B = g.B; da.Lb = g.Lb; da.mask_id = p->mask_id;
  da.tau1 = p->tau1; da.tau2 = p->tau2;
  da.force_top1 = !(p->flags & WINO_FLAG_NO_FORCE_TOP1);
  da.cap_fill = !(p->flags & WINO_FLAG_NO_CAP_FILL);
  da.cap = p->max_steps > 0 ? p->max_steps : p->block_len;
  da.standalone = 0;
  da.tokens = tokens; da.S = g.S; da.P = g.P; da.G = g.G;
  da.block_start = block_start; da.block_steps = block_steps; da.advance = advance;
  da.seq_steps = seq_steps; da.flags = flags; da.bitmap = nullptr; da.n_masked = n_masked;
  da.stats = stats;
  da.verify = shadow;
  da.topm = p->tokens_per_step;
  da.final_step = final_step;
  da.next_verify = c->next_verify();
  {
    Bracket br(c, K_DECIDE, st);
    HIP_TRY(c, launch_decide(da, st));
    br.done(0, 20.0 * R * n_part + 12.0 * R);
  }
  return WINO_OK;
}

wino_status drain_profile(wino_ctx* c) {
  for (auto& e : c->pending) {
    float ms = 0.f;
    HIP_TRY(c, hipEventSynchronize(e.b));
    HIP_TRY(c, hipEventElapsedTime(&ms, e.a, e.b));
    c->launches[e.cls] += 1;
    c->ms[e.cls] += ms;
    c->flops[e.cls] += e.flops;
    c->bytes[e.cls] += e.bytes;
    c->pool.push_back(e.a);
    c->pool.push_back(e.b);
  }
  c->pending.clear();
  return WINO_OK;
}

// Host-side argument checks of the standalone epilogue.
wino_status epilogue_check(const wino_params* p, int32_t vocab, const void* d_logits, const int32_t* d_cur_tokens,
                           const uint8_t* d_mask_bitmap) {
  if (!p || !d_logits || !d_cur_tokens || !d_mask_bitmap) return WINO_ERR_INVALID_ARG;
  if (!std::isfinite(p->tau1) || !std::isfinite(p->tau2)) return WINO_ERR_INVALID_ARG;
  if (p->tokens_per_step < 0) return WINO_ERR_INVALID_ARG;
  if (p->batch < 1 || p->block_len < 1 || vocab < 8 || vocab % 8) return WINO_ERR_SHAPE;
  if (p->mask_id < 0 || p->mask_id >= vocab) return WINO_ERR_INVALID_ARG;
  return WINO_OK;
}

// The standalone epilogue on a given workspace: partial statistics per
// (position, id chunk), then the merge and the decision.  Every partial the
// decision reads is written by the statistics kernel of the same call, so the
// workspace needs no clearing.
wino_status epilogue_impl(const wino_params* p, int32_t vocab, const void* d_logits, int32_t* d_cur_tokens,
                          uint8_t* d_mask_bitmap, uint8_t* d_flags, wino_row_stats* d_stats, void* d_workspace,
                          size_t workspace_bytes, void* stream) {
  wino_status s = epilogue_check(p, vocab, d_logits, d_cur_tokens, d_mask_bitmap);
  if (s != WINO_OK) return s;
  const size_t need = wino_epilogue_workspace_bytes(p->batch, p->block_len, vocab);
  if (workspace_bytes < need) return WINO_ERR_SHAPE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int R = p->batch * p->block_len;
  const int n_part = (vocab + kEpiChunk - 1) / kEpiChunk;
  char* ws = static_cast<char*>(d_workspace);
  float* pm = reinterpret_cast<float*>(ws);
  float* ps = pm + (size_t)R * n_part;
  float* pb = ps + (size_t)R * n_part;
  int32_t* pi = reinterpret_cast<int32_t*>(pb + (size_t)R * n_part);
  float* pt = reinterpret_cast<float*>(pi + (size_t)R * n_part);
  hipError_t e = launch_epilogue_stats(static_cast<const uint16_t*>(d_logits), d_cur_tokens, p->batch,
                                       p->block_len, vocab, p->mask_id, pm, ps, pb, pi, pt, st);
  if (e != hipSuccess) return WINO_ERR_HIP;
  DecideArgs da{};
  da.pm = pm; da.ps = ps; da.pb = pb; da.pi = pi; da.pt = pt; da.n_part = n_part;
  da.B = p->batch; da.Lb = p->block_len; da.mask_id = p->mask_id;
  da.tau1 = p->tau1; da.tau2 = p->tau2;
  da.force_top1 = !(p->flags & WINO_FLAG_NO_FORCE_TOP1);
  da.cap_fill = 0; da.cap = 0;
  da.topm = p->tokens_per_step;
  da.standalone = 1;
  da.tokens = d_cur_tokens;
  da.flags = d_flags; da.bitmap = d_mask_bitmap; da.stats = d_stats;
  e = launch_decide(da, st);
  return e == hipSuccess ? WINO_OK : WINO_ERR_HIP;
}

// The device address of each GPU's copy of `scratch` (above), looked up once
// per device with that device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

hipError_t noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

// Message of the last wino_create failure on this thread (no context exists
// to hold it); wino_last_error(NULL) returns it.
thread_local std::string t_create_err;

wino_status create_fail(wino_ctx* c, wino_status s, const char* what, hipError_t e = hipSuccess) {
  t_create_err = what;
  if (e != hipSuccess) t_create_err += std::string(": ") + hipGetErrorString(e);
  if (c) wino_destroy(c);
  return s;
}

}  // namespace

extern "C" {

size_t wino_workspace_bytes(const wino_model_config* cfg, int32_t max_batch, int32_t max_seq) {
  if (!cfg || max_batch < 1 || max_seq < 2) return 0;
  return make_layout(*cfg, max_batch, max_seq).total;
}

wino_status wino_create(const wino_model_config* cfg, const wino_weights* w, int32_t max_batch,
                        int32_t max_seq, wino_ctx** out) {
  if (!cfg || !w || !out) return create_fail(nullptr, WINO_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  if (max_batch < 1 || max_seq < 2) return create_fail(nullptr, WINO_ERR_SHAPE, "max_batch or max_seq");
  if (!shape_supported(*cfg)) return create_fail(nullptr, WINO_ERR_UNSUPPORTED, "model shape");
  if (!w->tok_emb || !w->attn_norm || !w->w_qkv || !w->w_o || !w->ffn_norm || !w->w_gate_up ||
      !w->w_down || !w->final_norm || !w->lm_head)
    return create_fail(nullptr, WINO_ERR_INVALID_ARG, "null weight pointer");
  for (int l = 0; l < cfg->n_layers; ++l)
    if (!w->attn_norm[l] || !w->w_qkv[l] || !w->w_o[l] || !w->ffn_norm[l] || !w->w_gate_up[l] ||
        !w->w_down[l])
      return create_fail(nullptr, WINO_ERR_INVALID_ARG, "null weight pointer");

  wino_ctx* c = new wino_ctx();
  c->cfg = *cfg;
  c->max_batch = max_batch;
  c->max_seq = max_seq;
  c->tok_emb = static_cast<const uint16_t*>(w->tok_emb);
  for (int l = 0; l < cfg->n_layers; ++l) {
    c->attn_norm.push_back(static_cast<const uint16_t*>(w->attn_norm[l]));
    c->w_qkv.push_back(static_cast<const uint16_t*>(w->w_qkv[l]));
    c->w_o.push_back(static_cast<const uint16_t*>(w->w_o[l]));
    c->ffn_norm.push_back(static_cast<const uint16_t*>(w->ffn_norm[l]));
    c->w_gu.push_back(static_cast<const uint16_t*>(w->w_gate_up[l]));
    c->w_down.push_back(static_cast<const uint16_t*>(w->w_down[l]));
  }
  c->final_norm = static_cast<const uint16_t*>(w->final_norm);
  c->lm_head = static_cast<const uint16_t*>(w->lm_head);
  c->lm_bias = w->lm_bias;
  c->L = make_layout(*cfg, max_batch, max_seq);

  // an optional cap on the workspace (bytes), checked before any HIP call
  const char* lim = std::getenv("WINO_WORKSPACE_LIMIT");
  if (lim && std::strtoull(lim, nullptr, 10) < c->L.total)
    return create_fail(c, WINO_ERR_NO_MEMORY, "workspace larger than WINO_WORKSPACE_LIMIT");
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) return create_fail(c, WINO_ERR_HIP, "hipGetDevice", e);
  e = hipMalloc(&c->ws, c->L.total);
  if (e != hipSuccess) { c->ws = nullptr; return create_fail(c, WINO_ERR_NO_MEMORY, "hipMalloc (workspace)", e); }
  e = hipHostMalloc(reinterpret_cast<void**>(&c->h_pinned), sizeof(int32_t) * 4 * max_batch);
  if (e != hipSuccess) {
    c->h_pinned = nullptr;
    return create_fail(c, WINO_ERR_NO_MEMORY, "hipHostMalloc", e);
  }
  // zeroed workspace: padding columns of the transposed values stay finite
  e = hipMemset(c->ws, 0, c->L.total);
  if (e != hipSuccess) return create_fail(c, WINO_ERR_HIP, "hipMemset (workspace)", e);
  // RoPE angles pos * theta^(-2i/hd), in double precision on the host, packed
  // as the QKV epilogue reads them: tab[pos][l][fn] = (cos, sin) of element
  // i = fn*32 + l (the lane of a 32-wide block and its block index)
  const int half = cfg->head_dim / 2, nblk = half / 32;
  std::vector<float> tab((size_t)max_seq * cfg->head_dim);
  for (int pos = 0; pos < max_seq; ++pos)
    for (int l = 0; l < 32; ++l)
      for (int fn = 0; fn < nblk; ++fn) {
        const int i = fn * 32 + l;
        const double inv = std::pow((double)cfg->rope_theta, -2.0 * i / cfg->head_dim);
        const double a = pos * inv;
        float* t = &tab[(((size_t)pos * 32 + l) * nblk + fn) * 2];
        t[0] = (float)std::cos(a);
        t[1] = (float)std::sin(a);
      }
  e = hipMemcpy(c->rope_tab(), tab.data(), tab.size() * 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) return create_fail(c, WINO_ERR_HIP, "hipMemcpy (RoPE table)", e);
  if (cfg->act_precision == WINO_ACT_FP16) {
    // fp16 copies of every matrix the matrix cores multiply (bf16 -> fp16 is
    // exact for |w| >= 2^-17 and moves smaller values by at most 2^-25)
    const size_t d = cfg->d_model, F = cfg->d_ff;
    const size_t per_layer = 3 * d * d + d * d + 2 * F * d + d * F;
    const size_t total = per_layer * cfg->n_layers + (size_t)cfg->vocab * d;
    e = hipMalloc(&c->wcopy, total * 2);
    if (e != hipSuccess) {
      c->wcopy = nullptr;
      return create_fail(c, WINO_ERR_NO_MEMORY, "hipMalloc (fp16 weight copies)", e);
    }
    c->f16 = 1;
    // the overflow flag lives in the first word of the (zeroed) workspace
    // until the copies are checked
    int* overflow = reinterpret_cast<int*>(c->ws);
    uint16_t* dst = c->wcopy;
    auto convert = [&](const uint16_t*& w, size_t n) {
      launch_bf16_to_f16(w, dst, n, overflow, nullptr);
      w = dst;
      dst += n;
    };
    for (int l = 0; l < cfg->n_layers; ++l) {
      convert(c->w_qkv[l], 3 * d * d);
      convert(c->w_o[l], d * d);
      convert(c->w_gu[l], 2 * F * d);
      convert(c->w_down[l], d * F);
    }
    convert(c->lm_head, (size_t)cfg->vocab * d);
    int h_overflow = 0;
    if ((e = hipGetLastError()) != hipSuccess || (e = hipDeviceSynchronize()) != hipSuccess ||
        (e = hipMemcpy(&h_overflow, overflow, sizeof(int), hipMemcpyDeviceToHost)) != hipSuccess ||
        (e = hipMemset(overflow, 0, sizeof(int))) != hipSuccess || (e = hipDeviceSynchronize()) != hipSuccess)
      return create_fail(c, WINO_ERR_HIP, "fp16 weight copies", e);
    // a weight beyond fp16's range has no fp16 copy
    if (h_overflow)
      return create_fail(c, WINO_ERR_UNSUPPORTED, "a weight matrix holds a value with no finite fp16 copy");
  }
  *out = c;
  return WINO_OK;
}

wino_status wino_destroy(wino_ctx* c) {
  if (!c) return WINO_ERR_INVALID_ARG;
  drain_profile(c);
  for (hipEvent_t e : c->pool) hipEventDestroy(e);
  if (c->ws) hipFree(c->ws);
  if (c->wcopy) hipFree(c->wcopy);
  if (c->h_pinned) hipHostFree(c->h_pinned);
  delete c;
  return WINO_OK;
}

wino_status wino_step(wino_ctx* c, const wino_params* p, int32_t* d_tokens,
                      const int32_t* d_block_start, int32_t* d_block_steps, uint8_t* d_flags,
                      int32_t* d_n_masked, wino_row_stats* d_stats, void* stream) {
  if (!c) return WINO_ERR_INVALID_ARG;
  wino_status s = validate_params(c, p);
  if (s != WINO_OK) return s;
  if (!d_tokens || !d_block_start) return WINO_ERR_INVALID_ARG;
  // Eq. 3 can only fire with tau2 > 0 (a probability is never below 0); the
  // device state is not known here without a synchronisation
  return step_impl(c, p, d_tokens, const_cast<int32_t*>(d_block_start), d_block_steps, d_flags,
                   d_n_masked, d_stats, 0, nullptr, p->tau2 > 0.f, static_cast<hipStream_t>(stream));
}

namespace {

// Steps one block may take: the cap, or the fixed schedule of the baselines.
int block_cap(const wino_params* p) {
  if (p->tokens_per_step > 0) return (p->block_len + p->tokens_per_step - 1) / p->tokens_per_step;
  return p->max_steps > 0 ? p->max_steps : p->block_len;
}

// Whether the coming step needs the shadow block: tau2 > 0 and some sequence
// may verify (next_verify, written by the decision kernel or the probe).
bool need_shadow(const wino_params* p, const int32_t* h_next_verify) {
  if (!(p->tau2 > 0.f) || p->tokens_per_step > 0) return false;
  for (int b = 0; b < p->batch; ++b)
    if (h_next_verify[b]) return true;
  return false;
}

}  // namespace

wino_status wino_decode_block(wino_ctx* c, const wino_params* p, int32_t* d_tokens,
                              const int32_t* d_block_start, int32_t* d_final_step, int32_t* h_steps,
                              void* stream) {
  if (!c) return WINO_ERR_INVALID_ARG;
  wino_status s = validate_params(c, p);
  if (s != WINO_OK) return s;
  if (!d_tokens || !d_block_start) return WINO_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int B = p->batch;
  const int cap = block_cap(p);
  HIP_TRY(c, hipMemsetAsync(c->block_steps(), 0, sizeof(int32_t) * 2 * c->max_batch, st));
  int32_t* h_nv = c->h_pinned + 2 * B;  // next_verify per sequence
  HIP_TRY(c, launch_probe_verify(make_geom(c, p, d_block_start), d_tokens, c->next_verify(), st,
                                 nullptr, nullptr, c->n_masked()));
  HIP_TRY(c, hipMemcpyAsync(h_nv, c->next_verify(), sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
  HIP_TRY(c, hipMemcpyAsync(c->h_pinned, c->n_masked(), sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
  HIP_TRY(c, hipStreamSynchronize(st));
  // no current block holds a mask: nothing to decode, no forward
  bool any_mask = false;
  for (int b = 0; b < B; ++b) any_mask |= c->h_pinned[b] > 0;
  for (int it = 0; any_mask; ++it) {
    s = step_impl(c, p, d_tokens, const_cast<int32_t*>(d_block_start), c->block_steps(), nullptr,
                  c->n_masked(), nullptr, 0, c->seq_steps(), need_shadow(p, h_nv), st, d_final_step);
    if (s != WINO_OK) return s;
    HIP_TRY(c, hipMemcpyAsync(c->h_pinned, c->n_masked(), sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
    HIP_TRY(c, hipMemcpyAsync(h_nv, c->next_verify(), sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
    HIP_TRY(c, hipStreamSynchronize(st));
    bool any = false;
    for (int b = 0; b < B; ++b) any |= c->h_pinned[b] > 0;
    if (!any) break;
    if (it + 1 >= cap) { c->err = "block did not finish within its step cap"; return WINO_ERR_STEP_CAP; }
  }
  if (h_steps) {
    HIP_TRY(c, hipMemcpy(h_steps, c->seq_steps(), sizeof(int32_t) * B, hipMemcpyDeviceToHost));
  }
  return WINO_OK;
}

wino_status wino_decode(wino_ctx* c, const wino_params* p, int32_t* d_tokens, int32_t* d_block_start,
                        int32_t* d_block_steps, int32_t* d_final_step, int32_t max_forwards,
                        int32_t* h_steps_per_seq, int32_t* h_forward_passes, void* stream) {
  if (!c) return WINO_ERR_INVALID_ARG;
  wino_status s = validate_params(c, p);
  if (s != WINO_OK) return s;
  if (!d_tokens || !d_block_start || max_forwards < 0) return WINO_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int B = p->batch;
  const int cap = block_cap(p);
  // every block takes at most `cap` steps, so this many forwards finish any state
  const long budget = (long)(p->gen_len / p->block_len) * cap;
  // block steps: the caller's (a resumed state) or zeros
  int32_t* bsteps = d_block_steps ? d_block_steps : c->block_steps();
  if (!d_block_steps)
    HIP_TRY(c, hipMemsetAsync(c->block_steps(), 0, sizeof(int32_t) * c->max_batch, st));
  HIP_TRY(c, hipMemsetAsync(c->seq_steps(), 0, sizeof(int32_t) * c->max_batch, st));
  int forwards = 0;
  int32_t* h_nv = c->h_pinned + 2 * B;  // next_verify per sequence
  // blocks holding no mask at the start (a resumed or pre-filled state) are skipped
  HIP_TRY(c, launch_probe_verify(make_geom(c, p, d_block_start), d_tokens, c->next_verify(), st,
                                 d_block_start, bsteps));
  HIP_TRY(c, hipMemcpyAsync(h_nv, c->next_verify(), sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
  HIP_TRY(c, hipMemcpyAsync(c->h_pinned, d_block_start, sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
  HIP_TRY(c, hipStreamSynchronize(st));
  for (;;) {
    bool all_done = true;
    for (int b = 0; b < B; ++b) all_done &= c->h_pinned[b] >= p->gen_len;
    if (all_done) break;
    if (max_forwards > 0 && forwards >= max_forwards) break;  // a resumable checkpoint
    if (forwards >= budget) {
      c->err = "decode exceeded its forward budget (a block hit its step cap)";
      return WINO_ERR_STEP_CAP;
    }
    s = step_impl(c, p, d_tokens, d_block_start, bsteps, nullptr, c->n_masked(), nullptr, 1,
                  c->seq_steps(), need_shadow(p, h_nv), st, d_final_step);
    if (s != WINO_OK) return s;
    ++forwards;
    HIP_TRY(c, hipMemcpyAsync(c->h_pinned, d_block_start, sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
    HIP_TRY(c, hipMemcpyAsync(c->h_pinned + B, bsteps, sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
    HIP_TRY(c, hipMemcpyAsync(h_nv, c->next_verify(), sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
    HIP_TRY(c, hipStreamSynchronize(st));
    if ((p->flags & WINO_FLAG_NO_CAP_FILL) && p->tokens_per_step == 0)
      for (int b = 0; b < B; ++b)
        if (c->h_pinned[b] < p->gen_len && c->h_pinned[B + b] >= cap) {
          c->err = "block did not finish within its step cap";
          return WINO_ERR_STEP_CAP;
        }
  }
  if (h_steps_per_seq)
    HIP_TRY(c, hipMemcpy(h_steps_per_seq, c->seq_steps(), sizeof(int32_t) * B, hipMemcpyDeviceToHost));
  if (h_forward_passes) *h_forward_passes = forwards;
  return WINO_OK;
}

wino_status wino_row_losses(wino_ctx* c, const wino_params* p, const int32_t* d_tokens,
                            const int32_t* d_targets, wino_row_loss* d_out, void* stream) {
  if (!c) return WINO_ERR_INVALID_ARG;
  wino_status s = validate_params(c, p);
  if (s != WINO_OK) return s;
  if (!d_tokens || !d_targets || !d_out) return WINO_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const wino_model_config& m = c->cfg;
  // a plain forward: no shadow rows, so the block cursor is never read for
  // positions (any valid [B] int32 buffer serves as its pointer)
  const StepGeom g = make_geom(c, p, c->block_steps(), false);
  s = run_forward(c, g, d_tokens, 2 * m.n_layers, st);
  if (s != WINO_OK) return s;
  GemmCall lc{};
  lc.f16 = c->f16;
  lc.A = c->hf(); lc.A2 = c->hf_lo(); lc.lda = m.d_model; lc.W = c->lm_head; lc.ldw = m.d_model;
  lc.N = m.vocab; lc.K = m.d_model; lc.epi = EPI_LMSTATS;
  const long total = (long)g.B * g.G;
  const int chunk = (int)std::min<size_t>(c->L.rows, 1 << 20);
  for (long r0 = 0; r0 < total; r0 += chunk) {
    const int n = (int)std::min<long>(chunk, total - r0);
    {
      Bracket br(c, K_SELECT_NORM, st);
      launch_select_norm(g, 2, d_tokens, c->x(), c->final_norm, m.rms_eps, m.d_model, c->hf(), c->hf_lo(),
                         c->target(), st, (int)r0, n, d_targets);
      HIP_TRY(c, hipGetLastError());
      br.done(0, (double)n * m.d_model * 8);
    }
    lc.M = n;
    const int bn = gemm_tile_n(lc);
    if (bn == 0) { c->err = "no LM-head tile for this shape"; return WINO_ERR_UNSUPPORTED; }
    const int n_part = m.vocab / bn;
    if (n_part > c->L.max_part) { c->err = "LM-head partials exceed the workspace"; return WINO_ERR_UNSUPPORTED; }
    lc.lm = LmStatsOut{c->lm_bias, c->target(), p->mask_id, n_part, c->at<float>(c->L.pm),
                       c->at<float>(c->L.ps), c->at<float>(c->L.pb), c->at<int32_t>(c->L.pi),
                       c->at<float>(c->L.pt), c->at<float>(c->L.pz)};
    {
      Bracket br(c, K_LM_HEAD, st);
      HIP_TRY(c, launch_gemm(lc, st));
      br.done(2.0 * n * (double)m.vocab * m.d_model,
              2.0 * ((double)n * m.d_model + (double)m.vocab * m.d_model) + 24.0 * n * n_part);
    }
    {
      Bracket br(c, K_DECIDE, st);
      HIP_TRY(c, launch_loss_merge(lc.lm, n, d_out + r0, st));
      br.done(0, 24.0 * n * n_part + 16.0 * n);
    }
  }
  return WINO_OK;
}

size_t wino_epilogue_workspace_bytes(int32_t batch, int32_t block_len, int32_t vocab) {
  if (batch < 1 || block_len < 1 || vocab < 1) return 0;
  const size_t n_part = (vocab + kEpiChunk - 1) / kEpiChunk;
  return (size_t)batch * block_len * n_part * 20 + 256;
}

wino_status wino_epilogue(const wino_params* p, int32_t vocab, const void* d_logits, int32_t* d_cur_tokens,
                          uint8_t* d_mask_bitmap, uint8_t* d_flags, wino_row_stats* d_stats,
                          void* d_workspace, size_t workspace_bytes, void* stream) {
  if (!d_workspace) return WINO_ERR_INVALID_ARG;
  return epilogue_impl(p, vocab, d_logits, d_cur_tokens, d_mask_bitmap, d_flags, d_stats, d_workspace,
                       workspace_bytes, stream);
}

wino_status wino_epilogue_noalloc(const wino_params* p, int32_t vocab, const void* d_logits,
                                  int32_t* d_cur_tokens, uint8_t* d_mask_bitmap, uint8_t* d_flags,
                                  wino_row_stats* d_stats, void* stream) {
  // host-side checks first: nothing below touches the device on a rejected call
  wino_status s = epilogue_check(p, vocab, d_logits, d_cur_tokens, d_mask_bitmap);
  if (s != WINO_OK) return s;
  if (wino_epilogue_workspace_bytes(p->batch, p->block_len, vocab) > kNoAllocScratchBytes)
    return WINO_ERR_SHAPE;
  void* ws = nullptr;
  if (noalloc_scratch(&ws) != hipSuccess) return WINO_ERR_HIP;
  return epilogue_impl(p, vocab, d_logits, d_cur_tokens, d_mask_bitmap, d_flags, d_stats, ws,
                       kNoAllocScratchBytes, stream);
}

wino_status wino_debug_logits(wino_ctx* c, const wino_params* p, const int32_t* d_tokens,
                              const int32_t* d_block_start, float* d_logits, void* stream) {
  if (!c) return WINO_ERR_INVALID_ARG;
  wino_status s = validate_params(c, p);
  if (s != WINO_OK) return s;
  if (!d_tokens || !d_block_start || !d_logits) return WINO_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const wino_model_config& m = c->cfg;
  const StepGeom g = make_geom(c, p, d_block_start);
  s = run_forward(c, g, d_tokens, 2 * m.n_layers, st);
  if (s != WINO_OK) return s;
  launch_select_norm(g, 1, d_tokens, c->x(), c->final_norm, m.rms_eps, m.d_model, c->hf(), c->hf_lo(),
                     c->target(), st);
  HIP_TRY(c, hipGetLastError());
  GemmCall lc{};
  lc.f16 = c->f16;
  lc.A = c->hf(); lc.A2 = c->hf_lo(); lc.lda = m.d_model; lc.W = c->lm_head; lc.ldw = m.d_model;
  lc.M = g.B * 2 * g.Lb; lc.N = m.vocab; lc.K = m.d_model; lc.epi = EPI_LOGITS;
  lc.outf = d_logits; lc.ldc = m.vocab; lc.bias = c->lm_bias;
  Bracket br(c, K_GEMM_DEBUG, st);
  HIP_TRY(c, launch_gemm(lc, st));
  br.done(2.0 * lc.M * (double)m.vocab * m.d_model, 0);
  return WINO_OK;
}

wino_status wino_debug_forward(wino_ctx* c, const wino_params* p, const int32_t* d_tokens,
                               const int32_t* d_block_start, int32_t n_sublayers, float* d_out,
                               void* stream) {
  if (!c) return WINO_ERR_INVALID_ARG;
  wino_status s = validate_params(c, p);
  if (s != WINO_OK) return s;
  if (!d_tokens || !d_block_start || !d_out) return WINO_ERR_INVALID_ARG;
  if (n_sublayers < 0 || n_sublayers > 2 * c->cfg.n_layers) return WINO_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const StepGeom g = make_geom(c, p, d_block_start);
  s = run_forward(c, g, d_tokens, n_sublayers, st);
  if (s != WINO_OK) return s;
  HIP_TRY(c, hipMemcpyAsync(d_out, c->x(), sizeof(float) * (size_t)g.B * g.T * c->cfg.d_model,
                            hipMemcpyDeviceToDevice, st));
  return WINO_OK;
}

wino_status wino_debug_gemm(const void* d_A, const void* d_W, int32_t M, int32_t N, int32_t K,
                            float* d_out, void* stream) {
  if (!d_A || !d_W || !d_out) return WINO_ERR_INVALID_ARG;
  if (M < 1 || N < 1 || K < 1) return WINO_ERR_SHAPE;
  GemmCall gc{};
  gc.A = static_cast<const uint16_t*>(d_A); gc.lda = K;
  gc.W = static_cast<const uint16_t*>(d_W); gc.ldw = K;
  gc.M = M; gc.N = N; gc.K = K; gc.epi = EPI_STORE_F32; gc.outf = d_out; gc.ldc = N;
  if (gemm_tile_n(gc) == 0) return WINO_ERR_UNSUPPORTED;
  return launch_gemm(gc, static_cast<hipStream_t>(stream)) == hipSuccess ? WINO_OK : WINO_ERR_HIP;
}

wino_status wino_profile(wino_ctx* c, uint32_t class_mask) {
  if (!c) return WINO_ERR_INVALID_ARG;
  c->prof_mask = class_mask;
  return WINO_OK;
}

wino_status wino_profile_read(wino_ctx* c, int64_t* h_launches, double* h_ms, double* h_flops,
                              double* h_bytes) {
  if (!c) return WINO_ERR_INVALID_ARG;
  wino_status s = drain_profile(c);
  if (s != WINO_OK) return s;
  for (int i = 0; i < WINO_N_KERNEL_CLASSES; ++i) {
    if (h_launches) h_launches[i] = c->launches[i];
    if (h_ms) h_ms[i] = c->ms[i];
    if (h_flops) h_flops[i] = c->flops[i];
    if (h_bytes) h_bytes[i] = c->bytes[i];
    c->launches[i] = 0;
    c->ms[i] = c->flops[i] = c->bytes[i] = 0;
  }
  return WINO_OK;
}

const char* wino_kernel_class_name(int32_t cls) {
  if (cls < 0 || cls >= WINO_N_KERNEL_CLASSES) return "";
  return kClassNames[cls];
}

const char* wino_status_string(wino_status s) {
  switch (s) {
    case WINO_OK: return "ok";
    case WINO_ERR_INVALID_ARG: return "invalid argument";
    case WINO_ERR_SHAPE: return "shape mismatch";
    case WINO_ERR_HIP: return "HIP runtime error";
    case WINO_ERR_NO_MEMORY: return "out of device memory";
    case WINO_ERR_STEP_CAP: return "block hit its step cap";
    case WINO_ERR_UNSUPPORTED: return "unsupported model shape";
  }
  return "unknown status";
}

const char* wino_last_error(const wino_ctx* c) { return c ? c->err.c_str() : t_create_err.c_str(); }

}  // extern "C"
