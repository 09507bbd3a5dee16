// Launch interface between the host library and the WINO kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wino {

// Geometry of one step over a batch of independent sequences.  Rows of the
// extended sequence are ordered [prompt | generation | shadow block]; the
// residual stream holds B*T rows, row b*T + t.
struct StepGeom {
  int B, P, G, Lb;      // batch, prompt length, generation length, block length
  // Ls shadow rows follow the S = P + G sequence rows: Lb, or 0 for a step in
  // which no position can be verified (Eq. 4 then reads current rows only, and
  // the other rows never see the shadow block, so dropping it changes nothing).
  int Ls;
  int S, T, Tp;         // T = S + Ls, Tp = T rounded up to 64
  int mask_id;
  const int32_t* block_start;  // [B] generation-relative start of Y_cur
  // activation type of the matrix-core operands: 0 bf16, 1 fp16 (the GEMM
  // weights are then fp16 copies)
  int f16;
};

// Absolute index of y_cur,1 for sequence b; finished sequences are clamped to
// the last block (their outputs are ignored).
__device__ __forceinline__ int cur_start(const StepGeom& g, int b) {
  int bs = g.block_start[b];
  bs = bs < 0 ? 0 : (bs > g.G - g.Lb ? g.G - g.Lb : bs);
  return g.P + bs;
}

// Position id of row t (Sec. 4.2.2): shadow row j reuses y_cur,j's id.
__device__ __forceinline__ int row_pos(const StepGeom& g, int b, int t) {
  return t < g.S ? t : cur_start(g, b) + (t - g.S);
}

// --------------------------------------------------------------- elementwise
// Activations h, q, k, v^T, the attention output and u are 16-bit values of
// the activation type (g.f16 or the f16 argument): bf16 or fp16.
// x[m] = E[token of row m] (fp32); h[m] = rmsnorm(x[m]) * gain.
void launch_embed_norm(const StepGeom& g, const int32_t* tokens, const uint16_t* emb, int vocab,
                       const uint16_t* gain, float eps, int d, float* x, uint16_t* h,
                       hipStream_t st);
// h[m] = rmsnorm(x[m]) * gain for m < M.  With n_part > 0 the split-K
// partials of rows m >= part_row0, part[s][m - part_row0] (s < n_part, fp32
// [n_part, M - part_row0, d]), are first added to x[m] in order s = 0, 1, ...
// and x is written back.
void launch_rmsnorm(float* x, const uint16_t* gain, float eps, int M, int d, uint16_t* h,
                    const float* part, int n_part, int part_row0, hipStream_t st, bool f16);
// out = fp16(in) for n bf16 values (n a multiple of 8), round to nearest even;
// *overflow is set to 1 if an output is not finite (|in| beyond fp16's range,
// or a non-finite input), else left as it is.
void launch_bf16_to_f16(const uint16_t* in, uint16_t* out, size_t n, int* overflow, hipStream_t st);
// x[m] += sum_s part[s][m - part_row0] (same order as above), for
// part_row0 <= m < M.
void launch_residual_reduce(float* x, const float* part, int n_part, int part_row0, int M, int d,
                            hipStream_t st);
// xc[b*(Lb+Ls) + i] = x row c0+i (i < Lb) or S+i-Lb (the shadow rows): the
// rows of the current block and the shadow block, fp32 [B*(Lb+Ls), d].
void launch_gather_block_rows(const StepGeom& g, const float* x, int d, float* xc, hipStream_t st);
// Rows the decision reads.  mode 0: one row per block position (current row
// if the token is the mask, else the shadow row) and target = current token
// (-1 for masked).  mode 1: all 2*Lb rows (current then shadow) per sequence.
// mode 2: response rows r0 .. r0+n-1 of the flattened [B, G] response (row
// P + j of sequence b for r = b*G + j), target = tgt_in[r].
// The normed row is written as hi = act(y) and lo = act(y - hi).
// With compact (mode 0 only) x holds the gathered block rows of
// launch_gather_block_rows instead of the full [B, T] stream.
void launch_select_norm(const StepGeom& g, int mode, const int32_t* tokens, const float* x,
                        const uint16_t* gain, float eps, int d, uint16_t* hf, uint16_t* hf_lo,
                        int32_t* target, hipStream_t st, int r0 = 0, int n = 0,
                        const int32_t* tgt_in = nullptr, bool compact = false);

// --------------------------------------------------------------- GEMM
// C = A * W^T with A [M, K] (row stride lda) and W [N, K] (row stride ldw)
// both bf16, or both fp16 (f16), fp32 accumulation, and one of the fused
// epilogues below.
struct RopeOut {      // QKV projection + rotate-half RoPE, head-major outputs
  uint16_t* q;        // [B, H, Tp, hd]
  uint16_t* k;        // [B, H, Tp, hd]
  uint16_t* vt;       // [B, H, hd, Tp]  (value transposed: token-contiguous)
  // cos and sin of the rotate-half angles, packed per lane of a 32-wide MFMA
  // block: tab[pos][l][fn] = (cos, sin) of element e = fn*32 + l of the first
  // half, fn < hd/64 - one 8*(hd/64)-byte load per (row, lane)
  const float* tab;   // [max_pos][32][hd/64][2]
  int H, hd;
};
struct LmStatsOut {   // LM head + streaming softmax statistics per (row, N-tile)
  const float* bias;  // [V] or null
  const int32_t* target;  // [M] id whose logit is recorded, or -1
  int mask_id;
  int n_part;         // partials per row (= N / BN)
  float* pm;          // [M, n_part] max logit of the tile
  float* ps;          // [M, n_part] sum exp(z - pm)
  float* pb;          // [M, n_part] max logit over ids != mask
  int32_t* pi;        // [M, n_part] lowest id reaching pb
  float* pt;          // [M, n_part] logit of target (kNegBig if not in tile)
  float* pz;          // [M, n_part] sum exp(z - pm) * (z - pm) (entropy), or null
};

enum GemmEpi {
  EPI_QKV_ROPE = 0, EPI_RESIDUAL = 1, EPI_SWIGLU = 2, EPI_LMSTATS = 3,
  EPI_STORE_F32 = 4,  // out = A W^T (plain A)
  EPI_LOGITS = 5      // out = (A + A2) W^T + bias (LM-head precision, test entry point)
};
constexpr int kMaxResidualSplits = 8;

struct GemmCall {
  int tile;  // 1 + tile shape index; 0 (zero-initialised call): chosen per call
  int f16;   // operand type: 0 bf16, 1 fp16 (activation outputs in the same type)
  // Residual epilogue only: rows [0, split_row0) are computed over the whole
  // K and added to outf; with splits > 1 each tile of rows [split_row0, M) is
  // computed as `splits` K-slices (slice s covers columns [s*K/splits,
  // (s+1)*K/splits)) that write fp32 partials part[s][m - split_row0][n]
  // (row stride N) for the next norm kernel to add.
  int splits, split_row0;
  float* part;
  const uint16_t* A; int lda;
  // LM-head epilogues take A as an unevaluated sum A + A2 of two 16-bit parts
  // (hi and lo of an fp32 row): both are multiplied with the same W tile.
  const uint16_t* A2;
  const uint16_t* W; int ldw;
  int M, N, K;
  GemmEpi epi;
  // residual: x[m*ldc + n] += acc ; store: out[m*ldc + n] = acc (+ bias[n])
  float* outf; int ldc; const float* bias;
  // swiglu: out[m*ldc + f] = silu(gate) * up (activation type); W rows: gate [0,F), up [F,2F)
  uint16_t* outh; int F;
  RopeOut rope;
  StepGeom geom;
  LmStatsOut lm;
};
// Picks a tile shape for the problem; returns the N-tile width used (the LM
// head needs it to size its partials) or 0 if no kernel fits.  The
// environment variable WINO_GEMM_TILE=<index> forces one tile shape (tuning).
int gemm_tile_n(const GemmCall& c);
hipError_t launch_gemm(const GemmCall& c, hipStream_t st);
// Plans a residual-add GEMM: tile shape and how many trailing row tiles are
// split over K (and how many ways), from a throughput model of whole-K tiles
// and thin K-slices filling the CUs; writes tile, splits and split_row0 into
// c.  part_elems bounds splits * (M - split_row0) * N.  The environment
// variables WINO_GEMM_TILE, WINO_GEMM_SPLIT and WINO_GEMM_TAIL (row tiles in
// the split tail) force choices (tuning).
void plan_residual_gemm(GemmCall& c, size_t part_elems);

// --------------------------------------------------------------- attention
// Bidirectional attention with the WINO shadow mask (Sec. 4.2.2): query row
// t < S sees keys [0, S); shadow query S+j sees keys [0, T) except c0+j.
// q, k, v^T and o in the activation type of g.f16; o: [B*T, H*hd] row-major.
// compact: query only each sequence's Lb current-block rows and Ls shadow
// rows; o then holds those rows, [B * (Lb + Ls), H*hd] (current rows first).
hipError_t launch_attention(const StepGeom& g, const uint16_t* q, const uint16_t* k,
                            const uint16_t* vt, int H, int hd, uint16_t* o, hipStream_t st,
                            bool compact = false);

// --------------------------------------------------------------- decision
// Per-position decision codes (same values as the public WINO_* flags).
constexpr int WINO_KEEP_FLAG = 0, WINO_DRAFT_FLAG = 1, WINO_REMASK_FLAG = 2,
              WINO_FORCED_FLAG = 3, WINO_CAPFILL_FLAG = 4;

struct DecideArgs {
  // partial softmax statistics [R, n_part] (R = B*Lb rows, row b*Lb + l)
  const float* pm; const float* ps; const float* pb; const int32_t* pi; const float* pt;
  int n_part;
  int B, Lb, mask_id;
  float tau1, tau2;
  int force_top1, cap_fill, cap;
  // fused-step mode: tokens [B, S] with Y_cur at P + block_start[b]
  int standalone;       // 1: tokens are [B, Lb] (Y_cur only), Eq. 4 always applied
  int32_t* tokens; int S, P, G;
  int32_t* block_start;  // [B]
  int32_t* block_steps;  // [B] or null
  int advance;           // move block_start to the next block holding a mask when Y_cur is full
  int32_t* seq_steps;    // [B] steps counter or null
  uint8_t* flags;        // [B, Lb] or null
  uint8_t* bitmap;       // [B, Lb] or null (standalone)
  int32_t* n_masked;     // [B] or null
  void* stats;           // wino_row_stats [B, Lb] or null
  int verify;            // shadow rows were computed: the Eq. 3 rule applies
  int topm;              // > 0: baseline mode, draft the topm most confident masks
  // [B, G] or null: step number (seq_steps after this step) written at every
  // response position the step changes (needs seq_steps)
  int32_t* final_step;
  // [B] or null: 1 if the sequence's next step may verify (it is active and
  // its next Y_cur holds both a mask and a drafted token), else 0
  int32_t* next_verify;
};
hipError_t launch_decide(const DecideArgs& a, hipStream_t st);
// WINO+ per-row quantities (Sec. 5.3) from LM-head partials of R rows (pz
// required): out[r] = {entropy, nll of the target, greedy confidence, argmax}
// (wino_loss_row layout).
hipError_t launch_loss_merge(const LmStatsOut& lm, int R, void* out, hipStream_t st);
// next_verify[b] as above for the state before any step (fused-step layout),
// and n_masked[b] (if given) the masks in that Y_cur (0 for a finished
// sequence).  With block_start (the same array as g.block_start, writable), a
// sequence whose Y_cur holds no mask first moves to the first later block
// holding one (or to G) and its block_steps entry (if given) restarts at 0.
hipError_t launch_probe_verify(const StepGeom& g, const int32_t* tokens, int32_t* next_verify,
                               hipStream_t st, int32_t* block_start = nullptr,
                               int32_t* block_steps = nullptr, int32_t* n_masked = nullptr);

// Standalone epilogue statistics: for each (b, l) pick the current row
// (masked) or the shadow row (unmasked) of bf16 logits [B, 2Lb, V], and write
// partials over chunks of kEpiChunk ids.
constexpr int kEpiChunk = 8192;
hipError_t launch_epilogue_stats(const uint16_t* logits, const int32_t* cur_tokens, int B, int Lb,
                                 int V, int mask_id, float* pm, float* ps, float* pb, int32_t* pi,
                                 float* pt, hipStream_t st);

}  // namespace wino
