// bf16 GEMM C = A * W^T on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16),
// with the epilogues of the WINO forward fused in:
//   QKV projection + rotate-half RoPE at the WINO position ids,
//   residual add into the fp32 stream (O projection, FFN down projection),
//   SwiGLU of interleaved gate/up tiles,
//   LM head + per-tile softmax statistics (max, sum-exp, best non-mask id,
//   logit of the current token) so the logits never reach memory,
//   plain fp32 store (+bias) for the test entry point.
//
// Tiling: a workgroup owns a BM x BN output tile and walks K in steps of 64.
// A and W tiles are staged global -> registers -> LDS (rows padded by 16 bytes
// so that the 16-byte fragment reads of 8 consecutive rows hit distinct bank
// groups); the next K step is fetched into registers while the matrix cores
// consume the current one.  Waves form a WM x WN grid, each owning a
// (BM/WM) x (BN/WN) sub-tile of 32x32 MFMA blocks.  Workgroups are renumbered
// so that each XCD works on one contiguous range of tiles (shared W tiles stay
// in that XCD's L2).
#include <climits>

#include "common.h"
#include "kernels.h"

namespace wino {
namespace {

constexpr int BK = 64;
constexpr int LDK = BK + 8;

// SwiGLU virtual columns come in blocks of WTN: the first half of a block is
// gate rows f0..f0+WTN/2-1, the second half the up rows of the same f range,
// so each lane holds both factors of its outputs.
template <int WTN>
__device__ __forceinline__ int swiglu_row(int vc, int F) {
  constexpr int half = WTN / 2;
  const int blk = vc / WTN, c = vc - blk * WTN;
  const int f = blk * half + (c < half ? c : c - half);
  return c < half ? f : F + f;
}

template <int FM, int FN>
__device__ __forceinline__ void epi_residual(const GemmCall& c, f32x16 (&acc)[FM][FN], int rowb,
                                             int colb, int lane) {
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = rowb + fm * 32 + mfma_row(i, lane);
      if (row >= c.M) continue;
      float* dst = c.outf + (size_t)row * c.ldc + colb + (lane & 31);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) dst[fn * 32] += acc[fm][fn][i];
    }
}

template <int FM, int FN>
__device__ __forceinline__ void epi_store(const GemmCall& c, f32x16 (&acc)[FM][FN], int rowb,
                                          int colb, int lane) {
  float bias[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) bias[fn] = c.bias ? c.bias[colb + fn * 32 + (lane & 31)] : 0.f;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = rowb + fm * 32 + mfma_row(i, lane);
      if (row >= c.M) continue;
      float* dst = c.outf + (size_t)row * c.ldc + colb + (lane & 31);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) dst[fn * 32] = acc[fm][fn][i] + bias[fn];
    }
}

template <int FM, int FN>
__device__ __forceinline__ void epi_swiglu(const GemmCall& c, f32x16 (&acc)[FM][FN], int rowb,
                                           int colb, int lane) {
  constexpr int H2 = FN / 2;
  const int fb = colb / 2 + (lane & 31);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = rowb + fm * 32 + mfma_row(i, lane);
      if (row >= c.M) continue;
      uint16_t* dst = c.outh + (size_t)row * c.ldc + fb;
#pragma unroll
      for (int fn = 0; fn < H2; ++fn) {
        const float g = acc[fm][fn][i], u = acc[fm][fn + H2][i];
        dst[fn * 32] = f2bf(g / (1.f + __expf(-g)) * u);
      }
    }
}

// Wave columns = one head (WTN == hd): lane holds columns e and e + hd/2 of
// the rotate-half pair in fragments fn and fn + FN/2.
template <int FM, int FN>
__device__ __forceinline__ void epi_qkv_rope(const GemmCall& c, f32x16 (&acc)[FM][FN], int rowb,
                                             int colb, int lane) {
  constexpr int H2 = FN / 2;
  const RopeOut& ro = c.rope;
  const StepGeom& g = c.geom;
  const int hd = ro.hd, half = hd / 2;
  const int d = ro.H * hd;
  const int which = colb / d;               // 0 q, 1 k, 2 v
  const int head = (colb - which * d) / hd;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = rowb + fm * 32 + mfma_row(i, lane);
      if (row >= c.M) continue;
      const int b = row / g.T, t = row - b * g.T;
      const size_t bh = (size_t)b * ro.H + head;
      if (which < 2) {
        const int pos = row_pos(g, b, t);
        uint16_t* dst = (which == 0 ? ro.q : ro.k) + (bh * g.Tp + t) * hd;
#pragma unroll
        for (int fn = 0; fn < H2; ++fn) {
          const int e = fn * 32 + (lane & 31);
          const float cs = ro.cos_t[(size_t)pos * half + e], sn = ro.sin_t[(size_t)pos * half + e];
          const float x1 = acc[fm][fn][i], x2 = acc[fm][fn + H2][i];
          dst[e] = f2bf(x1 * cs - x2 * sn);
          dst[e + half] = f2bf(x2 * cs + x1 * sn);
        }
      } else {
        uint16_t* dst = ro.vt + bh * hd * g.Tp + t;
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const int e = fn * 32 + (lane & 31);
          dst[(size_t)e * g.Tp] = f2bf(acc[fm][fn][i]);
        }
      }
    }
}

// LM head epilogue: per row of the tile, statistics over the BN columns.
template <int BM, int WM, int WN, int FM, int FN>
__device__ __forceinline__ void epi_lmstats(const GemmCall& c, f32x16 (&acc)[FM][FN], int m0,
                                            int tn, int rowb, int colb, int lane, int wm, int wn,
                                            uint16_t* smem_raw) {
  const LmStatsOut& lm = c.lm;
  float* red_m = reinterpret_cast<float*>(smem_raw);
  float* red_s = red_m + WN * BM;
  float* red_b = red_s + WN * BM;
  float* red_t = red_b + WN * BM;
  int* red_i = reinterpret_cast<int*>(red_t + WN * BM);
  float bias[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) bias[fn] = lm.bias ? lm.bias[colb + fn * 32 + (lane & 31)] : 0.f;
  __syncthreads();  // LDS is reused
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int lrow = wm * (BM / WM) + fm * 32 + mfma_row(i, lane);
      const int row = m0 + lrow;
      const int tgt = row < c.M ? lm.target[row] : -1;
      float mx = kNegBig, bz = kNegBig, tz = kNegBig;
      int bi = INT_MAX;
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int col = colb + fn * 32 + (lane & 31);
        const float v = acc[fm][fn][i] + bias[fn];
        mx = fmaxf(mx, v);
        if (col != lm.mask_id && v > bz) { bz = v; bi = col; }
        if (col == tgt) tz = v;
      }
#pragma unroll
      for (int o = 16; o > 0; o >>= 1) {
        mx = fmaxf(mx, __shfl_xor(mx, o, 64));
        tz = fmaxf(tz, __shfl_xor(tz, o, 64));
        const float ob = __shfl_xor(bz, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (ob > bz || (ob == bz && oi < bi)) { bz = ob; bi = oi; }
      }
      float se = 0.f;
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) se += __expf(acc[fm][fn][i] + bias[fn] - mx);
#pragma unroll
      for (int o = 16; o > 0; o >>= 1) se += __shfl_xor(se, o, 64);
      if ((lane & 31) == 0) {
        red_m[wn * BM + lrow] = mx;
        red_s[wn * BM + lrow] = se;
        red_b[wn * BM + lrow] = bz;
        red_t[wn * BM + lrow] = tz;
        red_i[wn * BM + lrow] = bi;
      }
    }
  __syncthreads();
  for (int r = threadIdx.x; r < BM; r += WM * WN * 64) {
    const int row = m0 + r;
    if (row >= c.M) continue;
    float m = kNegBig;
#pragma unroll
    for (int w = 0; w < WN; ++w) m = fmaxf(m, red_m[w * BM + r]);
    float s = 0.f, bz = kNegBig, tz = kNegBig;
    int bi = INT_MAX;
#pragma unroll
    for (int w = 0; w < WN; ++w) {
      s += red_s[w * BM + r] * __expf(red_m[w * BM + r] - m);
      const float ob = red_b[w * BM + r];
      const int oi = red_i[w * BM + r];
      if (ob > bz || (ob == bz && oi < bi)) { bz = ob; bi = oi; }
      tz = fmaxf(tz, red_t[w * BM + r]);
    }
    const size_t o = (size_t)row * lm.n_part + tn;
    lm.pm[o] = m;
    lm.ps[o] = s;
    lm.pb[o] = bz;
    lm.pi[o] = bi;
    lm.pt[o] = tz;
  }
}

template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(WM* WN * 64) void gemm_kernel(const GemmCall c) {
  constexpr int NT = WM * WN * 64;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int AC = BM * BK / 8 / NT;
  constexpr int BC = BN * BK / 8 / NT;
  static_assert(AC >= 1 && BC >= 1 && AC * NT * 8 == BM * BK && BC * NT * 8 == BN * BK,
                "tile / thread split");
  static_assert(FM >= 1 && FN >= 1, "wave tile");

  __shared__ __attribute__((aligned(16))) uint16_t smem[(BM + BN) * LDK];
  uint16_t* As = smem;
  uint16_t* Bs = smem + BM * LDK;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave - (wave / WN) * WN;
  const int nTM = (c.M + BM - 1) / BM;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int tm = tile % nTM, tn = tile / nTM;
  const int m0 = tm * BM, n0 = tn * BN;

  const uint16_t* ap[AC];
  int al[AC];
#pragma unroll
  for (int j = 0; j < AC; ++j) {
    const int q = tid + j * NT, r = q >> 3, kc = q & 7;
    const int gm = min(m0 + r, c.M - 1);
    ap[j] = c.A + (size_t)gm * c.lda + kc * 8;
    al[j] = r * LDK + kc * 8;
  }
  const uint16_t* bp[BC];
  int bl[BC];
#pragma unroll
  for (int j = 0; j < BC; ++j) {
    const int q = tid + j * NT, r = q >> 3, kc = q & 7;
    const int vc = n0 + r;
    const int wr = EPI == EPI_SWIGLU ? swiglu_row<WTN>(vc, c.F) : vc;
    bp[j] = c.W + (size_t)wr * c.ldw + kc * 8;
    bl[j] = r * LDK + kc * 8;
  }

  f32x16 acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[fm][fn][i] = 0.f;

  uint4 ra[AC], rb[BC];
#pragma unroll
  for (int j = 0; j < AC; ++j) ra[j] = *reinterpret_cast<const uint4*>(ap[j]);
#pragma unroll
  for (int j = 0; j < BC; ++j) rb[j] = *reinterpret_cast<const uint4*>(bp[j]);
#pragma unroll
  for (int j = 0; j < AC; ++j) *reinterpret_cast<uint4*>(As + al[j]) = ra[j];
#pragma unroll
  for (int j = 0; j < BC; ++j) *reinterpret_cast<uint4*>(Bs + bl[j]) = rb[j];
  __syncthreads();

  const int nk = c.K / BK;
  const int arow = wm * WTM + (lane & 31), brow = wn * WTN + (lane & 31);
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) {
      const int ko = (kt + 1) * BK;
#pragma unroll
      for (int j = 0; j < AC; ++j) ra[j] = *reinterpret_cast<const uint4*>(ap[j] + ko);
#pragma unroll
      for (int j = 0; j < BC; ++j) rb[j] = *reinterpret_cast<const uint4*>(bp[j] + ko);
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int koff = ks * 16 + (lane >> 5) * 8;
      bf16x8 af[FM], bf[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        af[fm] = as_bf16x8(*reinterpret_cast<const uint4*>(As + (arow + fm * 32) * LDK + koff));
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        bf[fn] = as_bf16x8(*reinterpret_cast<const uint4*>(Bs + (brow + fn * 32) * LDK + koff));
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma32(af[fm], bf[fn], acc[fm][fn]);
    }
    __syncthreads();
    if (more) {
#pragma unroll
      for (int j = 0; j < AC; ++j) *reinterpret_cast<uint4*>(As + al[j]) = ra[j];
#pragma unroll
      for (int j = 0; j < BC; ++j) *reinterpret_cast<uint4*>(Bs + bl[j]) = rb[j];
    }
    __syncthreads();
  }

  const int rowb = m0 + wm * WTM, colb = n0 + wn * WTN;
  if constexpr (EPI == EPI_RESIDUAL) epi_residual<FM, FN>(c, acc, rowb, colb, lane);
  else if constexpr (EPI == EPI_STORE_F32) epi_store<FM, FN>(c, acc, rowb, colb, lane);
  else if constexpr (EPI == EPI_SWIGLU) epi_swiglu<FM, FN>(c, acc, rowb, colb, lane);
  else if constexpr (EPI == EPI_QKV_ROPE) epi_qkv_rope<FM, FN>(c, acc, rowb, colb, lane);
  else epi_lmstats<BM, WM, WN, FM, FN>(c, acc, m0, tn, rowb, colb, lane, wm, wn, smem);
}

struct TileCfg {
  int BM, BN, WM, WN;
  int occ;     // workgroups a CU holds at once (registers / LDS)
  float eff;   // relative per-CU matrix-core efficiency when full
};

constexpr TileCfg kTiles[] = {
    {256, 256, 2, 2, 1, 1.00f},
    {128, 256, 2, 2, 1, 0.90f},
    {128, 128, 2, 2, 2, 0.80f},
    {64, 128, 2, 2, 4, 0.60f},
    {32, 256, 1, 4, 3, 0.50f},
};

bool tile_ok(const GemmCall& c, const TileCfg& t) {
  if (c.N % t.BN || c.K % BK) return false;
  const int WTN = t.BN / t.WN;
  switch (c.epi) {
    case EPI_QKV_ROPE:
      // the 256x256 tile spills registers in this epilogue
      return WTN == c.rope.hd && (c.rope.H * c.rope.hd) % t.BN == 0 && t.BM != 32 &&
             t.BM != 256;
    case EPI_SWIGLU:
      return (c.F % (WTN / 2)) == 0 && t.BM != 32;
    case EPI_RESIDUAL:
      return t.BM != 32;
    case EPI_LMSTATS:
    case EPI_STORE_F32:
      return t.BM == 32 || t.BM == 128 || t.BM == 256;
  }
  return false;
}

int pick_tile(const GemmCall& c) {
  int best = -1;
  double best_t = 0;
  for (int i = 0; i < (int)(sizeof(kTiles) / sizeof(kTiles[0])); ++i) {
    const TileCfg& t = kTiles[i];
    if (!tile_ok(c, t)) continue;
    const long tiles = (long)((c.M + t.BM - 1) / t.BM) * (c.N / t.BN);
    const long slots = 256L * t.occ;
    const long rounds = (tiles + slots - 1) / slots;
    const long per_cu = std::min<long>(t.occ, (tiles + 255) / 256);
    const double time = (double)rounds * per_cu * t.BM * t.BN / t.eff;
    if (best < 0 || time < best_t) { best = i; best_t = time; }
  }
  return best;
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_cfg(const GemmCall& c, hipStream_t st) {
  const int tiles = ((c.M + BM - 1) / BM) * (c.N / BN);
  dim3 grid(tiles), block(WM * WN * 64);
  switch (c.epi) {
    case EPI_QKV_ROPE: gemm_kernel<BM, BN, WM, WN, EPI_QKV_ROPE><<<grid, block, 0, st>>>(c); break;
    case EPI_RESIDUAL: gemm_kernel<BM, BN, WM, WN, EPI_RESIDUAL><<<grid, block, 0, st>>>(c); break;
    case EPI_SWIGLU: gemm_kernel<BM, BN, WM, WN, EPI_SWIGLU><<<grid, block, 0, st>>>(c); break;
    case EPI_LMSTATS: gemm_kernel<BM, BN, WM, WN, EPI_LMSTATS><<<grid, block, 0, st>>>(c); break;
    case EPI_STORE_F32: gemm_kernel<BM, BN, WM, WN, EPI_STORE_F32><<<grid, block, 0, st>>>(c); break;
  }
  return hipGetLastError();
}

}  // namespace

int gemm_tile_n(const GemmCall& c) {
  const int i = pick_tile(c);
  return i < 0 ? 0 : kTiles[i].BN;
}

hipError_t launch_gemm(const GemmCall& c, hipStream_t st) {
  const int i = pick_tile(c);
  if (i < 0) return hipErrorInvalidValue;
  if (c.M <= 0) return hipSuccess;
  switch (i) {
    case 0: return launch_cfg<256, 256, 2, 2>(c, st);
    case 1: return launch_cfg<128, 256, 2, 2>(c, st);
    case 2: return launch_cfg<128, 128, 2, 2>(c, st);
    case 3: return launch_cfg<64, 128, 2, 2>(c, st);
    case 4: return launch_cfg<32, 256, 1, 4>(c, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace wino
