// GEMM C = A * W^T on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16, or the
// _f16 form when activations and weights are fp16), with the epilogues of the
// WINO forward fused in:
//   QKV projection + rotate-half RoPE at the WINO position ids,
//   residual add into the fp32 stream (O projection, FFN down projection),
//   SwiGLU of interleaved gate/up tiles,
//   LM head + per-tile softmax statistics (max, sum-exp, best non-mask id,
//   logit of the current token) so the logits never reach memory,
//   plain fp32 store (+bias) for the test entry point.
//
// The LM-head epilogues read the final hidden rows as two 16-bit parts (hi and
// lo of the fp32 value) and multiply both with the same W tile, so the logits
// carry ~16 (bf16) or ~22 (fp16) mantissa bits of the hidden state.
//
// Tiling: a workgroup owns a BM x BN output tile and walks K in steps of 64.
// A and W tiles go straight from global memory into LDS (gfx950 LDS-DMA,
// global_load_lds_dwordx4: no staging registers), double-buffered so the next
// K step streams in while the matrix cores consume the current one.  Within a
// tile row the 16-byte chunks are XOR-swizzled by the row index, so the
// fragment reads of 8 consecutive rows hit distinct bank groups.  Waves form a WM x WN grid, each owning a
// (BM/WM) x (BN/WN) sub-tile of 32x32 MFMA blocks.  Workgroups are renumbered
// so that each XCD works on one contiguous range of tiles (shared W tiles stay
// in that XCD's L2).
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdlib>
#include <mutex>
#include <type_traits>

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

// The fp32 epilogues through the wave's LDS region (free once the K loop has
// drained): one 32-row block of accumulators at a time goes to LDS in the
// MFMA layout and comes back as 16-byte row chunks, so x (residual: read, add,
// write) or the partial buffer moves in 16-byte accesses - a quarter of the
// memory instructions of the 4-byte accesses straight from the MFMA layout.
// op(row, col, float4 v) gets 4 consecutive columns of one row.
template <int FM, int FN, class Op>
__device__ __forceinline__ void epi_rows16(f32x16 (&acc)[FM][FN], int lane, float* ws, Op op) {
  constexpr int WTN = FN * 32, C4 = WTN / 4;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i) ws[mfma_row(i, lane) * WTN + fn * 32 + (lane & 31)] = acc[fm][fn][i];
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int it = 0; it < 32 * C4 / 64; ++it) {
      const int idx = it * 64 + lane, r = idx / C4, c4 = idx - (idx / C4) * C4;
      op(fm * 32 + r, c4 * 4, *reinterpret_cast<const float4*>(ws + r * WTN + c4 * 4));
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

// x += acc for a wave tile whose rows all lie below M, through the wave's LDS
// region like epi_rows16: a 32-row block's x loads all go out before its
// adds and stores (in program order, so the compiler need not prove the
// runtime-strided stores and loads apart, and one memory round trip covers
// the block instead of one per 16-byte chunk).  xb: the tile's x at
// (rowb, colb), the same in every lane.
template <int FM, int FN>
__device__ __forceinline__ void epi_residual_full(f32x16 (&acc)[FM][FN], int lane, float* ws, float* xb,
                                                  int ldc) {
  constexpr int WTN = FN * 32, C4 = WTN / 4, IT = 32 * C4 / 64;
  const int r0 = lane / C4, c4 = lane % C4;
  float* xl = xb + (size_t)r0 * ldc + c4 * 4;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    float4 xv[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it)
      xv[it] = *reinterpret_cast<const float4*>(xl + (size_t)(fm * 32 + it * (64 / C4)) * ldc);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i) ws[mfma_row(i, lane) * WTN + fn * 32 + (lane & 31)] = acc[fm][fn][i];
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const float4 v = *reinterpret_cast<const float4*>(ws + (it * (64 / C4) + r0) * WTN + c4 * 4);
      float4 x = xv[it];
      x.x += v.x; x.y += v.y; x.z += v.z; x.w += v.w;
      *reinterpret_cast<float4*>(xl + (size_t)(fm * 32 + it * (64 / C4)) * ldc) = x;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

// K-slice `split` of a tile above split_row0: fp32 partial
// part[split][m - split_row0][n] (row stride N), summed into x later.
template <int FM, int FN>
__device__ __forceinline__ void epi_partial(const GemmCall& c, f32x16 (&acc)[FM][FN], int rowb,
                                            int colb, int lane, int split) {
  const size_t mt = (size_t)(c.M - c.split_row0);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int row = rowb + fm * 32 + mfma_row(i, lane);
      if (row >= c.M) continue;
      float* dst = c.part + (split * mt + (row - c.split_row0)) * c.N + colb + (lane & 31);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) dst[fn * 32] = acc[fm][fn][i];
    }
}

// out = silu(gate) * up = g u / (1 + 2^(-g log2 e)), with the hardware exp2
// and reciprocal (about 1 ulp of fp32 each, far below the bf16 rounding that
// follows; an IEEE divide is ~10 VALU instructions per element, and the
// epilogue runs while the matrix cores of the CU idle).  Stores are buffer
// stores: the row offset of each accumulator register is wave-uniform and
// goes in a scalar register, the lane's column in the vector offset.  In a
// tile that crosses the last row, rows past it get an offset beyond the
// buffer range, which drops their stores.
template <class A, int FM, int FN>
__device__ __forceinline__ void epi_swiglu(const GemmCall& c, f32x16 (&acc)[FM][FN], int rowb,
                                           int colb, int lane) {
  constexpr int H2 = FN / 2, WTM = FM * 32;
  // wave-uniform: the resource and the row offsets live in scalar registers
  rowb = __builtin_amdgcn_readfirstlane(rowb);
  colb = __builtin_amdgcn_readfirstlane(colb);
  if (rowb >= c.M) return;
  const int nrows = min(c.M - rowb, WTM), ld2 = c.ldc * 2;
  const auto rs = __builtin_amdgcn_make_buffer_rsrc(c.outh + (size_t)rowb * c.ldc + colb / 2, (short)0,
                                                    nrows * ld2, kBufferDword3);
  const int lrow = 4 * (lane >> 5);
  const int voff = lrow * ld2 + (lane & 31) * 2;
  auto body = [&](auto full) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int srow = fm * 32 + 8 * (i >> 2) + (i & 3);
        int vo = voff;
        if constexpr (!decltype(full)::value) vo = srow + lrow < nrows ? voff : kBufferOffNone;
#pragma unroll
        for (int fn = 0; fn < H2; ++fn) {
          const float g = acc[fm][fn][i], u = acc[fm][fn + H2][i];
          const float sg = __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(g * -1.44269504088896341f));
          __builtin_amdgcn_raw_buffer_store_b16(A::cvt(g * u * sg), rs, vo + fn * 64, srow * ld2, 0);
        }
      }
  };
  if (nrows == WTM) body(std::true_type{});
  else body(std::false_type{});
}

// Sequence b and position t of row rowb + lr of a wave's tile (rows are
// sequence-major, T per sequence).  TWO: the sequences are at least as long
// as the tile, so it spans at most two of them - one division per wave and a
// compare per row instead of a division per row.
template <bool TWO>
struct TileRows {
  int b0, t0, T;
  __device__ __forceinline__ TileRows(int rowb, int T_) : T(T_) {
    b0 = rowb / T;
    t0 = rowb - b0 * T;
  }
  __device__ __forceinline__ void at(int lr, int& b, int& t) const {
    if constexpr (TWO) {
      t = t0 + lr;
      const bool nx = t >= T;
      t = nx ? t - T : t;
      b = b0 + (int)nx;
    } else {
      const int r = b0 * T + t0 + lr;
      b = r / T;
      t = r - b * T;
    }
  }
};

// Wave columns = one head (WTN == hd): lane holds columns e and e + hd/2 of
// the rotate-half pair in fragments fn and fn + FN/2.  The wave's rotated q/k
// rows (or its v columns, transposed) are staged in the wave's own LDS region
// of WTM x hd bf16 and leave in 16-byte stores: whole q/k rows of hd elements,
// and runs of 8 consecutive positions of v^T.  Storing v^T straight from the
// MFMA layout would scatter 2-byte writes over hd rows of the transposed
// buffer.  16-byte chunks are XOR-swizzled by the row index, so the
// half-waves' writes (4 rows apart) land in distinct banks.
template <class A, int FM, int FN, bool TWO>
__device__ __forceinline__ void epi_qkv_rope(const GemmCall& c, f32x16 (&acc)[FM][FN], int rowb,
                                             int colb, int lane, uint16_t* ws) {
  constexpr int H2 = FN / 2;
  constexpr int WTM = FM * 32, HD = FN * 32;
  constexpr int QCH = HD / 8;   // 16-byte chunks per q/k row (power of two)
  constexpr int VCH = WTM / 8;  // 16-byte chunks per v^T row
  // v^T rows are 2*VCH slots of 8 bytes; slot s of row e sits at s ^ m(e),
  // m(e) = (e >> 1) & SMASK, so 32 consecutive rows written at one slot
  // cover 64 distinct banks.  A 16-byte chunk stays whole (its halves swap
  // when m(e) is odd).
  constexpr int SL = 2 * VCH;
  constexpr int SMASK = SL % 16 == 0 ? 15 : SL % 8 == 0 ? 7 : SL % 4 == 0 ? 3 : 1;
  static_assert((QCH & (QCH - 1)) == 0 && 64 % QCH == 0, "q/k chunking");
  static_assert((HD * VCH) % 64 == 0, "v^T chunking");
  const RopeOut& ro = c.rope;
  const StepGeom& g = c.geom;
  // wave-uniform: store bases and row offsets live in scalar registers
  rowb = __builtin_amdgcn_readfirstlane(rowb);
  colb = __builtin_amdgcn_readfirstlane(colb);
  const int half = HD / 2;
  const int d = ro.H * HD;
  const int which = colb / d;               // 0 q, 1 k, 2 v
  const int head = (colb - which * d) / HD;
  if (rowb >= c.M) return;  // a wave wholly past the last row
  const TileRows<TWO> tr(rowb, g.T);
  // the wave's first sequence and position, marked uniform (the division
  // runs on the vector unit) so the store bases below stay scalar
  const int b0u = __builtin_amdgcn_readfirstlane(tr.b0), t0u = __builtin_amdgcn_readfirstlane(tr.t0);
  // A wave whose rows are all normal rows of one sequence has position = t:
  // its table rows follow one base pointer at constant offsets, and each lane
  // writes its two rotated values (elements e and e + 64) as 16-bit stores.
  // The staged layout is the general path's: element e of row r in 16-byte
  // chunk (e >> 3) ^ (r & 15).  With r = lrc + 4*g (lrc the row's constant
  // part, g = lane / 32) that chunk is c8 | ((fn ^ g) << 2) | (q ^ (i & 3)),
  // q = (lane & 31) / 8, c8 = bit 3 of lrc, and element e + 64 flips bit 3:
  // a per-lane base and a compile-time offset for every store.
  bool plain = false;
  if constexpr (TWO && HD == 128) plain = which < 2 && tr.t0 + WTM <= g.S;
  if (plain) {
    const int g4 = lane >> 5, q8 = (lane & 31) >> 3;
    const float* tb = ro.tab + ((size_t)(t0u + 4 * g4) * 32 + (lane & 31)) * 4;
    uint16_t* wl = ws + 4 * g4 * HD + (lane & 7);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int i3 = i & 3, c8 = 8 * ((i >> 2) & 1);
        const int lrc = fm * 32 + 8 * (i >> 2) + i3;
        const float4 t4 = *reinterpret_cast<const float4*>(tb + (size_t)lrc * 128);
        const float cst[4] = {t4.x, t4.y, t4.z, t4.w};
#pragma unroll
        for (int fn = 0; fn < 2; ++fn) {
          const float cs = cst[2 * fn], sn = cst[2 * fn + 1];
          const float x1 = acc[fm][fn][i], x2 = acc[fm][fn + 2][i];
          const float r1 = fmaf(x1, cs, -(x2 * sn));  // element e
          const float r2 = fmaf(x2, cs, x1 * sn);     // element e + hd/2
          const uint32_t pk = A::pack2(r1, r2);
          uint16_t* row = wl + lrc * HD + (((((fn ^ g4) << 2) | (q8 ^ i3))) << 3);
          row[c8 << 3] = (uint16_t)pk;
          row[(c8 ^ 8) << 3] = (uint16_t)(pk >> 16);
        }
      }
  } else if (which < 2) {
    // block starts of the wave's first two sequences (the second clamped to
    // the batch: rows past the last compute a valid but unused position)
    const int cs0 = cur_start(g, tr.b0), cs1 = cur_start(g, min(tr.b0 + 1, g.B - 1));
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        // rows past the last are staged too (their q/k never leave LDS)
        const int lr = fm * 32 + mfma_row(i, lane);
        int b, t;
        tr.at(lr, b, t);
        int pos = t;
        if (t >= g.S) {
          if constexpr (TWO) pos = (b == tr.b0 ? cs0 : cs1) + (t - g.S);
          else pos = cur_start(g, min(b, g.B - 1)) + (t - g.S);
        }
        uint16_t* wr = ws + lr * HD;
        const int sw = lr & (QCH - 1);
        float cst[2 * H2];  // (cos, sin) of elements fn*32 + (lane & 31)
        const float* tp = ro.tab + ((size_t)pos * 32 + (lane & 31)) * (2 * H2);
        if constexpr (H2 == 2) {
          const float4 t4 = *reinterpret_cast<const float4*>(tp);
          cst[0] = t4.x; cst[1] = t4.y; cst[2] = t4.z; cst[3] = t4.w;
        } else {
#pragma unroll
          for (int j = 0; j < H2; ++j) {
            const float2 t2 = *reinterpret_cast<const float2*>(tp + 2 * j);
            cst[2 * j] = t2.x; cst[2 * j + 1] = t2.y;
          }
        }
#pragma unroll
        for (int fn = 0; fn < H2; ++fn) {
          const int e = fn * 32 + (lane & 31);
          const float cs = cst[2 * fn], sn = cst[2 * fn + 1];
          const float x1 = acc[fm][fn][i], x2 = acc[fm][fn + H2][i];
          // explicit FMAs: the rounding does not depend on how the compiler
          // contracts the products
          const float r1 = fmaf(x1, cs, -(x2 * sn));  // element e
          const float r2 = fmaf(x2, cs, x1 * sn);     // element e + hd/2
          // lane pairs trade one value: the even lane stores elements e, e+1,
          // the odd lane elements e+hd/2-1, e+hd/2 (one 4-byte write each)
          const bool odd = lane & 1;
          // (lane ^ 1 by a DPP quad swap, no LDS round trip)
          const float got = __uint_as_float(dpp_mov<0xB1>(__float_as_uint(odd ? r1 : r2)));
          const int ee = odd ? e + half - 1 : e;
          const uint32_t pk = odd ? A::pack2(got, r2) : A::pack2(r1, got);
          *reinterpret_cast<uint32_t*>(wr + (((ee >> 3) ^ sw) << 3) + (ee & 7)) = pk;
        }
      }
  }
  if (which < 2) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    uint16_t* base = which == 0 ? ro.q : ro.k;
    constexpr int RPI = 64 / QCH;  // rows per pass
    if (tr.t0 + WTM <= g.T && rowb + WTM <= c.M) {
      // the wave's rows are one contiguous block of one sequence: 16-byte
      // stores from a wave-uniform base at per-lane plus constant offsets
      // (no per-row position, address or bounds arithmetic).  Not buffer
      // stores with the row offset in a scalar register: after such a 16-byte
      // store the compiler let the next instruction overwrite its data
      // register with no wait state, and one dword of it was lost.
      const size_t bh = (size_t)b0u * ro.H + head;
      uint16_t* dst = uniform_ptr(base + (bh * g.Tp + t0u) * HD);
      const int lrl = lane / QCH, ch = lane & (QCH - 1);
      uint16_t* dl = dst + lrl * HD + ch * 8;
#pragma unroll
      for (int it = 0; it < WTM / RPI; ++it) {
        const int lr = it * RPI + lrl;
        const uint4 v = *reinterpret_cast<const uint4*>(ws + lr * HD + ((ch ^ (lr & (QCH - 1))) << 3));
        *reinterpret_cast<uint4*>(dl + it * RPI * HD) = v;
      }
    } else {
#pragma unroll
    for (int it = 0; it < WTM / RPI; ++it) {
      const int lr = it * RPI + lane / QCH, ch = lane & (QCH - 1);
      if (rowb + lr >= c.M) continue;
      int b, t;
      tr.at(lr, b, t);
      const size_t bh = (size_t)b * ro.H + head;
      const uint4 v = *reinterpret_cast<const uint4*>(ws + lr * HD + ((ch ^ (lr & (QCH - 1))) << 3));
      *reinterpret_cast<uint4*>(base + (bh * g.Tp + t) * HD + ch * 8) = v;
    }
    }
  } else {
    // v^T staging: LDS row e holds the WTM positions of this wave; lane writes
    // the 4 consecutive positions 8*(i/4) + 4*(lane/32) + 0..3 of fragment fm.
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int e = fn * 32 + (lane & 31);
      uint16_t* wr = ws + e * WTM;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int tl = fm * 32 + 8 * q + 4 * (lane >> 5);
          uint2 v;
          v.x = A::pack2(acc[fm][fn][4 * q], acc[fm][fn][4 * q + 1]);
          v.y = A::pack2(acc[fm][fn][4 * q + 2], acc[fm][fn][4 * q + 3]);
          const int slot = (tl >> 2) ^ ((e >> 1) & SMASK);
          *reinterpret_cast<uint2*>(wr + slot * 4) = v;
        }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (tr.t0 + WTM <= g.T && rowb + WTM <= c.M && (tr.t0 & 7) == 0) {
      // one sequence, no row past M, 16-byte aligned runs: the head's v^T
      // rows from a wave-uniform base (position t0) at per-lane offsets
      constexpr int EPP = 64 / VCH;  // v^T rows per pass
      const size_t bh = (size_t)b0u * ro.H + head;
      uint16_t* dst = uniform_ptr(ro.vt + bh * HD * g.Tp + t0u);
      const int el = lane / VCH, ch = lane % VCH;
      uint16_t* dl = dst + (size_t)el * g.Tp + ch * 8;
#pragma unroll
      for (int it = 0; it < HD * VCH / 64; ++it) {
        const int e = it * EPP + el;
        const int m = (e >> 1) & SMASK;
        uint4 v = *reinterpret_cast<const uint4*>(ws + e * WTM + ((ch ^ (m >> 1)) << 3));
        if (m & 1) v = make_uint4(v.z, v.w, v.x, v.y);
        *reinterpret_cast<uint4*>(dl + (size_t)it * EPP * g.Tp) = v;
      }
      return;
    }
#pragma unroll
    for (int it = 0; it < HD * VCH / 64; ++it) {
      const int idx = it * 64 + lane;
      const int e = idx / VCH, ch = idx - (idx / VCH) * VCH;
      const int m = (e >> 1) & SMASK;
      uint4 v = *reinterpret_cast<const uint4*>(ws + e * WTM + ((ch ^ (m >> 1)) << 3));
      if (m & 1) v = make_uint4(v.z, v.w, v.x, v.y);
      const int r0 = rowb + ch * 8;
      if (r0 >= c.M) continue;
      int b, t0;
      tr.at(ch * 8, b, t0);
      if (r0 + 7 < c.M && t0 + 7 < g.T && (t0 & 7) == 0) {
        const size_t bh = (size_t)b * ro.H + head;
        *reinterpret_cast<uint4*>(ro.vt + (bh * HD + e) * g.Tp + t0) = v;
      } else {
        // run crosses a sequence end or the last row, or T is not a multiple
        // of 8: element stores
        const uint16_t* h = reinterpret_cast<const uint16_t*>(&v);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int r = r0 + j;
          if (r >= c.M) break;
          const int bj = r / g.T, tj = r - bj * g.T;
          ro.vt[(((size_t)bj * ro.H + head) * HD + e) * g.Tp + tj] = h[j];
        }
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
  float* red_z = reinterpret_cast<float*>(red_i + WN * BM);  // entropy term (pz only)
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
      // over the 32 lanes (columns) of each half-wave
      mx = valu_max<32>(mx);
      tz = valu_max<32>(tz);
      valu_argmax<32>(bz, bi);
      float se = 0.f, sz = 0.f;
      if (lm.pz) {
        // sum exp(z - m) * (z - m): the entropy's expectation term, relative
        // to the tile max so nothing cancels against a large m
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const float u = acc[fm][fn][i] + bias[fn] - mx;
          const float e = __expf(u);
          se += e;
          sz += e * u;
        }
        se = valu_sum<32>(se);
        sz = valu_sum<32>(sz);
      } else {
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) se += __expf(acc[fm][fn][i] + bias[fn] - mx);
        se = valu_sum<32>(se);
      }
      if ((lane & 31) == 0) {
        red_m[wn * BM + lrow] = mx;
        red_s[wn * BM + lrow] = se;
        red_b[wn * BM + lrow] = bz;
        red_t[wn * BM + lrow] = tz;
        red_i[wn * BM + lrow] = bi;
        if (lm.pz) red_z[wn * BM + lrow] = sz;
      }
    }
  __syncthreads();
  for (int r = threadIdx.x; r < BM; r += WM * WN * 64) {
    const int row = m0 + r;
    if (row >= c.M) continue;
    float m = kNegBig;
#pragma unroll
    for (int w = 0; w < WN; ++w) m = fmaxf(m, red_m[w * BM + r]);
    float s = 0.f, z = 0.f, bz = kNegBig, tz = kNegBig;
    int bi = INT_MAX;
#pragma unroll
    for (int w = 0; w < WN; ++w) {
      const float dm = red_m[w * BM + r] - m, f = __expf(dm);
      s += red_s[w * BM + r] * f;
      // sum e^{z-m}(z-m) = e^{m_w-m} (sum e^{z-m_w}(z-m_w) + (m_w-m) sum e^{z-m_w})
      if (lm.pz) z += f * (red_z[w * BM + r] + dm * red_s[w * BM + r]);
      const float ob = red_b[w * BM + r];
      const int oi = red_i[w * BM + r];
      if (ob > bz || (ob == bz && oi < bi)) { bz = ob; bi = oi; }
      tz = fmaxf(tz, red_t[w * BM + r]);
    }
    const size_t o = (size_t)row * lm.n_part + tn;
    if (lm.pz) lm.pz[o] = z;
    lm.pm[o] = m;
    lm.ps[o] = s;
    lm.pb[o] = bz;
    lm.pi[o] = bi;
    lm.pt[o] = tz;
  }
}

// Physical 16-byte position of chunk kc of LDS tile row r: rows of KB bf16
// (KB/8 chunks) are XOR-swizzled so the fragment reads of 8 or 16
// consecutive rows at one chunk hit distinct bank groups.
//   KB = 64 (128-byte rows): kc ^ ((r ^ (r >> 3)) & 7): any 8 consecutive rows
//     use 8 positions, any 16 rows 16 (row parity, position) pairs.
//   KB = 32 (64-byte rows, 4 per 64 banks): kc ^ ((r >> 2) & 3): 16
//     consecutive rows give 16 distinct (r mod 4, position) pairs.
template <int KB>
__device__ __forceinline__ int lds_swz(int r) {
  if constexpr (KB == 64) return (r ^ (r >> 3)) & 7;
  else return (r >> 2) & 3;
}

// OCC workgroups per CU: the launch bound asks for OCC * waves / 4 waves per
// SIMD, which caps the registers per wave accordingly.  XW > 0 gives the W
// tiles XW more LDS stages than the two of A, so W copies have 1 + XW K
// steps to land instead of one (for weights that few row tiles share, whose
// copies mostly miss L2).
template <int BM, int BN, int WM, int WN, int EPI, int KB, int NST, int OCC, int XW, class A>
__global__ __launch_bounds__(WM* WN * 64, (OCC * WM * WN + 3) / 4) void gemm_kernel(const GemmCall c) {
  static_assert(KB == 32 || KB == 64, "K step");
  static_assert(NST >= 2, "pipeline stages");
  static_assert(XW == 0 || (XW <= 2 && NST == 2), "extra W stages beside two A stages");
  constexpr int NW = WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  // LM-head epilogues multiply W with both bf16 parts (hi, lo) of the fp32 rows
  constexpr bool SPLIT = EPI == EPI_LMSTATS || EPI == EPI_LOGITS;
  constexpr int AROWS = SPLIT ? 2 * BM : BM;
  // one LDS-DMA instruction moves 64 lanes x 16 bytes = 1 KB = RPI tile rows
  constexpr int CPR = KB / 8;    // 16-byte chunks per tile row
  constexpr int RPI = 64 / CPR;  // tile rows per DMA instruction
  constexpr int A_INS = AROWS / (RPI * NW);
  constexpr int B_INS = BN / (RPI * NW);
  constexpr int INS = A_INS + B_INS;
  static_assert(A_INS * RPI * NW == AROWS && B_INS * RPI * NW == BN, "loader split");
  static_assert(FM >= 1 && FN >= 1, "wave tile");
  constexpr int NSB = NST + XW;  // W stages
  constexpr int A_STAGE = AROWS * KB, B_STAGE = BN * KB;  // bf16 elements per stage
  constexpr int LDS_ELEMS = NST * A_STAGE + NSB * B_STAGE;  // A stages, then W stages

  __shared__ __attribute__((aligned(1024))) uint16_t smem[LDS_ELEMS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave - (wave / WN) * WN;
  // Tile order: each XCD takes a contiguous range of logical tiles, walked in
  // groups of GM M-tiles so the ~32 workgroups an XCD runs at once cover
  // GM A tiles x (32/GM) W tiles and reuse both from its L2.
  // Work units: whole-K tiles of the full row tiles first, then the rest:
  // with the residual epilogue and splits > 1, `splits` K-slices of each
  // tile from split_row0 on (a last partial round of whole tiles becomes a
  // full round of thin slices); otherwise the partial last row tile, whose
  // waves past M skip their MFMAs - these finish early, so they go last and
  // fill the CUs the full tiles leave free.
  constexpr int GM = 8;
  const int nTM = (c.M + BM - 1) / BM, nTN = c.N / BN;
  const bool ksplit = EPI == EPI_RESIDUAL && c.splits > 1;
  const int mainTM = ksplit ? c.split_row0 / BM : c.M / BM;
  const int n_main = mainTM * nTN;
  const bool tail = (int)blockIdx.x >= n_main;
  const int tailTM = nTM - mainTM;
  const int u = tail ? xcd_remap(blockIdx.x - n_main, gridDim.x - n_main)
                     : xcd_remap(blockIdx.x, n_main);
  const int split = tail ? u / (tailTM * nTN) : 0;
  const int t = tail ? u - split * (tailTM * nTN) : u;
  const int rTM = tail ? tailTM : mainTM;
  const int first_m = (t / (GM * nTN)) * GM;
  const int gsz = min(rTM - first_m, GM);
  const int tm = (tail ? mainTM : 0) + first_m + (t % (GM * nTN)) % gsz;
  const int tn = (t % (GM * nTN)) / gsz;
  const int Ku = ksplit && tail ? c.K / c.splits : c.K;  // K depth of this unit
  const int m0 = tm * BM, n0 = tn * BN;

  // The lane that fills position (lane % CPR) of row RPI*i + lane/CPR of a
  // tile fetches the chunk that belongs there: position ^ lds_swz(row).
  const int lrow = lane / CPR, lpos = lane % CPR;
  const int kbase = split * Ku;  // first K column of this unit
  // In a partial row tile (8-wave shapes; the 4-wave ones would need more
  // registers for the extra code paths) a wave skips the MFMAs of its rows
  // past M and the copies of A rows past M (they feed only output rows past
  // M); with two stages every later wait is for all of a wave's copies, so
  // only the first wait changes.
  constexpr bool CAN_SKIP = NST == 2 && !SPLIT && NW == 8;  // (W copies are never skipped)
  constexpr bool BIG2 = NW == 8 && BM == 256 && BN == 256 && XW == 0;
  constexpr int CROSS = BIG2 ? 3 : 1;
  static_assert(CROSS != 3 || (XW == 0 && NST == 2), "the W-first crossing relies on waiting for every copy");
  bool alive[A_INS];
  const uint16_t* asrc[A_INS];
#pragma unroll
  for (int i = 0; i < A_INS; ++i) {
    alive[i] = m0 + (wave * A_INS + i) * RPI < c.M;
    const int gi = wave * A_INS + i;
    const int row = gi * RPI + lrow;
    const int lkc = lpos ^ lds_swz<KB>(row);
    const bool lo = SPLIT && row >= BM;
    const int gm = min(m0 + (lo ? row - BM : row), c.M - 1);
    asrc[i] = (lo ? c.A2 : c.A) + (size_t)gm * c.lda + kbase + lkc * 8;
  }
  const uint16_t* bsrc[B_INS];
#pragma unroll
  for (int i = 0; i < B_INS; ++i) {
    const int gi = wave * B_INS + i;
    const int lkc = lpos ^ lds_swz<KB>(gi * RPI + lrow);
    const int vc = n0 + gi * RPI + lrow;
    const int wr = EPI == EPI_SWIGLU ? swiglu_row<WTN>(vc, c.F) : vc;
    bsrc[i] = c.W + (size_t)wr * c.ldw + kbase + lkc * 8;
  }

  // A wave's copies land in consecutive 1 KB blocks; groups of four share
  // one LDS base (M0) and differ in the instruction offset.
  auto stage_a = [&](int s) { return smem + s * A_STAGE; };
  auto stage_b = [&](int s) { return smem + NST * A_STAGE + s * B_STAGE; };
  auto issue_a = [&](int kt, int stage, auto skip_tag) {
    uint16_t* sA = stage_a(stage);
#pragma unroll
    for (int i = 0; i < A_INS; ++i)
      if (!decltype(skip_tag)::value || alive[i])
        dma16(asrc[i] + kt * KB - (i & 3) * 512, sA + (wave * A_INS + (i & ~3)) * 512, i & 3);
  };
  auto issue_b = [&](int kt, int stage) {
    uint16_t* sB = stage_b(stage);
#pragma unroll
    for (int i = 0; i < B_INS; ++i)
      dma16(bsrc[i] + kt * KB - (i & 3) * 512, sB + (wave * B_INS + (i & ~3)) * 512, i & 3);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[fm][fn][i] = 0.f;

  const int nk = Ku / KB;
  const int arow = wm * WTM + (lane & 31), brow = wn * WTN + (lane & 31);
  // swizzle of each fragment row this lane reads (fixed over the K loop)
  int aswz[FM], alswz[SPLIT ? FM : 1], bswz[FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int r = arow + fm * 32;
    aswz[fm] = lds_swz<KB>(r);
    if constexpr (SPLIT) alswz[fm] = lds_swz<KB>(BM + r);
  }
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int r = brow + fn * 32;
    bswz[fn] = lds_swz<KB>(r);
  }
  constexpr int KS = KB / 16;
  static_assert(KS % 2 == 0, "fragment buffers alternate per step");
  typename A::v8 af[2][FM], bf[2][FN], al[2][SPLIT ? FM : 1];

  // The K loop for a wave whose first FMV of its FM 32-row blocks hold rows
  // below M (FMV = FM everywhere but in a partial last row tile): the other
  // blocks' fragment reads and MFMAs are skipped; the wave still issues its
  // share of the tile copies and meets every barrier.
  auto pipeline = [&](auto fmv_tag, auto skip_tag) {
  constexpr int FMV = decltype(fmv_tag)::value;
  constexpr bool SKIP = decltype(skip_tag)::value;
  constexpr int NR = FMV ? FMV + FN + (SPLIT ? FMV : 0) : 0;  // LDS fragment reads per 16-deep step
  constexpr int NM = FMV * FN * (SPLIT ? 2 : 1);              // MFMAs per step
  constexpr int RI = NR < NM ? NR : NM;                       // reads interleaved with MFMAs
  auto load_frags = [&](const uint16_t* sA, const uint16_t* sB, int ks, int buf) {
    if constexpr (FMV > 0) {
    const int kc = ks * 2 + (lane >> 5);
#pragma unroll
    for (int fm = 0; fm < FMV; ++fm)
      af[buf][fm] = A::frag(*reinterpret_cast<const uint4*>(
          sA + (arow + fm * 32) * KB + ((kc ^ aswz[fm]) << 3)));
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
      bf[buf][fn] = A::frag(*reinterpret_cast<const uint4*>(
          sB + (brow + fn * 32) * KB + ((kc ^ bswz[fn]) << 3)));
    if constexpr (SPLIT) {
#pragma unroll
      for (int fm = 0; fm < FMV; ++fm)
        al[buf][fm] = A::frag(*reinterpret_cast<const uint4*>(
            sA + (BM + arow + fm * 32) * KB + ((kc ^ alswz[fm]) << 3)));
    }
    }
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int fm = 0; fm < FMV; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = A::mma(af[buf][fm], bf[buf][fn], acc[fm][fn]);
    if constexpr (SPLIT) {
#pragma unroll
      for (int fm = 0; fm < FMV; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = A::mma(al[buf][fm], bf[buf][fn], acc[fm][fn]);
    }
  };
  // steps 0..KS-2 of a tile: the reads of step ks+1 go between the MFMAs of ks
  auto inner_steps = [&](const uint16_t* sA, const uint16_t* sB) {
#pragma unroll
    for (int ks = 0; ks + 1 < KS; ++ks) {
      load_frags(sA, sB, ks + 1, (ks + 1) & 1);
      mfmas(ks & 1);
    }
    if constexpr (NR > 0) {
#pragma unroll
    for (int ks = 0; ks + 1 < KS; ++ks) {
#pragma unroll
      for (int r = 0; r < RI; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      if (NR > RI) __builtin_amdgcn_sched_group_barrier(0x100, NR - RI, 0);
      if (NM > RI) __builtin_amdgcn_sched_group_barrier(0x008, NM - RI, 0);
    }
    }
  };

  // Pipeline over NST LDS stages: K tile t sits in stage t % NST and its DMA
  // is issued NST tiles ahead.  Crossing from tile t to t+1, each wave (1)
  // waits for its copies of tile t+1 (the NST-2 later tiles may still be in
  // flight), (2) meets the others at the barrier - after which every wave
  // has read all of tile t, (3) issues the first fragment reads of tile t+1
  // and tile t+NST's copy into tile t's stage, and (4) runs the last MFMAs
  // of tile t, which cover the latency of those reads.  The order of the
  // reads, the copies and the MFMAs at that crossing (CROSS) is measured per
  // tile against copies-then-reads: 1 = reads, copies, MFMAs (544-row
  // gate/up 112 -> 100 us); 3 = W copy, reads, A copy, MFMAs for the
  // two-stage 8-wave 256x256 tile (8704 rows, runs alternating with 1:
  // gate/up 1359 -> 1339 us, QKV 724 -> 711 us, down 713 -> 702 us).  3 needs the wait for every copy of
  // the two-stage tile: with a third W stage the waits count on A copies
  // being issued before W copies at each crossing.  Tiles past
  // the end are refetches of the last one, which keeps the wait counts fixed.
  // With XW extra W stages the crossing issues the A copy of tile t+2 and the
  // W copy of tile t+2+XW, and the copies are ordered so that one wait for
  // all but the last W copies covers both operands of tile t+1: A0, W0..WXW,
  // A1, W(XW+1) up front, then A(t+2) W(t+2+XW) per crossing (copies
  // complete in issue order).
  auto kclamp = [&](int k) { return k < nk ? k : nk - 1; };
  if constexpr (XW == 0) {
#pragma unroll
    for (int s0 = 0; s0 < NST; ++s0) {
      issue_a(kclamp(s0), s0, skip_tag);
      issue_b(kclamp(s0), s0);
    }
  } else {
    issue_a(0, 0, skip_tag);
#pragma unroll
    for (int s0 = 0; s0 <= XW; ++s0) issue_b(kclamp(s0), s0);
    issue_a(kclamp(1), 1, skip_tag);
    issue_b(kclamp(XW + 1), XW + 1);
  }
  // (a wave that may have skipped copies has fewer in flight: it waits for all)
  if constexpr (SKIP) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (XW == 0) asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NST - 1) * INS) : "memory");
  else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(A_INS + (XW + 1) * B_INS) : "memory");
  __syncthreads();
  load_frags(stage_a(0), stage_b(0), 0, 0);
  int ca = 0, cb = 0;  // stages of tile kt
  for (int kt = 0; kt + 1 < nk; ++kt) {
    inner_steps(stage_a(ca), stage_b(cb));
    if constexpr (XW == 0) asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NST - 2) * INS) : "memory");
    else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(B_INS) : "memory");
    __syncthreads();
    const int na = ca + 1 == NST ? 0 : ca + 1, nb = cb + 1 == NSB ? 0 : cb + 1;
    if constexpr (CROSS == 3) issue_b(kclamp(kt + NSB), cb);
    load_frags(stage_a(na), stage_b(nb), 0, 0);
    if constexpr (CROSS == 1) issue_a(kclamp(kt + NST), ca, skip_tag);
    if constexpr (CROSS == 1) issue_b(kclamp(kt + NSB), cb);
    if constexpr (CROSS == 3) issue_a(kclamp(kt + NST), ca, skip_tag);
    mfmas((KS - 1) & 1);
    if constexpr (NR > 0) {
      __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
    }
    ca = na;
    cb = nb;
  }
  inner_steps(stage_a(ca), stage_b(cb));
  mfmas((KS - 1) & 1);
  };  // pipeline

  using Full = std::integral_constant<int, FM>;
  using Keep = std::false_type;
  const int vrows = c.M - (m0 + wm * WTM);  // rows of this wave's tile below M
  if constexpr (CAN_SKIP) {
    using Skip = std::true_type;
    if (m0 + BM <= c.M) pipeline(Full{}, Keep{});
    else if (vrows <= 0) pipeline(std::integral_constant<int, 0>{}, Skip{});
    else if (FM > 1 && vrows <= 32) pipeline(std::integral_constant<int, 1>{}, Skip{});
    else pipeline(Full{}, Skip{});
  } else {
    pipeline(Full{}, Keep{});
  }
  // the refetch issued last may still be landing: finish it before the
  // epilogue reuses LDS
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  const int rowb = m0 + wm * WTM, colb = n0 + wn * WTN;
  if constexpr (EPI == EPI_RESIDUAL) {
    // a wave's LDS region holds one 32-row fp32 block of its tile
    constexpr bool STAGED = NW * 32 * WTN * 2 <= LDS_ELEMS;
    if constexpr (STAGED) {
      float* ws = reinterpret_cast<float*>(smem + wave * (32 * WTN * 2));
      // (the batched x loads need 64 registers beside the accumulators: only
      // for wave tiles of at most 8 MFMA blocks)
      if (FM * FN <= 8 && !(ksplit && tail) && rowb + WTM <= c.M) {
        const int rbu = __builtin_amdgcn_readfirstlane(rowb), cbu = __builtin_amdgcn_readfirstlane(colb);
        if constexpr (FM * FN <= 8)
          epi_residual_full<FM, FN>(acc, lane, ws, c.outf + (size_t)rbu * c.ldc + cbu, c.ldc);
      } else if (!(ksplit && tail)) {
        epi_rows16<FM, FN>(acc, lane, ws, [&](int lr, int lc, float4 v) {
          const int row = rowb + lr;
          if (row >= c.M) return;
          float4* dst = reinterpret_cast<float4*>(c.outf + (size_t)row * c.ldc + colb + lc);
          float4 x = *dst;
          x.x += v.x; x.y += v.y; x.z += v.z; x.w += v.w;
          *dst = x;
        });
      } else {
        const size_t mt = (size_t)(c.M - c.split_row0);
        epi_rows16<FM, FN>(acc, lane, ws, [&](int lr, int lc, float4 v) {
          const int row = rowb + lr;
          if (row >= c.M) return;
          *reinterpret_cast<float4*>(c.part + (split * mt + (row - c.split_row0)) * c.N + colb + lc) = v;
        });
      }
    } else {
      if (!(ksplit && tail)) epi_residual<FM, FN>(c, acc, rowb, colb, lane);
      else epi_partial<FM, FN>(c, acc, rowb, colb, lane, split);
    }
  }
  else if constexpr (EPI == EPI_STORE_F32 || EPI == EPI_LOGITS) epi_store<FM, FN>(c, acc, rowb, colb, lane);
  else if constexpr (EPI == EPI_SWIGLU) epi_swiglu<A, FM, FN>(c, acc, rowb, colb, lane);
  else if constexpr (EPI == EPI_QKV_ROPE) {
    // each wave stages its WTM x WTN tile in its own LDS region
    static_assert(BM * BN <= LDS_ELEMS, "QKV staging fits the pipeline LDS");
    if (c.geom.T >= WTM) epi_qkv_rope<A, FM, FN, true>(c, acc, rowb, colb, lane, smem + wave * (WTM * WTN));
    else epi_qkv_rope<A, FM, FN, false>(c, acc, rowb, colb, lane, smem + wave * (WTM * WTN));
  }
  else epi_lmstats<BM, WM, WN, FM, FN>(c, acc, m0, tn, rowb, colb, lane, wm, wn, smem);
}

struct TileCfg {
  int BM, BN, WM, WN;
  int KB, NST;  // K step of a pipeline stage, number of LDS stages
  int occ;      // workgroups a CU holds at once (LDS / registers)
  float eff;    // relative per-CU matrix-core throughput when the chip is full
                // (measured on the 8704x24576x4096 gate/up shape)
  int xw = 0;   // 1: a third LDS stage for the W tiles
};

// eff: measured relative throughput of each shape (8704 x 24576 x 4096, and
// the O / down residual shapes for the 192-row tile, whose single wave per
// SIMD exposes the residual read-add-write).  Deeper pipelines of 32-deep K
// stages and two-per-CU 128x256 tiles were measured slower than entry 6.
// Entry 9 gives the QKV GEMM (a head per wave) two waves per SIMD at few
// rows: 678 vs 598 TFLOP/s at 544 rows.  Entry 4 is set from the 544-row O
// projection (split 2: 40.8 us against 34.6 us for entry 3), where its three
// workgroups per CU are rarely all resident.  Entry 10 keeps two K tiles in
// flight instead of one: at 544 rows each weight strip is read by few row
// tiles, so most of its copies miss L2, and the QKV GEMM takes 66 instead
// of 74 us (weights streamed from HBM); where the weights are shared by many
// row tiles the third stage does not pay (deeper pipelines lost there).
constexpr TileCfg kTiles[] = {
    {256, 256, 2, 2, 64, 2, 1, 0.95f},  // 0
    {192, 256, 2, 2, 64, 2, 1, 0.75f},  // 1
    {128, 256, 2, 2, 64, 2, 1, 0.76f},  // 2
    {128, 128, 2, 2, 64, 2, 2, 0.78f},  // 3
    {64, 128, 2, 2, 64, 2, 3, 0.50f},   // 4
    {32, 256, 1, 4, 64, 2, 2, 0.60f},   // 5
    {256, 256, 4, 2, 64, 2, 1, 1.00f},  // 6  (8 waves)
    {256, 256, 2, 4, 64, 2, 1, 0.98f},  // 7  (8 waves)
    {128, 256, 2, 4, 64, 2, 1, 0.74f},  // 8  (8 waves)
    {128, 256, 4, 2, 64, 2, 1, 0.77f},  // 9  (8 waves, 32-row wave tiles)
    {128, 256, 4, 2, 64, 3, 1, 0.78f},  // 10 (8 waves, three stages)
    {256, 256, 4, 2, 64, 2, 1, 1.00f, 1},  // 11 (8 waves, third W stage)
    {128, 256, 4, 2, 64, 2, 1, 0.77f, 1},  // 12 (8 waves, third W stage)
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

// Which epilogues each tile is built for.  The LM-head epilogues double the A
// tile (hi and lo parts), which fits LDS only for BM <= 128 (the 8-wave
// 128x256 tile: 1.19 -> 0.97 ms for the 512-row LM head); the thin 32-row
// tile serves only them (it loses to wider tiles elsewhere); the 4-wave
// 256x256 tile spills registers in the RoPE epilogue.  (RoPE also needs a
// wave to own exactly one head, WTN == hd: 64 or 128 here, checked per call.)
constexpr bool tile_epi(int BM, int BN, int WM, int WN, int EPI) {
  return (EPI == EPI_LMSTATS || EPI == EPI_LOGITS)
             ? (BM == 32 || (BM == 128 && BN == 256))
             : (BM != 32 && (EPI == EPI_QKV_ROPE ? !(BM == 256 && WM == 2 && WN == 2) &&
                                                       (BN / WN == 64 || BN / WN == 128)
                                                 : true));
}

bool tile_ok(const GemmCall& c, const TileCfg& t) {
  if (c.N % t.BN || c.K % BK) return false;
  if (!tile_epi(t.BM, t.BN, t.WM, t.WN, c.epi)) return false;
  const int arows = (c.epi == EPI_LMSTATS || c.epi == EPI_LOGITS) ? 2 * t.BM : t.BM;
  const int lds_elems = (t.NST * arows + (t.NST + t.xw) * t.BN) * t.KB;
  if (t.xw && (arows != t.BM || t.NST != 2)) return false;
  if (t.occ * lds_elems * 2 > 160 * 1024) return false;
  if (c.epi == EPI_QKV_ROPE && t.BM * t.BN > lds_elems) return false;
  const int WTN = t.BN / t.WN;
  if (c.epi == EPI_QKV_ROPE) return WTN == c.rope.hd && (c.rope.H * c.rope.hd) % t.BN == 0;
  if (c.epi == EPI_SWIGLU) return (c.F % (WTN / 2)) == 0;
  return true;
}

int env_int(const char* name, int dflt) {
  const char* e = std::getenv(name);
  return e ? std::atoi(e) : dflt;
}

// Throughput model: a CU sustains ~6.5 TFLOP/s of bf16 MFMA (~1.7 PFLOP/s
// over 256 CUs) times the tile's relative efficiency, shared by the `occ`
// workgroups it holds; epilogue traffic moves at ~4 TB/s shared by all slots.
constexpr double kCuFlops = 6.5e12, kEpiBw = 4.0e12, kPartBw = 2.5e12;

// Makespan of n_main jobs of length T followed by n_units jobs of length U,
// each started on the slot that frees first (the hardware dispatcher's order).
double makespan(long n_main, double T, long n_units, double U, long slots) {
  const long R = n_main / slots, r = n_main % slots;
  const double main_end = (R + (r ? 1 : 0)) * T;
  if (n_units == 0) return main_end;
  const long early = slots - r;  // slots free at R*T; the other r at (R+1)*T
  double best = 0;
  for (long j = 1;; ++j) {
    const double X = R * T + j * U;
    const long late = r ? (long)std::floor(std::max(0.0, (X - (R + 1) * T) / U) + 1e-9) : 0;
    if (early * j + r * late >= n_units) { best = X; break; }
  }
  if (r) {
    for (long j = 1;; ++j) {
      const double X = (R + 1) * T + j * U;
      if (X >= best) break;
      const long e = (long)std::floor((X - R * T) / U + 1e-9);
      if (early * e + r * j >= n_units) { best = X; break; }
    }
  }
  return std::max(main_end, best);
}

// eff of a tile for a unit of ksteps 64-deep K steps.  A W strip is read by
// the ceil(M / BM) row tiles of its column; at five or fewer most of its
// copies miss L2 and a two-stage pipeline waits on them, which a third W
// stage covers once the unit is long enough to fill it (weights streamed
// from HBM; 544 rows: 256x256 gate/up 138 -> 116 us, 128x256 down 72 -> 65
// us, QKV 70 -> 67 us; 512 rows: gate/up 141 -> 103 us).  Where the
// weights are shared by many row tiles (8704 rows: -1%) or the unit is short
// (K slices of 8-16 steps: 10-17% slower) it does not pay.
double eff_of(const GemmCall& c, const TileCfg& t, int ksteps) {
  if (!t.xw) return t.eff;
  const bool cold = (c.M + t.BM - 1) / t.BM <= 5;
  return cold && ksteps >= 24 ? 1.2 * t.eff : 0.9 * t.eff;
}

// Time of the partial last row tile (rem = M mod BM rows) relative to a full
// one.  8-wave shapes skip the MFMAs of rows past M per wave (the kernel's
// rule: a wave keeps all its 32-row blocks, only the first, or none), so the
// busiest SIMD's remaining share sets the time, floored at kPartialFloor for
// the copies and barriers every wave still makes.  Other shapes: a full tile.
constexpr double kPartialFloor = 0.3;
double partial_share(const GemmCall& c, const TileCfg& t, int rem) {
  const bool lm = c.epi == EPI_LMSTATS || c.epi == EPI_LOGITS;
  if (rem == 0 || lm || t.WM * t.WN != 8 || t.NST != 2) return 1.0;  // (XW tiles skip too)
  const int WTM = t.BM / t.WM, FM = WTM / 32;
  double load[4] = {0, 0, 0, 0};
  for (int w = 0; w < 8; ++w) {
    const int v = rem - (w / t.WN) * WTM;
    const int fmv = v <= 0 ? 0 : (FM > 1 && v <= 32 ? 1 : FM);
    load[w % 4] += (double)fmv / FM;
  }
  const double busiest = std::max(std::max(load[0], load[1]), std::max(load[2], load[3])) / 2.0;
  return std::max(busiest, kPartialFloor);
}

// Estimated seconds for whole-K tiles: the full row tiles, then the partial
// last row tile (the kernel's order), dealt to 256 CUs as they free up (a CU
// holding fewer tiles than it could runs proportionally less efficiently).
double tile_time(const GemmCall& c, const TileCfg& t) {
  const long nTN = c.N / t.BN;
  const int rem = c.M % t.BM;
  const long n_full = (long)(c.M / t.BM) * nTN, n_part = rem ? nTN : 0;
  const long per_cu = std::min<long>(t.occ, (n_full + n_part + 255) / 256);
  const double util = 0.5 + 0.5 * (double)per_cu / t.occ;
  const double tile_s = 2.0 * t.BM * t.BN * (double)c.K / (eff_of(c, t, c.K / BK) * util * kCuFlops);
  return makespan(n_full, tile_s, n_part, partial_share(c, t, rem) * tile_s, 256);
}

// Residual GEMM: whole-K tiles read-add-write 8 bytes of x per output; the
// `splits` K-slices of the last tail_tm row tiles write 4-byte partials that
// the next norm kernel reads back.
double residual_time(const GemmCall& c, const TileCfg& t, int tail_tm, int splits) {
  const int nTM = (c.M + t.BM - 1) / t.BM, nTN = c.N / t.BN;
  const long slots = 256L * t.occ;
  const double rate = eff_of(c, t, c.K / BK) * kCuFlops / t.occ;
  const double out_s = (double)t.BM * t.BN / (kEpiBw / slots);
  const double T = 2.0 * t.BM * t.BN * (double)c.K / rate + 8.0 * out_s;
  const long n_main = (long)(nTM - tail_tm) * nTN;
  if (tail_tm == 0) {
    const int rem = c.M % t.BM;
    return makespan(n_main - (rem ? nTN : 0), T, rem ? nTN : 0, partial_share(c, t, rem) * T, slots);
  }
  const double urate = eff_of(c, t, c.K / splits / BK) * kCuFlops / t.occ;
  const double U = 2.0 * t.BM * t.BN * ((double)c.K / splits + 2 * BK) / urate + 4.0 * out_s;
  const long n_units = (long)tail_tm * nTN * splits;
  const double tail_rows = c.M - (double)(nTM - tail_tm) * t.BM;
  return makespan(n_main, T, n_units, U, slots) + splits * tail_rows * c.N * 4.0 / kPartBw;
}

int pick_tile(const GemmCall& c) {
  const int f = env_int("WINO_GEMM_TILE", -1);
  if (f >= 0 && f < kNumTiles && tile_ok(c, kTiles[f])) return f;
  int best = -1;
  double best_t = 0;
  for (int i = 0; i < kNumTiles; ++i) {
    if (!tile_ok(c, kTiles[i])) continue;
    const double time = tile_time(c, kTiles[i]);
    if (best < 0 || time < best_t) { best = i; best_t = time; }
  }
  return best;
}

struct PlanEntry { int M, N, K; size_t part_elems; int tile, splits, split_row0; };
std::mutex g_plan_mu;
PlanEntry g_plans[32];
int g_n_plans = 0;

template <int BM, int BN, int WM, int WN, int EPI, int KB, int NST, int OCC, int XW, class A>
hipError_t launch_one(const GemmCall& c, hipStream_t st) {
  constexpr bool split = EPI == EPI_LMSTATS || EPI == EPI_LOGITS;
  constexpr int arows = split ? 2 * BM : BM;
  constexpr int lds = (NST * arows + (NST + XW) * BN) * KB * 2;
  constexpr bool qkv_fits = EPI != EPI_QKV_ROPE || BM * BN * 2 <= lds;
  if constexpr (tile_epi(BM, BN, WM, WN, EPI) && lds * OCC <= 160 * 1024 && qkv_fits &&
                (XW == 0 || !split)) {
    const int nTM = (c.M + BM - 1) / BM, nTN = c.N / BN;
    int units = nTM * nTN;
    if (EPI == EPI_RESIDUAL && c.splits > 1) {
      const int mainTM = c.split_row0 / BM;
      units = mainTM * nTN + (nTM - mainTM) * nTN * c.splits;
    }
    gemm_kernel<BM, BN, WM, WN, EPI, KB, NST, OCC, XW, A><<<dim3(units), dim3(WM * WN * 64), 0, st>>>(c);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

template <int BM, int BN, int WM, int WN, int KB, int NST, int OCC, int XW, class A>
hipError_t launch_cfg_t(const GemmCall& c, hipStream_t st) {
  switch (c.epi) {
    case EPI_QKV_ROPE: return launch_one<BM, BN, WM, WN, EPI_QKV_ROPE, KB, NST, OCC, XW, A>(c, st);
    case EPI_RESIDUAL: return launch_one<BM, BN, WM, WN, EPI_RESIDUAL, KB, NST, OCC, XW, A>(c, st);
    case EPI_SWIGLU: return launch_one<BM, BN, WM, WN, EPI_SWIGLU, KB, NST, OCC, XW, A>(c, st);
    case EPI_LMSTATS: return launch_one<BM, BN, WM, WN, EPI_LMSTATS, KB, NST, OCC, XW, A>(c, st);
    case EPI_STORE_F32: return launch_one<BM, BN, WM, WN, EPI_STORE_F32, KB, NST, OCC, XW, A>(c, st);
    case EPI_LOGITS: return launch_one<BM, BN, WM, WN, EPI_LOGITS, KB, NST, OCC, XW, A>(c, st);
  }
  return hipErrorInvalidValue;
}

template <int BM, int BN, int WM, int WN, int KB, int NST, int OCC, int XW = 0>
hipError_t launch_cfg(const GemmCall& c, hipStream_t st) {
  return c.f16 ? launch_cfg_t<BM, BN, WM, WN, KB, NST, OCC, XW, ActF16>(c, st)
               : launch_cfg_t<BM, BN, WM, WN, KB, NST, OCC, XW, ActBf16>(c, st);
}

}  // namespace

void plan_residual_gemm(GemmCall& c, size_t part_elems) {
  const int f_tile = env_int("WINO_GEMM_TILE", -1);
  const int f_split = env_int("WINO_GEMM_SPLIT", 0), f_tail = env_int("WINO_GEMM_TAIL", -1);
  const bool forced = f_tile >= 0 || f_split > 0 || f_tail >= 0;
  if (!forced) {
    std::lock_guard<std::mutex> lk(g_plan_mu);
    for (int i = 0; i < g_n_plans; ++i) {
      const PlanEntry& e = g_plans[i];
      if (e.M == c.M && e.N == c.N && e.K == c.K && e.part_elems == part_elems) {
        c.tile = e.tile; c.splits = e.splits; c.split_row0 = e.split_row0;
        return;
      }
    }
  }
  const int nk = c.K / BK;
  int best = -1, best_s = 1, best_tail = 0;
  double best_t = 0;
  c.epi = EPI_RESIDUAL;
  for (int i = 0; i < kNumTiles; ++i) {
    const TileCfg& t = kTiles[i];
    if (!tile_ok(c, t) || (f_tile >= 0 && i != f_tile)) continue;
    const int nTM = (c.M + t.BM - 1) / t.BM;
    for (int tail = 0; tail <= nTM; ++tail) {
      if (f_tail >= 0 && tail != std::min(f_tail, nTM)) continue;
      const double tail_rows = c.M - (double)(nTM - tail) * t.BM;
      for (int s = tail ? 2 : 1; s <= (tail ? kMaxResidualSplits : 1); ++s) {
        if (tail && (nk % s || nk / s < 4 || s * tail_rows * c.N > (double)part_elems)) continue;
        if (tail && f_split > 0 && s != f_split) continue;
        const double time = residual_time(c, t, tail, s);
        if (best < 0 || time < best_t) { best = i; best_t = time; best_s = s; best_tail = tail; }
      }
    }
  }
  if (best < 0) {  // no candidate under the overrides: plain whole-K tiles
    c.tile = 0; c.splits = 1; c.split_row0 = c.M;
    return;
  }
  const int nTM = (c.M + kTiles[best].BM - 1) / kTiles[best].BM;
  c.tile = best + 1;
  c.splits = best_tail ? best_s : 1;
  c.split_row0 = best_tail ? (nTM - best_tail) * kTiles[best].BM : c.M;
  if (!forced) {
    std::lock_guard<std::mutex> lk(g_plan_mu);
    g_plans[g_n_plans % 32] = PlanEntry{c.M, c.N, c.K, part_elems, c.tile, c.splits, c.split_row0};
    g_n_plans = std::min(g_n_plans + 1, 32);
  }
}

int gemm_tile_n(const GemmCall& c) {
  const int i = pick_tile(c);
  return i < 0 ? 0 : kTiles[i].BN;
}

hipError_t launch_gemm(const GemmCall& c, hipStream_t st) {
  const int i = (c.tile > 0 && c.tile <= kNumTiles) ? c.tile - 1 : pick_tile(c);
  if (i < 0 || !tile_ok(c, kTiles[i])) return hipErrorInvalidValue;
  if (c.M <= 0) return hipSuccess;
  if (c.epi == EPI_RESIDUAL && c.splits > 1) {
    const int nk = c.K / BK;
    if (!c.part || c.split_row0 < 0 || c.split_row0 >= c.M || c.split_row0 % kTiles[i].BM ||
        nk % c.splits)
      return hipErrorInvalidValue;
  }
  switch (i) {
    case 0: return launch_cfg<256, 256, 2, 2, 64, 2, 1>(c, st);
    case 1: return launch_cfg<192, 256, 2, 2, 64, 2, 1>(c, st);
    case 2: return launch_cfg<128, 256, 2, 2, 64, 2, 1>(c, st);
    case 3: return launch_cfg<128, 128, 2, 2, 64, 2, 2>(c, st);
    case 4: return launch_cfg<64, 128, 2, 2, 64, 2, 3>(c, st);
    case 5: return launch_cfg<32, 256, 1, 4, 64, 2, 2>(c, st);
    case 6: return launch_cfg<256, 256, 4, 2, 64, 2, 1>(c, st);
    case 7: return launch_cfg<256, 256, 2, 4, 64, 2, 1>(c, st);
    case 8: return launch_cfg<128, 256, 2, 4, 64, 2, 1>(c, st);
    case 9: return launch_cfg<128, 256, 4, 2, 64, 2, 1>(c, st);
    case 10: return launch_cfg<128, 256, 4, 2, 64, 3, 1>(c, st);
    case 11: return launch_cfg<256, 256, 4, 2, 64, 2, 1, 1>(c, st);
    case 12: return launch_cfg<128, 256, 4, 2, 64, 2, 1, 1>(c, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace wino
