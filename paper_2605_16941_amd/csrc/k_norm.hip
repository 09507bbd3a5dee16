// Embedding gather and RMSNorm kernels: one wave per row, the row held in
// registers (16-byte chunks of 8 elements per lane), fp32 sum of squares by a
// wave butterfly, output in the activation type A (bf16 or fp16) rounded to
// nearest even.  Gains and the embedding table are bf16 weights.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace wino {

namespace {

template <class A, int CPL>
__device__ __forceinline__ void norm_store(float (&v)[CPL][8], float ss, const uint16_t* gain,
                                           float eps, int d, int lane, uint16_t* out,
                                           uint16_t* out_lo = nullptr) {
  const int nch = d >> 3;
  ss = wave_sum(ss);
  const float r = rsqrtf(ss / (float)d + eps);
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = lane + c * 64;
    if (ch < nch) {
      const uint4 graw = *reinterpret_cast<const uint4*>(gain + ch * 8);
      const uint16_t* gp = reinterpret_cast<const uint16_t*>(&graw);
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = v[c][e] * r * bf2f(gp[e]);
      uint4 o;
      uint32_t* op = reinterpret_cast<uint32_t*>(&o);
#pragma unroll
      for (int e = 0; e < 4; ++e) op[e] = A::pack2(y[2 * e], y[2 * e + 1]);
      *reinterpret_cast<uint4*>(out + ch * 8) = o;
      if (out_lo) {
        const uint16_t* hi = reinterpret_cast<const uint16_t*>(&o);
        uint4 lo;
        uint32_t* lp = reinterpret_cast<uint32_t*>(&lo);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          lp[e] = A::pack2(y[2 * e] - A::val(hi[2 * e]), y[2 * e + 1] - A::val(hi[2 * e + 1]));
        *reinterpret_cast<uint4*>(out_lo + ch * 8) = lo;
      }
    }
  }
}

template <class A, int CPL>
__global__ __launch_bounds__(256) void embed_norm_kernel(StepGeom g, const int32_t* __restrict__ tokens,
                                                         const uint16_t* __restrict__ emb, int vocab,
                                                         const uint16_t* __restrict__ gain, float eps,
                                                         int d, float* __restrict__ x,
                                                         uint16_t* __restrict__ h) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= g.B * g.T) return;
  const int b = m / g.T, t = m - b * g.T;
  int tok = t < g.S ? tokens[(size_t)b * g.S + t] : g.mask_id;
  tok = tok < 0 ? 0 : (tok >= vocab ? vocab - 1 : tok);  // ids outside [0,V) are clamped
  const uint16_t* src = emb + (size_t)tok * d;
  float* xr = x + (size_t)m * d;
  const int nch = d >> 3;
  float v[CPL][8];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = lane + c * 64;
    if (ch < nch) {
      const uint4 raw = *reinterpret_cast<const uint4*>(src + ch * 8);
      const uint16_t* p = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[c][e] = bf2f(p[e]);
        ss += v[c][e] * v[c][e];
      }
      float4* xo = reinterpret_cast<float4*>(xr + ch * 8);
      xo[0] = make_float4(v[c][0], v[c][1], v[c][2], v[c][3]);
      xo[1] = make_float4(v[c][4], v[c][5], v[c][6], v[c][7]);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[c][e] = 0.f;
    }
  }
  norm_store<A, CPL>(v, ss, gain, eps, d, lane, h + (size_t)m * d);
}

template <int CPL>
__device__ __forceinline__ float load_row_f32(const float* xr, int d, int lane, float (&v)[CPL][8]) {
  const int nch = d >> 3;
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = lane + c * 64;
    if (ch < nch) {
      const float4* xi = reinterpret_cast<const float4*>(xr + ch * 8);
      const float4 a = xi[0], bq = xi[1];
      v[c][0] = a.x; v[c][1] = a.y; v[c][2] = a.z; v[c][3] = a.w;
      v[c][4] = bq.x; v[c][5] = bq.y; v[c][6] = bq.z; v[c][7] = bq.w;
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[c][e] * v[c][e];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[c][e] = 0.f;
    }
  }
  return ss;
}

// x[m] (+)= sum of split-K partials, in split order; returns the row in v.
// The loads of one split for all of the lane's chunks are independent, so
// they are in flight together.
template <int CPL>
__device__ __forceinline__ float load_row_reduce(float* xr, const float* part, int n_part,
                                                 size_t pstride, int d, int lane, float (&v)[CPL][8]) {
  const int nch = d >> 3;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = lane + c * 64;
    if (ch < nch) {
      const float4* xi = reinterpret_cast<const float4*>(xr + ch * 8);
      const float4 a = xi[0], b = xi[1];
      v[c][0] = a.x; v[c][1] = a.y; v[c][2] = a.z; v[c][3] = a.w;
      v[c][4] = b.x; v[c][5] = b.y; v[c][6] = b.z; v[c][7] = b.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[c][e] = 0.f;
    }
  }
  for (int s = 0; s < n_part; ++s) {
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int ch = lane + c * 64;
      if (ch < nch) {
        const float4* pi = reinterpret_cast<const float4*>(part + s * pstride + ch * 8);
        const float4 a = pi[0], b = pi[1];
        v[c][0] += a.x; v[c][1] += a.y; v[c][2] += a.z; v[c][3] += a.w;
        v[c][4] += b.x; v[c][5] += b.y; v[c][6] += b.z; v[c][7] += b.w;
      }
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = lane + c * 64;
    if (ch < nch) {
      if (n_part) {
        float4* xo = reinterpret_cast<float4*>(xr + ch * 8);
        xo[0] = make_float4(v[c][0], v[c][1], v[c][2], v[c][3]);
        xo[1] = make_float4(v[c][4], v[c][5], v[c][6], v[c][7]);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[c][e] * v[c][e];
    }
  }
  return ss;
}

template <class A, int CPL>
__global__ __launch_bounds__(256) void rmsnorm_kernel(float* __restrict__ x,
                                                      const uint16_t* __restrict__ gain, float eps,
                                                      int M, int d, uint16_t* __restrict__ h,
                                                      const float* __restrict__ part, int n_part,
                                                      int part_row0) {
  const int lane = threadIdx.x & 63;
  // rows carrying partials (m >= part_row0) are the slow ones: take them first
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= M) return;
  const int n_tail = n_part ? M - part_row0 : 0;
  const int m = r < n_tail ? part_row0 + r : r - n_tail;
  float v[CPL][8];
  const bool has = m >= part_row0;
  const float ss = load_row_reduce<CPL>(x + (size_t)m * d, part + (size_t)(has ? m - part_row0 : 0) * d,
                                        has ? n_part : 0, (size_t)(M - part_row0) * d, d, lane, v);
  norm_store<A, CPL>(v, ss, gain, eps, d, lane, h + (size_t)m * d);
}

// RMSNorm with a whole workgroup per row (d = 2048 * CPT): 256 threads hold
// CPT 8-element chunks each, so a row's loads (x, every partial and the gain)
// are all in flight at once.  Against one wave per row: 6.3 vs 4.7 TB/s at
// 8704 x 4096, and 11 vs 17 us per launch at 544 rows.  NP is the number of
// split-K partials when known at compile time (their loads are then all
// issued before the first wait; -1: a runtime loop over them, one round trip
// each), added in split order either way.
template <class A, int CPT, int NP>
__global__ __launch_bounds__(256) void rmsnorm_row_kernel(float* __restrict__ x,
                                                          const uint16_t* __restrict__ gain, float eps,
                                                          int M, int d, uint16_t* __restrict__ h,
                                                          const float* __restrict__ part, int n_part,
                                                          int part_row0) {
  __shared__ float red[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = blockIdx.x;
  const int n_tail = n_part ? M - part_row0 : 0;
  const int m = r < n_tail ? part_row0 + r : r - n_tail;  // partial rows first
  const bool has = n_part && m >= part_row0;
  float* xr = x + (size_t)m * d;
  float v[CPT][8];
  uint4 graw[CPT];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const float4* xi = reinterpret_cast<const float4*>(xr + (c * 256 + tid) * 8);
    const float4 a = xi[0], b = xi[1];
    v[c][0] = a.x; v[c][1] = a.y; v[c][2] = a.z; v[c][3] = a.w;
    v[c][4] = b.x; v[c][5] = b.y; v[c][6] = b.z; v[c][7] = b.w;
    graw[c] = *reinterpret_cast<const uint4*>(gain + (c * 256 + tid) * 8);
  }
  auto add = [&](int c, float4 a, float4 b) {
    v[c][0] += a.x; v[c][1] += a.y; v[c][2] += a.z; v[c][3] += a.w;
    v[c][4] += b.x; v[c][5] += b.y; v[c][6] += b.z; v[c][7] += b.w;
  };
  if (has) {
    const float* pr = part + (size_t)(m - part_row0) * d;
    const size_t pstride = (size_t)(M - part_row0) * d;
    if constexpr (NP > 0) {
      float4 pa[NP][CPT][2];
#pragma unroll
      for (int s = 0; s < NP; ++s)
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
          const float4* pi = reinterpret_cast<const float4*>(pr + s * pstride + (c * 256 + tid) * 8);
          pa[s][c][0] = pi[0];
          pa[s][c][1] = pi[1];
        }
#pragma unroll
      for (int s = 0; s < NP; ++s)
#pragma unroll
        for (int c = 0; c < CPT; ++c) add(c, pa[s][c][0], pa[s][c][1]);
    } else if constexpr (NP < 0) {
      for (int s = 0; s < n_part; ++s)
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
          const float4* pi = reinterpret_cast<const float4*>(pr + s * pstride + (c * 256 + tid) * 8);
          add(c, pi[0], pi[1]);
        }
    }
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      float4* xo = reinterpret_cast<float4*>(xr + (c * 256 + tid) * 8);
      xo[0] = make_float4(v[c][0], v[c][1], v[c][2], v[c][3]);
      xo[1] = make_float4(v[c][4], v[c][5], v[c][6], v[c][7]);
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[c][e] * v[c][e];
  ss = wave_sum(ss);
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  ss = (red[0] + red[1]) + (red[2] + red[3]);
  const float rs = rsqrtf(ss / (float)d + eps);
  uint16_t* out = h + (size_t)m * d;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int ch = c * 256 + tid;
    const uint16_t* gp = reinterpret_cast<const uint16_t*>(&graw[c]);
    uint4 o;
    uint32_t* op = reinterpret_cast<uint32_t*>(&o);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      op[e] = A::pack2(v[c][2 * e] * rs * bf2f(gp[2 * e]), v[c][2 * e + 1] * rs * bf2f(gp[2 * e + 1]));
    *reinterpret_cast<uint4*>(out + ch * 8) = o;
  }
}

template <int CPL>
__global__ __launch_bounds__(256) void residual_reduce_kernel(float* __restrict__ x,
                                                              const float* __restrict__ part,
                                                              int n_part, int part_row0, int M,
                                                              int d) {
  const int lane = threadIdx.x & 63;
  const int m = part_row0 + blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  float v[CPL][8];
  load_row_reduce<CPL>(x + (size_t)m * d, part + (size_t)(m - part_row0) * d, n_part,
                       (size_t)(M - part_row0) * d, d, lane, v);
}

template <class A, int CPL>
__global__ __launch_bounds__(256) void select_norm_kernel(StepGeom g, int mode,
                                                          const int32_t* __restrict__ tokens,
                                                          const float* __restrict__ x,
                                                          const uint16_t* __restrict__ gain,
                                                          float eps, int d, uint16_t* __restrict__ hf,
                                                          uint16_t* __restrict__ hf_lo,
                                                          int32_t* __restrict__ target, int r0,
                                                          int n, const int32_t* __restrict__ tgt_in,
                                                          int compact) {
  const int lane = threadIdx.x & 63;
  const int rows_per_seq = mode == 0 ? g.Lb : mode == 1 ? 2 * g.Lb : g.G;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= n) return;
  const int ra = r0 + r;  // row of the flattened [B, rows_per_seq] selection
  const int b = ra / rows_per_seq, j = ra - b * rows_per_seq;
  int src;
  if (mode == 2) {  // response row j (WINO+ training state, no shadow block)
    src = g.P + j;
    if (lane == 0) target[r] = tgt_in[ra];
  } else if (mode == 0) {
    const int c0 = cur_start(g, b);
    const int tok = tokens[(size_t)b * g.S + c0 + j];
    // Eq. 4: draft reads Y_cur, verify reads Y_shad (without shadow rows no
    // position is verified; the current row's statistics then go unused)
    const bool verify = tok != g.mask_id && g.Ls > 0;
    src = verify ? g.S + j : c0 + j;
    if (compact) src = verify ? g.Lb + j : j;  // gathered rows: current block, then shadow
    if (lane == 0) target[r] = verify ? tok : -1;
  } else {
    src = j < g.Lb ? cur_start(g, b) + j : g.S + (j - g.Lb);
    if (lane == 0) target[r] = -1;
  }
  float v[CPL][8];
  const size_t xrow = compact ? (size_t)b * (g.Lb + g.Ls) + src : (size_t)b * g.T + src;
  const float ss = load_row_f32<CPL>(x + xrow * d, d, lane, v);
  norm_store<A, CPL>(v, ss, gain, eps, d, lane, hf + (size_t)r * d, hf_lo + (size_t)r * d);
}

// Copy of the current-block and shadow rows of every sequence (fp32).
__global__ __launch_bounds__(256) void gather_block_rows_kernel(StepGeom g, const float* __restrict__ x,
                                                                int d, float* __restrict__ xc) {
  const int nq = g.Lb + g.Ls;
  const int r = blockIdx.x;  // b * nq + i
  const int b = r / nq, i = r - b * nq;
  const int t = i < g.Lb ? cur_start(g, b) + i : g.S + (i - g.Lb);
  const float4* src = reinterpret_cast<const float4*>(x + ((size_t)b * g.T + t) * d);
  float4* dst = reinterpret_cast<float4*>(xc + (size_t)r * d);
  for (int c = threadIdx.x; c < d / 4; c += 256) dst[c] = src[c];
}

// Weights bf16 -> fp16 (round to nearest even), 8 elements per thread; n is
// a multiple of 8.
__global__ __launch_bounds__(256) void bf16_to_f16_kernel(const uint16_t* __restrict__ in,
                                                          uint16_t* __restrict__ out, size_t n8,
                                                          int* __restrict__ overflow) {
  bool bad = false;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += (size_t)gridDim.x * 256) {
    const uint4 raw = reinterpret_cast<const uint4*>(in)[i];
    const uint32_t* w = &raw.x;
    uint4 o;
    uint32_t* op = &o.x;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      op[e] = ActF16::pack2(__uint_as_float(w[e] << 16), __uint_as_float(w[e] & 0xFFFF0000u));
      // an all-ones exponent: the value overflowed fp16 (or was not finite)
      bad |= (op[e] & 0x7C00u) == 0x7C00u || (op[e] & 0x7C000000u) == 0x7C000000u;
    }
    reinterpret_cast<uint4*>(out)[i] = o;
  }
  if (bad) *overflow = 1;
}

}  // namespace

void launch_bf16_to_f16(const uint16_t* in, uint16_t* out, size_t n, int* overflow, hipStream_t st) {
  const size_t n8 = n / 8;
  if (n8 == 0) return;
  const size_t blocks = std::min<size_t>((n8 + 255) / 256, 8192);
  bf16_to_f16_kernel<<<blocks, 256, 0, st>>>(in, out, n8, overflow);
}

// The library accepts d <= 4096 (up to 8 chunks of 8 elements per lane).
template <class A>
void embed_norm_impl(const StepGeom& g, const int32_t* tokens, const uint16_t* emb, int vocab,
                     const uint16_t* gain, float eps, int d, float* x, uint16_t* h, hipStream_t st) {
  const int M = g.B * g.T;
  dim3 grid((M + 3) / 4), block(256);
  if (d <= 512) embed_norm_kernel<A, 1><<<grid, block, 0, st>>>(g, tokens, emb, vocab, gain, eps, d, x, h);
  else if (d <= 1024) embed_norm_kernel<A, 2><<<grid, block, 0, st>>>(g, tokens, emb, vocab, gain, eps, d, x, h);
  else if (d <= 2048) embed_norm_kernel<A, 4><<<grid, block, 0, st>>>(g, tokens, emb, vocab, gain, eps, d, x, h);
  else embed_norm_kernel<A, 8><<<grid, block, 0, st>>>(g, tokens, emb, vocab, gain, eps, d, x, h);
}

void launch_embed_norm(const StepGeom& g, const int32_t* tokens, const uint16_t* emb, int vocab,
                       const uint16_t* gain, float eps, int d, float* x, uint16_t* h,
                       hipStream_t st) {
  if (g.f16) embed_norm_impl<ActF16>(g, tokens, emb, vocab, gain, eps, d, x, h, st);
  else embed_norm_impl<ActBf16>(g, tokens, emb, vocab, gain, eps, d, x, h, st);
}

template <class A, int CPT>
void launch_row_norm(float* x, const uint16_t* gain, float eps, int M, int d, uint16_t* h,
                     const float* part, int n_part, int part_row0, hipStream_t st) {
  // the split counts the residual planner uses get their own instance
  switch (n_part) {
    case 0: rmsnorm_row_kernel<A, CPT, 0><<<M, 256, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0); break;
    case 2: rmsnorm_row_kernel<A, CPT, 2><<<M, 256, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0); break;
    case 3: rmsnorm_row_kernel<A, CPT, 3><<<M, 256, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0); break;
    case 4: rmsnorm_row_kernel<A, CPT, 4><<<M, 256, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0); break;
    case 8: rmsnorm_row_kernel<A, CPT, 8><<<M, 256, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0); break;
    default: rmsnorm_row_kernel<A, CPT, -1><<<M, 256, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0);
  }
}

template <class A>
void rmsnorm_impl(float* x, const uint16_t* gain, float eps, int M, int d, uint16_t* h,
                  const float* part, int n_part, int part_row0, hipStream_t st) {
  const dim3 grid((M + 3) / 4), block(256);
  if (!part) n_part = 0;
  if (d == 2048 || d == 4096) {  // measured faster at 544 and 8704 rows
    if (d == 2048) launch_row_norm<A, 1>(x, gain, eps, M, d, h, part, n_part, part_row0, st);
    else launch_row_norm<A, 2>(x, gain, eps, M, d, h, part, n_part, part_row0, st);
    return;
  }
  if (d <= 512) rmsnorm_kernel<A, 1><<<grid, block, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0);
  else if (d <= 1024) rmsnorm_kernel<A, 2><<<grid, block, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0);
  else if (d <= 2048) rmsnorm_kernel<A, 4><<<grid, block, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0);
  else rmsnorm_kernel<A, 8><<<grid, block, 0, st>>>(x, gain, eps, M, d, h, part, n_part, part_row0);
}

void launch_rmsnorm(float* x, const uint16_t* gain, float eps, int M, int d, uint16_t* h,
                    const float* part, int n_part, int part_row0, hipStream_t st, bool f16) {
  if (f16) rmsnorm_impl<ActF16>(x, gain, eps, M, d, h, part, n_part, part_row0, st);
  else rmsnorm_impl<ActBf16>(x, gain, eps, M, d, h, part, n_part, part_row0, st);
}

void launch_residual_reduce(float* x, const float* part, int n_part, int part_row0, int M, int d,
                            hipStream_t st) {
  if (M - part_row0 <= 0) return;
  const dim3 grid((M - part_row0 + 3) / 4), block(256);
  if (d <= 512) residual_reduce_kernel<1><<<grid, block, 0, st>>>(x, part, n_part, part_row0, M, d);
  else if (d <= 1024) residual_reduce_kernel<2><<<grid, block, 0, st>>>(x, part, n_part, part_row0, M, d);
  else if (d <= 2048) residual_reduce_kernel<4><<<grid, block, 0, st>>>(x, part, n_part, part_row0, M, d);
  else residual_reduce_kernel<8><<<grid, block, 0, st>>>(x, part, n_part, part_row0, M, d);
}

template <class A>
void select_norm_impl(const StepGeom& g, int mode, const int32_t* tokens, const float* x,
                      const uint16_t* gain, float eps, int d, uint16_t* hf, uint16_t* hf_lo,
                      int32_t* target, hipStream_t st, int r0, int n, const int32_t* tgt_in, int cp) {
  dim3 grid((n + 3) / 4), block(256);
  if (d <= 512) select_norm_kernel<A, 1><<<grid, block, 0, st>>>(g, mode, tokens, x, gain, eps, d, hf, hf_lo, target, r0, n, tgt_in, cp);
  else if (d <= 1024) select_norm_kernel<A, 2><<<grid, block, 0, st>>>(g, mode, tokens, x, gain, eps, d, hf, hf_lo, target, r0, n, tgt_in, cp);
  else if (d <= 2048) select_norm_kernel<A, 4><<<grid, block, 0, st>>>(g, mode, tokens, x, gain, eps, d, hf, hf_lo, target, r0, n, tgt_in, cp);
  else select_norm_kernel<A, 8><<<grid, block, 0, st>>>(g, mode, tokens, x, gain, eps, d, hf, hf_lo, target, r0, n, tgt_in, cp);
}

void launch_select_norm(const StepGeom& g, int mode, const int32_t* tokens, const float* x,
                        const uint16_t* gain, float eps, int d, uint16_t* hf, uint16_t* hf_lo,
                        int32_t* target, hipStream_t st, int r0, int n, const int32_t* tgt_in,
                        bool compact) {
  if (mode != 2) { r0 = 0; n = g.B * (mode == 0 ? g.Lb : 2 * g.Lb); }
  if (mode != 0) compact = false;
  if (n <= 0) return;
  const int cp = compact ? 1 : 0;
  if (g.f16) select_norm_impl<ActF16>(g, mode, tokens, x, gain, eps, d, hf, hf_lo, target, st, r0, n, tgt_in, cp);
  else select_norm_impl<ActBf16>(g, mode, tokens, x, gain, eps, d, hf, hf_lo, target, st, r0, n, tgt_in, cp);
}

void launch_gather_block_rows(const StepGeom& g, const float* x, int d, float* xc, hipStream_t st) {
  const int rows = g.B * (g.Lb + g.Ls);
  if (rows > 0) gather_block_rows_kernel<<<rows, 256, 0, st>>>(g, x, d, xc);
}

}  // namespace wino
