// Bidirectional flash attention with the WINO shadow-block mask (Sec. 4.2.2).
//
// Rows of the extended sequence: t < S are Y_left / Y_cur / Y_right and see
// keys [0, S) (never the shadow block); shadow row S+j sees every key in
// [0, T) except y_cur,j at c0+j - including all shadow rows and itself.
// No causal mask and no cache: every step recomputes all rows.
//
// Layout: q, k bf16 [B, H, Tp, hd] (RoPE already applied), v transposed
// [B, H, hd, Tp]; output o bf16 [B*T, H*hd] row-major.
//
// Each wave owns 32 query rows.  Scores are computed transposed, S^T = K Q^T,
// so after the 32x32x16 MFMA a lane holds 32 keys of ONE query row: the
// online-softmax max / sum stay inside the lane (plus its partner lane 32
// apart).  The same registers, split into hi and lo bf16 parts, are the B
// operand of O^T = V^T P^T, whose A operand comes from the transposed V tile
// in LDS; the per-lane key order of P and V^T is matched slot by slot.
#include "common.h"
#include "kernels.h"

namespace wino {
namespace {

constexpr int BKV = 64;

template <int HD, int NW>
__global__ __launch_bounds__(NW * 64) void attn_kernel(StepGeom g, const uint16_t* __restrict__ q,
                                                       const uint16_t* __restrict__ k,
                                                       const uint16_t* __restrict__ vt, int H,
                                                       uint16_t* __restrict__ o, float scale_log2) {
  constexpr int LDKS = HD + 8;  // K tile row stride (bf16), 16-byte padded
  constexpr int LDV = BKV + 8;  // V^T tile row stride
  constexpr int FE = HD / 32;   // 32-wide output blocks over the head dim
  constexpr int KS = HD / 16;   // 16-deep k steps over the head dim
  constexpr int NT = NW * 64;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BKV * LDKS];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[HD * LDV];

  const int b = blockIdx.z, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, grp = lane >> 5;
  const int q0 = blockIdx.x * (NW * 32);
  const int myq = q0 + wave * 32 + (lane & 31);
  const int c0 = cur_start(g, b);
  const bool shadow = myq >= g.S;
  const int excl = shadow ? c0 + (myq - g.S) : -1;
  const int klim = shadow ? g.T : g.S;
  const size_t bh = (size_t)b * H + h;
  const uint16_t* qb = q + bh * g.Tp * HD;
  const uint16_t* kb = k + bh * g.Tp * HD;
  const uint16_t* vb = vt + bh * HD * g.Tp;

  bf16x8 qf[KS];
  {
    const int qrow = myq < g.T ? myq : g.T - 1;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qb + (size_t)qrow * HD + ks * 16 + grp * 8));
  }

  f32x16 oacc[FE];
#pragma unroll
  for (int fe = 0; fe < FE; ++fe)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[fe][i] = 0.f;
  float mrun = kNegBig, lrun = 0.f;

  const int q_last = min(q0 + NW * 32, g.T) - 1;
  const int kend = q_last >= g.S ? g.T : g.S;  // shadow rows also see keys S..T-1

  for (int kv0 = 0; kv0 < kend; kv0 += BKV) {
    __syncthreads();
    for (int ci = tid; ci < BKV * HD / 8; ci += NT) {
      const int r = ci / (HD / 8), cc = ci - r * (HD / 8);
      const int key = kv0 + r;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (key < g.T) v = *reinterpret_cast<const uint4*>(kb + (size_t)key * HD + cc * 8);
      *reinterpret_cast<uint4*>(Ks + r * LDKS + cc * 8) = v;
    }
    for (int ci = tid; ci < HD * BKV / 8; ci += NT) {
      const int e = ci / (BKV / 8), cc = ci - e * (BKV / 8);
      // Tp is a multiple of 64, so the whole tile row is inside the buffer;
      // columns >= T get probability 0 below.
      const uint4 v = *reinterpret_cast<const uint4*>(vb + (size_t)e * g.Tp + kv0 + cc * 8);
      *reinterpret_cast<uint4*>(Vs + e * LDV + cc * 8) = v;
    }
    __syncthreads();

    f32x16 s[2];
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
      for (int i = 0; i < 16; ++i) s[kb2][i] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 kf = as_bf16x8(
            *reinterpret_cast<const uint4*>(Ks + (kb2 * 32 + (lane & 31)) * LDKS + ks * 16 + grp * 8));
        s[kb2] = mfma32(kf, qf[ks], s[kb2]);
      }
    }

    float tmax = kNegBig;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = kv0 + kb2 * 32 + mfma_row(i, lane);
        const bool ok = key < klim && key != excl;
        const float v = ok ? s[kb2][i] * scale_log2 : kNegBig;
        s[kb2][i] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(mrun, tmax);
    const float alpha = exp2f(mrun - mnew);
    float psum = 0.f;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = s[kb2][i] == kNegBig ? 0.f : exp2f(s[kb2][i] - mnew);
        s[kb2][i] = p;
        psum += p;
      }
    lrun = lrun * alpha + psum;
    mrun = mnew;
#pragma unroll
    for (int fe = 0; fe < FE; ++fe)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[fe][i] *= alpha;

#pragma unroll
    for (int ks4 = 0; ks4 < BKV / 16; ++ks4) {
      // P as hi + lo bf16 parts: the product with V keeps ~16 mantissa bits
      // of the probabilities instead of bf16's 8
      const int base = 8 * (ks4 & 1);
      uint32_t ph[4], pl[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = s[ks4 >> 1][base + 2 * e], p1 = s[ks4 >> 1][base + 2 * e + 1];
        ph[e] = pack2bf(p0, p1);
        pl[e] = pack2bf(p0 - bf2f((uint16_t)(ph[e] & 0xFFFFu)), p1 - bf2f((uint16_t)(ph[e] >> 16)));
      }
      const bf16x8 pf_hi = as_bf16x8(make_uint4(ph[0], ph[1], ph[2], ph[3]));
      const bf16x8 pf_lo = as_bf16x8(make_uint4(pl[0], pl[1], pl[2], pl[3]));
#pragma unroll
      for (int fe = 0; fe < FE; ++fe) {
        const uint16_t* vr = Vs + (fe * 32 + (lane & 31)) * LDV + 16 * ks4 + 4 * grp;
        const uint2 lo = *reinterpret_cast<const uint2*>(vr);
        const uint2 hi = *reinterpret_cast<const uint2*>(vr + 8);
        const bf16x8 vf = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
        oacc[fe] = mfma32(vf, pf_hi, oacc[fe]);
        oacc[fe] = mfma32(vf, pf_lo, oacc[fe]);
      }
    }
  }

  lrun += __shfl_xor(lrun, 32, 64);
  if (myq < g.T) {
    const float inv = 1.f / lrun;
    uint16_t* dst = o + ((size_t)b * g.T + myq) * (size_t)(H * HD) + (size_t)h * HD;
#pragma unroll
    for (int fe = 0; fe < FE; ++fe)
#pragma unroll
      for (int i = 0; i < 16; ++i) dst[fe * 32 + mfma_row(i, lane)] = f2bf(oacc[fe][i] * inv);
  }
}

}  // namespace

hipError_t launch_attention(const StepGeom& g, const uint16_t* q, const uint16_t* k,
                            const uint16_t* vt, int H, int hd, uint16_t* o, hipStream_t st) {
  constexpr int NW = 4;
  dim3 grid((g.T + NW * 32 - 1) / (NW * 32), H, g.B), block(NW * 64);
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
  if (hd == 128)
    attn_kernel<128, NW><<<grid, block, 0, st>>>(g, q, k, vt, H, o, scale_log2);
  else if (hd == 64)
    attn_kernel<64, NW><<<grid, block, 0, st>>>(g, q, k, vt, H, o, scale_log2);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace wino
