// Bidirectional flash attention with the WINO shadow-block mask (Sec. 4.2.2).
//
// Rows of the extended sequence: t < S are Y_left / Y_cur / Y_right and see
// keys [0, S) (never the shadow block); shadow row S+j sees every key in
// [0, T) except y_cur,j at c0+j - including all shadow rows and itself.
// No causal mask and no cache: every step recomputes all rows.
//
// Layout: q, k [B, H, Tp, hd] (RoPE already applied), v transposed
// [B, H, hd, Tp]; output o [B*T, H*hd] row-major; all in the activation type
// A (bf16 or fp16), whose MFMA form the kernel uses.
//
// Each wave owns 32 query rows.  Scores are computed transposed, S^T = K Q^T
// (32x32x16 MFMA), so a lane holds 32 keys of ONE query row and the online
// softmax max / sum stay inside the lane (plus its partner lane 32 apart).
// The same registers, rounded to A, are the B operand of O^T = V^T P^T
// (the softmax and its running sum stay in fp32).
//
// K and V^T tiles of 64 keys stream global -> LDS by LDS-DMA into two stages
// (the next tile loads while the current one is used), with 16-byte chunks
// XOR-swizzled per row so fragment reads are free of bank conflicts.  Within
// each 32-key block the K rows are stored in a permuted key order (bits 2 and
// 3 of the key index swapped): the MFMA then leaves each lane's P values for
// 8 CONSECUTIVE keys of a 16-key step, so its V^T operand is one 16-byte read.
#include "common.h"
#include "kernels.h"

namespace wino {
namespace {

constexpr int BKV = 64;

// key (within a 32-key block) held by MFMA output register i of lane group g
__device__ __forceinline__ int key_of(int i, int g) {
  const int ih = i >> 2;
  return 16 * (ih >> 1) + 8 * g + 4 * (ih & 1) + (i & 3);
}
// LDS row r of a K tile holds key perm(r): bits 2 and 3 swapped within 32
__device__ __forceinline__ int perm_key(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// CQ (compact queries): only each sequence's current-block rows and shadow
// rows are queried - compact query i < Lb is row c0 + i, i >= Lb is row
// S + i - Lb - and output row i of sequence b goes to o row b*(Lb+Ls) + i.
template <int HD, int NW, bool CQ, int NS, class A>
__global__ __launch_bounds__(NW * 64, 8 / NW) void attn_kernel(StepGeom g, const uint16_t* __restrict__ q,
                                                       const uint16_t* __restrict__ k,
                                                       const uint16_t* __restrict__ vt, int H,
                                                       uint16_t* __restrict__ o, float scale_log2) {
  constexpr int FE = HD / 32;        // 32-wide output blocks over the head dim
  constexpr int KS = HD / 16;        // 16-deep k steps over the head dim
  constexpr int KCH = HD / 8;        // 16-byte chunks per K row
  constexpr int KROWS = 1024 / (2 * HD);  // K rows per 1 KB DMA instruction
  constexpr int K_INS = BKV / KROWS / NW;  // K DMA instructions per wave
  constexpr int V_INS = HD / 8 / NW;       // V^T DMA instructions per wave (8 rows each)
  static_assert(K_INS * KROWS * NW == BKV && V_INS * 8 * NW == HD, "loader split");
  constexpr int KTILE = BKV * HD;    // 16-bit elements
  constexpr int STAGE = 2 * KTILE;   // K tile then V^T tile
  static_assert(NS >= 2, "pipeline stages");
  __shared__ __attribute__((aligned(1024))) uint16_t smem[NS * STAGE];

  // Workgroups are dealt to the 8 XCDs round-robin; remapped, each XCD takes a
  // contiguous range of (query tile, head, sequence) ids, so the query tiles
  // of one head share that XCD's L2 copy of its K and V^T
  const int nqt = gridDim.x, nwg = nqt * gridDim.y * gridDim.z;
  const int lin = xcd_remap(blockIdx.x + nqt * (blockIdx.y + gridDim.y * blockIdx.z), nwg);
  const int qt = lin % nqt, h = (lin / nqt) % gridDim.y, b = lin / (nqt * gridDim.y);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, grp = lane >> 5;
  const int q0 = qt * (NW * 32);
  const int c0 = cur_start(g, b);
  const int NQ = g.Lb + g.Ls;                    // compact queries per sequence
  const int ci = q0 + wave * 32 + (lane & 31);   // compact query index (CQ)
  const bool qvalid = CQ ? ci < NQ : q0 + wave * 32 + (lane & 31) < g.T;
  const int myq = CQ ? (ci < g.Lb ? c0 + ci : g.S + (ci - g.Lb)) : q0 + wave * 32 + (lane & 31);
  const bool shadow = myq >= g.S;
  const int excl = shadow ? c0 + (myq - g.S) : -1;
  const int klim = shadow ? g.T : g.S;
  const size_t bh = (size_t)b * H + h;
  const uint16_t* qb = q + bh * g.Tp * HD;
  const uint16_t* kb = k + bh * g.Tp * HD;
  const uint16_t* vb = vt + bh * HD * g.Tp;

  // DMA sources (per lane, fixed offsets; the key tile start is added later)
  int koff[K_INS];   // element offset of this lane's 16 bytes for K row r, relative to key 0
  int krow[K_INS];   // tile-relative key of that row
#pragma unroll
  for (int i = 0; i < K_INS; ++i) {
    const int gi = wave * K_INS + i;
    const int r = gi * KROWS + lane / (KCH);
    const int pos = lane % KCH;
    const int swz = KCH == 16 ? (r & 15) : ((r ^ (r >> 3)) & 7);
    krow[i] = (r & ~31) | perm_key(r & 31);
    koff[i] = (pos ^ swz) * 8;
  }
  const uint16_t* vsrc[V_INS];
#pragma unroll
  for (int i = 0; i < V_INS; ++i) {
    const int gi = wave * V_INS + i;
    const int e = gi * 8 + (lane >> 3);
    const int pos = lane & 7;
    vsrc[i] = vb + (size_t)e * g.Tp + (pos ^ ((e ^ (e >> 3)) & 7)) * 8;
  }
  auto issue = [&](int kv0, int stage) {
    uint16_t* sK = smem + stage * STAGE;
    uint16_t* sV = sK + KTILE;
    // (groups of four consecutive 1 KB blocks share one LDS base)
#pragma unroll
    for (int i = 0; i < K_INS; ++i) {
      // rows [T, Tp) of the padded buffer (zero from creation, or finite
      // rows of an earlier call) are read like the V^T padding and masked
      dma16(kb + (size_t)(kv0 + krow[i]) * HD + koff[i] - (i & 3) * 512,
            sK + (wave * K_INS + (i & ~3)) * 512, i & 3);
    }
    // Tp is a multiple of 64: the whole V^T tile row lies inside the buffer
#pragma unroll
    for (int i = 0; i < V_INS; ++i)
      dma16(vsrc[i] + kv0 - (i & 3) * 512, sV + (wave * V_INS + (i & ~3)) * 512, i & 3);
  };

  typename A::v8 qf[KS];
  {
    const int qrow = qvalid && myq < g.T ? myq : g.T - 1;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = A::frag(*reinterpret_cast<const uint4*>(qb + (size_t)qrow * HD + ks * 16 + grp * 8));
  }

  f32x16 oacc[FE];
#pragma unroll
  for (int fe = 0; fe < FE; ++fe)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[fe][i] = 0.f;
  float mrun = kNegBig, lrun = 0.f;
  const float rescale_gap = 8.f / scale_log2;

  const bool has_shadow = CQ ? g.Ls > 0 && q0 + NW * 32 > g.Lb : min(q0 + NW * 32, g.T) - 1 >= g.S;
  // A wave whose 32 query rows all lie past the last one (the tail of the
  // last query tile) only copies tiles and meets the barriers: its SIMD is
  // left to the other workgroup's wave.
  const bool wave_live = q0 + wave * 32 < (CQ ? NQ : g.T);
  const int kend = has_shadow ? g.T : g.S;  // shadow rows also see keys S..T-1
  const int ntile = (kend + BKV - 1) / BKV;

  // fragment-read swizzles of the rows this lane reads (fixed over tiles)
  const int kr = lane & 31;                    // K rows kb2*32 + kr
  int kswz[2];
#pragma unroll
  for (int kb2 = 0; kb2 < 2; ++kb2) {
    const int r = kb2 * 32 + kr;
    kswz[kb2] = KCH == 16 ? (r & 15) : ((r ^ (r >> 3)) & 7);
  }
  int vswz[FE];
#pragma unroll
  for (int fe = 0; fe < FE; ++fe) {
    const int e = fe * 32 + (lane & 31);
    vswz[fe] = (e ^ (e >> 3)) & 7;
  }

  // The copies of tile t are issued NS-1 tiles ahead, into stage t % NS; with
  // more than two stages the tiles past the last are fetches of the last one
  // again, which keeps the number of copies in flight fixed.
#pragma unroll
  for (int s0 = 0; s0 + 1 < NS; ++s0) issue(min(s0, ntile - 1) * BKV, s0);
  for (int t = 0; t < ntile; ++t) {
    const int kv0 = t * BKV;
    // own copies of tile t landed (the NS-2 tiles after it may still be in
    // flight); after the barrier everyone's have, and everyone finished tile
    // t-1, whose stage tile t+NS-1 may now overwrite
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 2) * (K_INS + V_INS)) : "memory");
    __syncthreads();
    if (NS > 2 || t + 1 < ntile) issue(min(t + NS - 1, ntile - 1) * BKV, (t + NS - 1) % NS);
    if (!wave_live) continue;
    const uint16_t* sK = smem + (t % NS) * STAGE;
    const uint16_t* sV = sK + KTILE;

    // S^T for the two 32-key blocks: the two MFMA chains alternate, and the
    // K fragments of step ks + 2 are read while step ks multiplies (one step
    // ahead leaves the LDS latency exposed: bs16 133 -> 131 us, two steps 129)
    auto vfrag = [&](int ks4, int fe) {
      const int row = fe * 32 + (lane & 31);
      const int ch = (ks4 * 2 + grp) ^ vswz[fe];
      return A::frag(*reinterpret_cast<const uint4*>(sV + row * BKV + ch * 8));
    };
    typename A::v8 vf[2][FE];
    f32x16 s[2];
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int i = 0; i < 16; ++i) s[kb2][i] = 0.f;
    auto kfrag = [&](int ks, int kb2) {
      const int ch = (ks * 2 + grp) ^ kswz[kb2];
      return A::frag(*reinterpret_cast<const uint4*>(sK + (kb2 * 32 + kr) * HD + ch * 8));
    };
    typename A::v8 kf[3][2];
    kf[0][0] = kfrag(0, 0);
    kf[0][1] = kfrag(0, 1);
    kf[1][0] = kfrag(1, 0);
    kf[1][1] = kfrag(1, 1);
    // the order is pinned: left to itself the compiler keeps one fragment
    // set and waits for each pair of reads right before its MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 2 < KS) {
        kf[(ks + 2) % 3][0] = kfrag(ks + 2, 0);
        kf[(ks + 2) % 3][1] = kfrag(ks + 2, 1);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
      }
      s[0] = A::mma(kf[ks % 3][0], qf[ks], s[0]);
      s[1] = A::mma(kf[ks % 3][1], qf[ks], s[1]);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 1);
    }
    // the first V^T fragments load while the softmax runs
#pragma unroll
    for (int fe = 0; fe < FE; ++fe) vf[0][fe] = vfrag(0, fe);

    // Only tiles that reach past S or hold an excluded shadow column need the
    // mask predicate; the test is uniform over the workgroup.
    const bool edge = kv0 + BKV > g.S || (has_shadow && kv0 < c0 + g.Lb && kv0 + BKV > c0);
    float tmax = kNegBig;
    if (edge) {
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kv0 + kb2 * 32 + key_of(i, grp);
          const bool ok = key < klim && key != excl;
          s[kb2][i] = ok ? s[kb2][i] : kNegBig;
        }
    }
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int i = 0; i < 16; ++i) tmax = fmaxf(tmax, s[kb2][i]);
    tmax = max_xor32(tmax);
    // Reference max mrun in raw score units; probabilities exp2(s*c - m*c)
    // with c = log2(e)/sqrt(hd): one FMA per score.  The reference moves
    // (and O, l are rescaled) only when a score exceeds it by more than
    // 8/c, so probabilities stay below 2^8 and the rescale is rare after
    // the first tile; p and l share the reference, so O / l is unchanged.
    const bool resc = tmax > mrun + rescale_gap;
    if (__any(resc)) {
      const float mnew = resc ? tmax : mrun;
      const float alpha = __builtin_amdgcn_exp2f((mrun - mnew) * scale_log2);
      lrun *= alpha;
      mrun = mnew;
#pragma unroll
      for (int fe = 0; fe < FE; ++fe)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[fe][i] *= alpha;
    }
    const float mc = mrun == kNegBig ? 0.f : mrun * scale_log2;
    // the hardware exp2 (v_exp_f32): results below 2^-126 flush to zero,
    // which next to a running sum of at least one changes nothing; the
    // library exp2f adds five instructions per score to keep them
    float psum = 0.f;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[kb2][i], scale_log2, -mc));
        s[kb2][i] = p;
        psum += p;
      }
    lrun += psum;

#pragma unroll
    for (int ks4 = 0; ks4 < BKV / 16; ++ks4) {
      // V^T fragments of the next 16-key step are read while this one multiplies
      if (ks4 + 1 < BKV / 16) {
#pragma unroll
        for (int fe = 0; fe < FE; ++fe) vf[(ks4 + 1) & 1][fe] = vfrag(ks4 + 1, fe);
      }
      // P in A (values up to 2^8): registers 8*(ks4&1)..+7 of block ks4/2 hold keys
      // 16*ks4 + 8*grp + 0..7.
      const int base = 8 * (ks4 & 1);
      uint32_t ph[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        ph[e] = A::pack2(s[ks4 >> 1][base + 2 * e], s[ks4 >> 1][base + 2 * e + 1]);
      const typename A::v8 pf = A::frag(make_uint4(ph[0], ph[1], ph[2], ph[3]));
#pragma unroll
      for (int fe = 0; fe < FE; ++fe) oacc[fe] = A::mma(vf[ks4 & 1][fe], pf, oacc[fe]);
    }
  }

  lrun = sum_xor32(lrun);
  if (qvalid) {
    const float inv = 1.f / lrun;
    const size_t orow = CQ ? (size_t)b * NQ + ci : (size_t)b * g.T + myq;
    uint16_t* dst = o + orow * (size_t)(H * HD) + (size_t)h * HD;
#pragma unroll
    for (int fe = 0; fe < FE; ++fe)
#pragma unroll
      for (int i = 0; i < 16; i += 4) {
        // rows 8*(i/4) + 4*grp + 0..3 of this e block: 4 consecutive outputs
        uint2 w;
        w.x = A::pack2(oacc[fe][i] * inv, oacc[fe][i + 1] * inv);
        w.y = A::pack2(oacc[fe][i + 2] * inv, oacc[fe][i + 3] * inv);
        *reinterpret_cast<uint2*>(dst + fe * 32 + mfma_row(i, lane)) = w;
      }
  }
}

template <int HD, class A>
hipError_t launch_hd(const StepGeom& g, const uint16_t* q, const uint16_t* k, const uint16_t* vt,
                     int H, uint16_t* o, float scale_log2, bool compact, hipStream_t st) {
  if (compact) {
    // (four waves here too: 16.1 against 19.4 us at 544 rows and batch 1,
    // 48 against 58 us at 2112 rows and batch 4, for 64 compact queries per
    // sequence; the two idle waves only copy tiles)
    dim3 grid((g.Lb + g.Ls + 127) / 128, H, g.B);
    attn_kernel<HD, 4, true, 2, A><<<grid, 256, 0, st>>>(g, q, k, vt, H, o, scale_log2);
    return hipGetLastError();
  }
  // 128-query workgroups (four waves) at every size: at 544 rows they take
  // 16.6 us against 21.3 us for twice as many 64-query workgroups (whose
  // two-wave kernel spends 96 accumulation registers and runs one wave per
  // SIMD), and three or four K/V stages did not pay there either.
  dim3 grid((g.T + 127) / 128, H, g.B);
  attn_kernel<HD, 4, false, 2, A><<<grid, 256, 0, st>>>(g, q, k, vt, H, o, scale_log2);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const StepGeom& g, const uint16_t* q, const uint16_t* k,
                            const uint16_t* vt, int H, int hd, uint16_t* o, hipStream_t st,
                            bool compact) {
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
  if (g.f16) {
    if (hd == 128) return launch_hd<128, ActF16>(g, q, k, vt, H, o, scale_log2, compact, st);
    if (hd == 64) return launch_hd<64, ActF16>(g, q, k, vt, H, o, scale_log2, compact, st);
  } else {
    if (hd == 128) return launch_hd<128, ActBf16>(g, q, k, vt, H, o, scale_log2, compact, st);
    if (hd == 64) return launch_hd<64, ActBf16>(g, q, k, vt, H, o, scale_log2, compact, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace wino
