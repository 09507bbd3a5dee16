// WINO decision on device.
//
// epi_stats_kernel: for the standalone epilogue, each workgroup streams one
//   chunk of one needed logits row (the current row of a masked position, the
//   shadow row of an unmasked one) and writes partial softmax statistics.
// decide_kernel: one workgroup per sequence merges the partials of its block
//   positions (log-sum-exp merge; best non-mask id with lowest-id ties), turns
//   them into the draft confidence (Eq. 2) or the verify probability (Eq. 3),
//   and applies Eq. 4 with the forced draft (Eq. 1) and the step cap.
#include <climits>

#include "common.h"
#include "kernels.h"

namespace wino {
namespace {

struct RowStats {  // layout of wino_row_stats
  float m_all, sumexp, z_best, z_target;
  int32_t argmax, row_kind;
};

struct Part {
  float m, s, b, t;
  int i;
};

__device__ __forceinline__ void merge(Part& a, const Part& o) {
  const float m = fmaxf(a.m, o.m);
  a.s = a.s * __expf(a.m - m) + o.s * __expf(o.m - m);
  a.m = m;
  if (o.b > a.b || (o.b == a.b && o.i < a.i)) { a.b = o.b; a.i = o.i; }
  a.t = fmaxf(a.t, o.t);
}

// Merge across aligned groups of gs lanes (gs a power of two <= 64).
__device__ __forceinline__ Part group_merge(Part p, int gs) {
  for (int o = gs >> 1; o > 0; o >>= 1) {
    Part q;
    q.m = __shfl_xor(p.m, o, 64);
    q.s = __shfl_xor(p.s, o, 64);
    q.b = __shfl_xor(p.b, o, 64);
    q.t = __shfl_xor(p.t, o, 64);
    q.i = __shfl_xor(p.i, o, 64);
    merge(p, q);
  }
  return p;
}

// First response position in [from, G) of sequence b holding the mask, or G;
// a block-wide minimum over 256 threads.
__device__ int first_mask_from(const DecideArgs& a, int b, int from) {
  __shared__ int s_first;
  if (threadIdx.x == 0) s_first = a.G;
  __syncthreads();
  const int32_t* resp = a.tokens + (size_t)b * a.S + a.P;
  for (int j = from + (int)threadIdx.x; j < a.G; j += 256)
    if (resp[j] == a.mask_id) { atomicMin(&s_first, j); break; }
  __syncthreads();
  const int f = s_first;
  __syncthreads();
  return f;
}

// End of a fused step for an active sequence whose Y_cur holds nmask_after
// masks.  In decode mode (advance) a sequence whose block holds no mask moves
// to the first later block that still holds one - blocks filled beforehand
// (a resumed or pre-filled state) are skipped - or to G when none is left
// (Sec. 3: blocks left to right; Sec. 4.2.3: a block ends when Y_cur holds no
// mask), and its block step count restarts.  next_verify then describes the
// Y_cur the next step will see.  All 256 threads call this.
__device__ void advance_block(const DecideArgs& a, int b, int nmask_after) {
  __shared__ int s_m, s_k;
  const int bs = a.block_start[b];
  int nbs = bs;
  if (a.advance && nmask_after == 0 && bs < a.G) {
    const int f = first_mask_from(a, b, bs + a.Lb);
    nbs = f >= a.G ? a.G : bs + (f - bs) / a.Lb * a.Lb;
  }
  if (a.next_verify) {
    if (threadIdx.x == 0) { s_m = 0; s_k = 0; }
    __syncthreads();
    if (nbs < a.G) {
      const int c = nbs > a.G - a.Lb ? a.G - a.Lb : nbs;
      const int32_t* nxt = a.tokens + (size_t)b * a.S + a.P + c;
      for (int l = threadIdx.x; l < a.Lb; l += 256) {
        if (nxt[l] == a.mask_id) atomicAdd(&s_m, 1);
        else atomicAdd(&s_k, 1);
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) a.next_verify[b] = s_m > 0 && s_k > 0;
  }
  if (threadIdx.x == 0 && nbs != bs) {
    a.block_start[b] = nbs;
    if (a.block_steps) a.block_steps[b] = 0;
  }
}

// Lanes per block position in the partial merge: the largest power of two
// (at most 64) with lanes * Lb <= 256, so one pass covers the block when
// Lb <= 256.
__host__ __device__ __forceinline__ int merge_lanes(int Lb) {
  int gs = 1;
  while (gs < 64 && gs * 2 * Lb <= 256) gs *= 2;
  return gs;
}

// Partials j0, j0 + gs, ..., j0 + (U-1)*gs of row `row` (indices past n_part
// read partial 0 again and are not merged).
template <int U>
__device__ __forceinline__ void load_parts(const DecideArgs& a, size_t row, int j0, int gs, Part (&q)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int j = j0 + u * gs;
    const size_t o = row * a.n_part + (j < a.n_part ? j : 0);
    q[u] = Part{a.pm[o], a.ps[o], a.pb[o], a.pt[o], a.pi[o]};
  }
}

// The decision of sequence b by one 256-thread workgroup (all threads call
// it): merge the partial statistics of its block positions, then Eq. 4 (or the
// baseline rule), the forced draft and the step cap.  smem_i holds 4*Lb ints.
// U: partials each merge lane loads at once.
template <int U>
__device__ void decide_sequence(const DecideArgs& a, int b, int* smem_i) {
  int* s_cur = smem_i;                                   // [Lb] token before the step
  float* s_val = reinterpret_cast<float*>(s_cur + a.Lb);  // [Lb] conf (masked) or s (unmasked)
  int* s_hat = reinterpret_cast<int*>(s_val + a.Lb);      // [Lb] draft id
  int* s_flag = s_hat + a.Lb;                             // [Lb] decision
  __shared__ int s_nmask, s_nmask_after, s_any_draft, s_forced;

  const int tid = threadIdx.x;
  const int Lb = a.Lb;
  RowStats* stats = reinterpret_cast<RowStats*>(a.stats);

  int32_t* cur_ptr;
  int32_t* fin_ptr = nullptr;  // finalization-step record of Y_cur, or null
  bool done = false;
  if (a.standalone) {
    cur_ptr = a.tokens + (size_t)b * Lb;
  } else {
    const int bs = a.block_start[b];
    done = bs >= a.G;
    // same clamping as the forward kernels: Y_cur always lies inside the response
    const int bsc = bs < 0 ? 0 : (bs > a.G - Lb ? a.G - Lb : bs);
    cur_ptr = a.tokens + (size_t)b * a.S + a.P + bsc;
    if (a.final_step && a.seq_steps) fin_ptr = a.final_step + (size_t)b * a.G + bsc;
  }
  // With one batch per lane (PRE: the launch guarantees n_part <= gs * U and
  // Lb <= 256) the partial loads go out before the token loads, so the two
  // memory round trips overlap; otherwise the batches load in the merge loop.
  constexpr bool PRE = U == 2;
  const int gs = merge_lanes(Lb), per_pass = 256 / gs;
  const int sl = tid & (gs - 1);
  Part q0[U];
  if constexpr (PRE) load_parts<U>(a, (size_t)b * Lb + (tid / gs < Lb ? tid / gs : 0), sl, gs, q0);
  if (tid == 0) { s_nmask = 0; s_nmask_after = 0; s_any_draft = 0; s_forced = -1; }
  __syncthreads();
  if (!done) {
    for (int l = tid; l < Lb; l += 256) {
      const int t = cur_ptr[l];
      s_cur[l] = t;
      if (t == a.mask_id) atomicAdd(&s_nmask, 1);
    }
  }
  __syncthreads();
  // A finished sequence, or (fused step) a block with no mask left, is idle:
  // no decision, and in decode mode it only moves on to its next block below.
  const bool idle = done || (!a.standalone && s_nmask == 0);
  if (idle) {
    for (int l = tid; l < Lb; l += 256) {
      if (a.flags) a.flags[(size_t)b * Lb + l] = WINO_KEEP_FLAG;
      if (a.bitmap) a.bitmap[(size_t)b * Lb + l] = done ? 0 : (s_cur[l] == a.mask_id);
      if (stats) {
        RowStats z = {0.f, 0.f, 0.f, 0.f, -1, -1};
        stats[(size_t)b * Lb + l] = z;
      }
    }
    if (tid == 0 && a.n_masked) a.n_masked[b] = 0;
    if (done) {
      if (tid == 0 && a.next_verify) a.next_verify[b] = 0;
      return;
    }
    advance_block(a, b, 0);
    return;
  }

  // merge partials: a group of gs lanes per position, every position of a
  // pass at once, U partials' loads in flight per lane before they merge
  for (int base = 0; base < Lb; base += per_pass) {
    const int l = base + tid / gs;
    const size_t row = (size_t)b * Lb + (l < Lb ? l : 0);
    Part p = {kNegBig, 0.f, kNegBig, kNegBig, INT_MAX};
    if (l < Lb) {
      for (int j0 = sl; j0 < a.n_part; j0 += gs * U) {
        Part q[U];
        if constexpr (PRE) {
#pragma unroll
          for (int u = 0; u < U; ++u) q[u] = q0[u];
        } else {
          load_parts<U>(a, row, j0, gs, q);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (j0 + u * gs < a.n_part) merge(p, q[u]);
      }
    }
    p = group_merge(p, gs);
    if (sl == 0 && l < Lb) {
      const bool masked = s_cur[l] == a.mask_id;
      const float z = masked ? p.b : p.t;
      s_val[l] = __expf(z - p.m) / p.s;  // Eq. 2 confidence / Eq. 3 probability
      s_hat[l] = p.i;
      if (stats) {
        const bool ver = !masked && (a.verify || a.standalone);
        RowStats r = {p.m, p.s, p.b, ver ? p.t : kNegBig, p.i, masked ? 0 : (ver ? 1 : 2)};
        stats[row] = r;
      }
    }
  }
  __syncthreads();

  const int steps_before = (!a.standalone && a.block_steps) ? a.block_steps[b] : 0;
  const bool cap_now = !a.standalone && a.cap_fill && a.topm == 0 && (steps_before + 1 >= a.cap);
  for (int l = tid; l < Lb; l += 256) {
    const bool masked = s_cur[l] == a.mask_id;
    int f = WINO_KEEP_FLAG;
    if (a.topm > 0) {
      // baseline (Sec. 3): draft when fewer than topm masked positions rank
      // above this one (higher confidence, or equal at a lower position)
      if (masked) {
        const float v = s_val[l];
        int rank = 0;
        for (int j = 0; j < Lb && rank < a.topm; ++j)
          rank += s_cur[j] == a.mask_id && (s_val[j] > v || (s_val[j] == v && j < l));
        if (rank < a.topm) { f = WINO_DRAFT_FLAG; s_any_draft = 1; }
      }
    } else if (masked) {
      if (cap_now) f = WINO_CAPFILL_FLAG;
      else if (s_val[l] > a.tau1) { f = WINO_DRAFT_FLAG; s_any_draft = 1; }
    } else if ((a.verify || a.standalone) && !cap_now && s_val[l] < a.tau2) {
      f = WINO_REMASK_FLAG;
    }
    s_flag[l] = f;
  }
  __syncthreads();
  if (tid < 64 && a.topm == 0 && !cap_now && a.force_top1 && s_nmask > 0 && !s_any_draft) {
    // Eq. 1: the most confident masked position (lowest position on ties),
    // one wave: per-lane scan, then a shuffle reduction
    int best = INT_MAX;
    float bv = kNegBig;
    for (int l = tid; l < Lb; l += 64)
      if (s_cur[l] == a.mask_id && (best == INT_MAX || s_val[l] > bv)) { best = l; bv = s_val[l]; }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int ob = __shfl_xor(best, o, 64);
      if (ob != INT_MAX && (best == INT_MAX || ov > bv || (ov == bv && ob < best))) { bv = ov; best = ob; }
    }
    if (tid == 0) s_flag[best] = WINO_FORCED_FLAG;
  }
  __syncthreads();
  const int step_no = fin_ptr ? a.seq_steps[b] + 1 : 0;
  for (int l = tid; l < Lb; l += 256) {
    const int f = s_flag[l];
    int t = s_cur[l];
    if (f == WINO_DRAFT_FLAG || f == WINO_FORCED_FLAG || f == WINO_CAPFILL_FLAG) t = s_hat[l];
    else if (f == WINO_REMASK_FLAG) t = a.mask_id;
    if (t != s_cur[l]) {
      cur_ptr[l] = t;
      if (fin_ptr) fin_ptr[l] = step_no;  // Sec. 5.1: last change = finalization
    }
    if (t == a.mask_id) atomicAdd(&s_nmask_after, 1);
    if (a.flags) a.flags[(size_t)b * Lb + l] = (uint8_t)f;
    if (a.bitmap) a.bitmap[(size_t)b * Lb + l] = t == a.mask_id;
  }
  __syncthreads();
  if (a.standalone) {
    if (tid == 0) {
      if (a.n_masked) a.n_masked[b] = s_nmask_after;
      if (a.seq_steps) a.seq_steps[b] += 1;
    }
    return;
  }
  if (tid == 0) {
    if (a.n_masked) a.n_masked[b] = s_nmask_after;
    if (a.seq_steps) a.seq_steps[b] += 1;
    if (a.block_steps) a.block_steps[b] = steps_before + 1;
  }
  advance_block(a, b, s_nmask_after);
}

template <int U>
__global__ __launch_bounds__(256) void decide_kernel(const DecideArgs a) {
  extern __shared__ int smem_i[];
  decide_sequence<U>(a, blockIdx.x, smem_i);
}

// State before the first step of a call.  With advance (decode mode) a
// sequence whose Y_cur holds no mask first moves to the first later block that
// holds one, or to G, and its block step count restarts (a resumed or
// pre-filled state).  Then next_verify[b] = the sequence is active and its
// Y_cur holds both a mask and a non-mask token.  One wave per sequence.
__global__ __launch_bounds__(64) void probe_verify_kernel(const StepGeom g,
                                                          const int32_t* __restrict__ tokens,
                                                          int32_t* __restrict__ next_verify,
                                                          int32_t* block_start, int32_t* block_steps,
                                                          int advance, int32_t* n_masked) {
  const int b = blockIdx.x, lane = threadIdx.x;
  int bs = g.block_start[b];
  const int32_t* resp = tokens + (size_t)b * g.S + g.P;
  if (advance && bs >= 0 && bs < g.G) {
    int first = g.G;
    for (int j = bs + lane; j < g.G; j += 64)
      if (resp[j] == g.mask_id) { first = j; break; }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) first = min(first, __shfl_xor(first, o, 64));
    const int nbs = first >= g.G ? g.G : bs + (first - bs) / g.Lb * g.Lb;
    if (nbs != bs && lane == 0) {
      block_start[b] = nbs;
      if (block_steps) block_steps[b] = 0;
    }
    bs = nbs;
  }
  int nmask = 0, nkeep = 0;
  if (bs < g.G) {
    const int c = bs < 0 ? 0 : (bs > g.G - g.Lb ? g.G - g.Lb : bs);
    for (int l = lane; l < g.Lb; l += 64) {
      const bool m = resp[c + l] == g.mask_id;
      nmask += m;
      nkeep += !m;
    }
  }
  nmask = (int)wave_sum((float)nmask);
  nkeep = (int)wave_sum((float)nkeep);
  if (lane == 0) {
    next_verify[b] = nmask > 0 && nkeep > 0;
    if (n_masked) n_masked[b] = nmask;
  }
}

// Partial softmax statistics of one chunk of CHUNK ids of one needed logits
// row r (the current row of a masked position, the shadow row of an unmasked
// one), written by thread 0 to slot (r, chunk) of the partial arrays.
// Per logit the common path costs a conversion, a max, and one FMA + exp2 +
// add for the sum; the best non-mask id is looked up afterwards only by the
// threads whose maximum equals the chunk's, the mask id is excluded only by
// the thread that holds it, and the target logit is one load.
template <int CHUNK>
__device__ void chunk_stats(const uint16_t* __restrict__ logits, const int32_t* __restrict__ cur, int Lb,
                            int V, int mask_id, int r, int chunk, int n_part, float* pm, float* ps,
                            float* pb, int32_t* pi, float* pt) {
  constexpr int IT = CHUNK / (256 * 8);
  constexpr int STRIDE = 256 * 8;  // ids between a thread's consecutive 16-byte loads
  constexpr float kLog2e = 1.4426950408889634f;
  __shared__ float red[3][4];
  __shared__ int redi[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = r / Lb, l = r - b * Lb;
  const int tok = cur[r];
  const bool masked = tok == mask_id;
  const uint16_t* row = logits + ((size_t)b * 2 * Lb + (masked ? l : Lb + l)) * V;
  const int tgt = masked ? -1 : tok;
  const int v0 = chunk * CHUNK;
  const int v1 = min(V, v0 + CHUNK);
  // the target logit's load goes out with the chunk's, every lane reading the
  // same address (a chunk without the target reads its first id, unused)
  const bool has_tgt = tgt >= v0 && tgt < v1;
  const uint16_t t_raw = row[has_tgt ? tgt : v0];

  uint4 raw[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int idx = v0 + it * STRIDE + tid * 8;
    raw[it] = idx < v1 ? *reinterpret_cast<const uint4*>(row + idx) : make_uint4(0xFF7FFF7Fu, 0xFF7FFF7Fu, 0xFF7FFF7Fu, 0xFF7FFF7Fu);
  }
  // (ids past V read as the most negative finite bf16 and never win)
  auto elem = [&](int it, int e) {
    const uint32_t w = (&raw[it].x)[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
  };
  float mx = kNegBig;
#pragma unroll
  for (int it = 0; it < IT; ++it)
#pragma unroll
    for (int e = 0; e < 8; ++e) mx = fmaxf(mx, elem(it, e));
  // best value over non-mask ids: differs from mx only in the thread holding mask_id
  float nm = mx;
  const int my0 = v0 + tid * 8;  // this thread's ids: my0 + it*STRIDE + e
  if (mask_id >= v0 && mask_id < v1 && (mask_id - my0) >= 0 && ((mask_id - my0) % STRIDE) < 8) {
    nm = kNegBig;
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (my0 + it * STRIDE + e != mask_id) nm = fmaxf(nm, elem(it, e));
  }
  // bz differs from m only in the chunk holding mask_id
  const bool mask_here = mask_id >= v0 && mask_id < v1;
  float m = valu_max<64>(mx), bz = mask_here ? valu_max<64>(nm) : m;
  if (lane == 0) { red[0][wave] = m; red[1][wave] = bz; }
  __syncthreads();
  m = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
  bz = fmaxf(fmaxf(red[1][0], red[1][1]), fmaxf(red[1][2], red[1][3]));
  // lowest non-mask id holding bz (ids grow with it, then e, within a thread)
  int bi = INT_MAX;
  if (nm == bz) {
#pragma unroll
    for (int it = IT - 1; it >= 0; --it)
#pragma unroll
      for (int e = 7; e >= 0; --e) {
        const int id = my0 + it * STRIDE + e;
        if (id < v1 && id != mask_id && elem(it, e) == bz) bi = id;
      }
  }
  const float mc = m * kLog2e;
  // hardware exp2: terms below 2^-126 flush to zero, nothing next to the
  // max's term of one
  float se = 0.f;
#pragma unroll
  for (int it = 0; it < IT; ++it)
#pragma unroll
    for (int e = 0; e < 8; ++e) se += __builtin_amdgcn_exp2f(fmaf(elem(it, e), kLog2e, -mc));
  se = valu_sum<64>(se);
  bi = valu_min<64>(bi);
  if (lane == 0) { red[2][wave] = se; redi[wave] = bi; }
  __syncthreads();
  if (tid == 0) {
    const float s = (red[2][0] + red[2][1]) + (red[2][2] + red[2][3]);
    const int ii = min(min(redi[0], redi[1]), min(redi[2], redi[3]));
    const float tt = has_tgt ? bf2f(t_raw) : kNegBig;
    const size_t o = (size_t)r * n_part + chunk;
    pm[o] = m; ps[o] = s; pb[o] = bz; pi[o] = ii; pt[o] = tt;
  }
}

// Standalone epilogue statistics: workgroup (chunk, r) writes the partial
// statistics of its chunk of row r; decide_kernel then merges and decides.
// (One launch, with the last workgroup of each sequence deciding, was 2.7-6x
// slower: the device-scope release each workgroup needs before counting
// itself done writes back its XCD's L2.)
template <int CHUNK>
__global__ __launch_bounds__(256) void epi_stats_kernel(const uint16_t* __restrict__ logits,
                                                        const int32_t* __restrict__ cur, int Lb, int V,
                                                        int mask_id, float* pm, float* ps, float* pb,
                                                        int32_t* pi, float* pt, int n_part) {
  chunk_stats<CHUNK>(logits, cur, Lb, V, mask_id, blockIdx.y, blockIdx.x, n_part, pm, ps, pb, pi, pt);
}

}  // namespace

// WINO+ per-row quantities: one wave per row merges the n_part tile partials
// (max, sum-exp, entropy term, best non-mask id, target logit).
__global__ __launch_bounds__(256) void loss_merge_kernel(const LmStatsOut lm, int R,
                                                         float4* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= R) return;
  float m = kNegBig, s = 0.f, z = 0.f, bz = kNegBig, tz = kNegBig;
  int bi = INT_MAX;
  for (int j = lane; j < lm.n_part; j += 64) {
    const size_t o = (size_t)r * lm.n_part + j;
    const float pm = lm.pm[o], ps = lm.ps[o], pz = lm.pz[o];
    const float mn = fmaxf(m, pm);
    const float fa = __expf(m - mn), fb = __expf(pm - mn);
    // sum e^{z-mn}(z-mn) over both parts, each rebased from its own max
    z = fa * (z + (m - mn) * s) + fb * (pz + (pm - mn) * ps);
    s = s * fa + ps * fb;
    m = mn;
    const float ob = lm.pb[o];
    const int oi = lm.pi[o];
    if (ob > bz || (ob == bz && oi < bi)) { bz = ob; bi = oi; }
    tz = fmaxf(tz, lm.pt[o]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float om = __shfl_xor(m, off, 64), os = __shfl_xor(s, off, 64), oz = __shfl_xor(z, off, 64);
    const float mn = fmaxf(m, om);
    const float fa = __expf(m - mn), fb = __expf(om - mn);
    z = fa * (z + (m - mn) * s) + fb * (oz + (om - mn) * os);
    s = s * fa + os * fb;
    m = mn;
    const float ob = __shfl_xor(bz, off, 64);
    const int oi = __shfl_xor(bi, off, 64);
    if (ob > bz || (ob == bz && oi < bi)) { bz = ob; bi = oi; }
    tz = fmaxf(tz, __shfl_xor(tz, off, 64));
  }
  if (lane == 0) {
    const float ls = __logf(s);
    // H = log S - sum e^{z-m}(z-m) / S;  -log p(t) = m + log S - z_t
    out[r] = make_float4(ls - z / s, m + ls - tz, __expf(bz - m) / s, __int_as_float(bi));
  }
}

hipError_t launch_loss_merge(const LmStatsOut& lm, int R, void* out, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  loss_merge_kernel<<<(R + 3) / 4, 256, 0, st>>>(lm, R, static_cast<float4*>(out));
  return hipGetLastError();
}

hipError_t launch_probe_verify(const StepGeom& g, const int32_t* tokens, int32_t* next_verify,
                               hipStream_t st, int32_t* block_start, int32_t* block_steps,
                               int32_t* n_masked) {
  probe_verify_kernel<<<g.B, 64, 0, st>>>(g, tokens, next_verify, block_start, block_steps,
                                          block_start != nullptr, n_masked);
  return hipGetLastError();
}

hipError_t launch_decide(const DecideArgs& a, hipStream_t st) {
  const size_t shm = (size_t)a.Lb * 16;
  // U = 2 covers up to 2*gs partials per position in one batch (the
  // standalone epilogue); the LM head's many vocabulary tiles take batches of 8
  if (a.n_part <= 2 * merge_lanes(a.Lb) && a.Lb <= 256) decide_kernel<2><<<a.B, 256, shm, st>>>(a);
  else decide_kernel<8><<<a.B, 256, shm, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_epilogue_stats(const uint16_t* logits, const int32_t* cur_tokens, int B, int Lb,
                                 int V, int mask_id, float* pm, float* ps, float* pb, int32_t* pi,
                                 float* pt, hipStream_t st) {
  const int n_part = (V + kEpiChunk - 1) / kEpiChunk;
  dim3 grid(n_part, B * Lb);
  epi_stats_kernel<kEpiChunk><<<grid, 256, 0, st>>>(logits, cur_tokens, Lb, V, mask_id, pm, ps, pb, pi, pt,
                                                    n_part);
  return hipGetLastError();
}

}  // namespace wino
