// Device-side helpers shared by the WINO kernels (gfx950 / CDNA4, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace wino {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr float kNegBig = -3.0e38f;  // finite "minus infinity" for max-reductions

__device__ __forceinline__ float bf2f(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;

// fp32 -> bf16 pairs, round to nearest even: one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint16_t f2bf(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// 32x32x16 bf16 MFMA, fp32 accumulate.  Operand layout (wave64): lane l holds
// row (A) / column (B) l%32 and the 8 consecutive k of group l/32.  Result:
// lane l holds column l%32, rows 8*(i/4) + 4*(l/32) + i%4 for i = 0..15.
__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ int mfma_row(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

// Butterfly reductions over a full wave (64 lanes) or over 32-lane halves.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Activation element types of the matrix-core operands (activations and the
// weights they multiply): bf16, or fp16 for three more mantissa bits where
// decisions near a threshold need them.  Storage is 16-bit either way;
// conversions round to nearest even; accumulation is fp32.
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;
struct ActBf16 {
  typedef bf16x8 v8;
  static constexpr bool kF16 = false;
  __device__ static __forceinline__ v8 frag(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }
  __device__ static __forceinline__ f32x16 mma(const v8& a, const v8& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ uint32_t pack2(float lo, float hi) { return pack2bf(lo, hi); }
  __device__ static __forceinline__ uint16_t cvt(float f) { return f2bf(f); }
  __device__ static __forceinline__ float val(uint16_t v) { return bf2f(v); }
};
struct ActF16 {
  typedef f16x8 v8;
  static constexpr bool kF16 = true;
  __device__ static __forceinline__ v8 frag(const uint4& v) { return __builtin_bit_cast(f16x8, v); }
  __device__ static __forceinline__ f32x16 mma(const v8& a, const v8& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ uint32_t pack2(float lo, float hi) {
    const f16x2 v = {(_Float16)lo, (_Float16)hi};
    return __builtin_bit_cast(uint32_t, v);
  }
  __device__ static __forceinline__ uint16_t cvt(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
  __device__ static __forceinline__ float val(uint16_t v) { return (float)__builtin_bit_cast(_Float16, v); }
};

// Reductions on the vector ALU alone, without the LDS round trip of a
// shuffle per step: DPP lane swaps inside quads (xor 1, xor 2), the half-row
// and row mirrors (groups of 8 and 16 lanes), then rows 0<->1 and 2<->3
// (v_permlane16_swap: groups of 32) and the two halves (v_permlane32_swap:
// 64).  op must be commutative and associative; every lane of a group ends
// with the group's result (both lanes of each pair combine the same two
// values).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
template <int LANES, class Op>
__device__ __forceinline__ uint32_t valu_reduce(uint32_t v, Op op) {
  static_assert(LANES == 32 || LANES == 64, "groups of 32 or 64 lanes");
  v = op(v, dpp_mov<0xB1>(v));   // quad_perm [1,0,3,2]
  v = op(v, dpp_mov<0x4E>(v));   // quad_perm [2,3,0,1]
  v = op(v, dpp_mov<0x141>(v));  // row_half_mirror
  v = op(v, dpp_mov<0x140>(v));  // row_mirror
  auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = op(r[0], r[1]);
  if constexpr (LANES == 64) {
    r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    v = op(r[0], r[1]);
  }
  return v;
}
template <int LANES>
__device__ __forceinline__ float valu_max(float x) {
  return __uint_as_float(valu_reduce<LANES>(__float_as_uint(x), [](uint32_t a, uint32_t b) {
    return __float_as_uint(fmaxf(__uint_as_float(a), __uint_as_float(b)));
  }));
}
template <int LANES>
__device__ __forceinline__ float valu_sum(float x) {
  return __uint_as_float(valu_reduce<LANES>(__float_as_uint(x), [](uint32_t a, uint32_t b) {
    return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
  }));
}
template <int LANES>
__device__ __forceinline__ int valu_min(int x) {
  return (int)valu_reduce<LANES>((uint32_t)x, [](uint32_t a, uint32_t b) { return (uint32_t)min((int)a, (int)b); });
}
// (value, id) pairs: the largest value, the lowest id among equal values.
template <int LANES>
__device__ __forceinline__ void valu_argmax(float& v, int& id) {
  auto take = [&](float ov, int oi) {
    if (ov > v || (ov == v && oi < id)) { v = ov; id = oi; }
  };
  auto step = [&](auto ctrl) {
    constexpr int C = decltype(ctrl)::value;
    take(__uint_as_float(dpp_mov<C>(__float_as_uint(v))), (int)dpp_mov<C>((uint32_t)id));
  };
  step(std::integral_constant<int, 0xB1>{});
  step(std::integral_constant<int, 0x4E>{});
  step(std::integral_constant<int, 0x141>{});
  step(std::integral_constant<int, 0x140>{});
  auto swap = [&](auto rv, auto ri) {
    // rv / ri: this lane's value and its partner's, in some order
    const float a = __uint_as_float(rv[0]), b = __uint_as_float(rv[1]);
    const int ia = (int)ri[0], ib = (int)ri[1];
    const bool second = b > a || (b == a && ib < ia);
    v = second ? b : a;
    id = second ? ib : ia;
  };
  swap(__builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false),
       __builtin_amdgcn_permlane16_swap((uint32_t)id, (uint32_t)id, false, false));
  if constexpr (LANES == 64)
    swap(__builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false),
         __builtin_amdgcn_permlane32_swap((uint32_t)id, (uint32_t)id, false, false));
}

// Reductions over the lane pair (l, l ^ 32): v_permlane32_swap exchanges the
// two 32-lane halves between registers, where a shuffle goes through the LDS
// crossbar (ds_bpermute) and its latency.  Both lanes get the same value.
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS-DMA of 16 bytes per lane (global_load_lds_dwordx4) into the 1 KB block
// at l + j KB (j = 0..3): the LDS base goes to M0 and j KB into the
// instruction's offset, which applies to the global address as well, so g
// is the source pointer minus j KB.  Up to four consecutive blocks of a wave
// then share one M0 value; every M0 write costs issue time next to the MFMAs.
__device__ __forceinline__ void dma16(const uint16_t* g, uint16_t* l, int j) {
  auto* ld = (__attribute__((address_space(3))) void*)l;
  switch (j) {
    case 0: __builtin_amdgcn_global_load_lds((const void*)g, ld, 16, 0, 0); break;
    case 1: __builtin_amdgcn_global_load_lds((const void*)g, ld, 16, 1024, 0); break;
    case 2: __builtin_amdgcn_global_load_lds((const void*)g, ld, 16, 2048, 0); break;
    default: __builtin_amdgcn_global_load_lds((const void*)g, ld, 16, 3072, 0); break;
  }
}

// A pointer known to be the same in every lane, moved to scalar registers
// (values computed on the vector unit, e.g. from a division, otherwise make
// the compiler loop over lanes to build a buffer resource from them).
template <class T>
__device__ __forceinline__ T* uniform_ptr(T* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<T*>(((uint64_t)hi << 32) | lo);
}

// Raw buffer resources (stride 0; the range is in bytes): word 3 for the gfx9
// family, and a vector offset beyond any range used here, whose access the
// range check drops (loads return 0).
constexpr int kBufferDword3 = 0x00020000;
constexpr int kBufferOffNone = INT32_MIN;

// Map a hardware workgroup id to a logical tile id so that each XCD (work is
// dealt round-robin to 8 XCDs) receives one contiguous range of logical tiles;
// neighbouring tiles then share that XCD's L2.
__device__ __forceinline__ int xcd_remap(int p, int n) {
  const int q = n >> 3, r = n & 7;
  const int x = p & 7, slot = p >> 3;
  return x * q + (x < r ? x : r) + slot;
}

}  // namespace wino
