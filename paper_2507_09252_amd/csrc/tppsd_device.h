// Device helpers shared by the HIP translation units of libtppsd: bf16
// conversions, typed loads/stores, the value-cache index, cross-lane
// reductions and the MFMA operand vector types.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tppsd_internal.h"

namespace tppsd {

// bf16 MFMA operands are only ever produced by whole-vector loads or by
// bit-casting packed 32-bit words; individual __bf16 elements are never read
// or written (element access on __bf16 vectors gave wrong values on gfx950).
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// scalar helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// float -> bf16, round to nearest even: gfx950's conversion instruction
// (v_cvt_pk_bf16_f32, two values per instruction; for finite values it
// gives the same bits as adding 0x7FFF + the kept lsb and truncating)
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
// the pair (lo, hi) packed into one word, lo in the low half
__device__ __forceinline__ uint32_t pk2bf(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, (bf16x2_t){(__bf16)lo, (__bf16)hi});
}

// acc + w.lo x.lo + w.hi x.hi over two packed bf16 pairs (v_dot2c_f32_bf16;
// each product is exact in fp32)
__device__ __forceinline__ float dot2_bf(uint32_t w, uint32_t x, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w), __builtin_bit_cast(bf16x2_t, x), acc, false);
}

template <typename T> __device__ __forceinline__ float ld(const T *p, size_t i);
template <> __device__ __forceinline__ float ld<float>(const float *p, size_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t *p, size_t i) { return bf2f(p[i]); }

template <typename T> __device__ __forceinline__ void st(T *p, size_t i, float v);
template <> __device__ __forceinline__ void st<float>(float *p, size_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<bf16_t>(bf16_t *p, size_t i, float v) { p[i] = f2bf(v); }

// Value cache element (position pos, column j) of the (sequence, head) slab
// whose first position is row0 = (b H + h) kv_cap. fp32 values are stored
// row per position like the keys; bf16 values in blocks of 8 positions,
// [kv_cap / 8][dh][8], so that 8 consecutive positions of one column are one
// 16-byte load (the operand layout of the P V matrix product).
template <typename ACT> __device__ __forceinline__ size_t v_at(size_t row0, int pos, int j, int dh);
template <> __device__ __forceinline__ size_t v_at<float>(size_t row0, int pos, int j, int dh) {
  return (row0 + pos) * dh + j;
}
template <> __device__ __forceinline__ size_t v_at<bf16_t>(size_t row0, int pos, int j, int dh) {
  return row0 * dh + (size_t)(pos >> 3) * (8 * dh) + j * 8 + (pos & 7);
}

// Cross-lane moves: DPP within rows of 16 lanes (quad permutes, row
// rotations), LDS swizzles (xor masks within 32 lanes) and one bpermute for
// lane ^ 32. The whole wave must be active.
template <int CTRL> __device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int XOR> __device__ __forceinline__ float swz_xor(float v) {
  static_assert(XOR < 32, "swizzle reaches 32 lanes");
  return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), (XOR << 10) | 0x1F));
}
// sum / max over aligned groups of `width` lanes (a power of two <= 64),
// left in every lane of the group
__device__ __forceinline__ float group_sum(float v, int width) {
  if (width >= 2) v += dpp_mov<0xB1>(v);   // quad_perm(1, 0, 3, 2): lane ^ 1
  if (width >= 4) v += dpp_mov<0x4E>(v);   // quad_perm(2, 3, 0, 1): lane ^ 2
  if (width >= 8) v += swz_xor<4>(v);
  if (width >= 16) v += swz_xor<8>(v);
  if (width >= 32) v += swz_xor<16>(v);
  if (width >= 64) v += __shfl_xor(v, 32, 64);
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x124>(v);   // row_ror:4
  v += dpp_mov<0x128>(v);   // row_ror:8 -> every lane holds its row's sum
  return (__int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)) +
          __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16))) +
         (__int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32)) +
          __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48)));
}
// inclusive running sum over the wave (lane i: v_0 + ... + v_i), DPP only:
// shifts by 1, 2, 4, 8 within rows of 16 lanes, then each row's last lane
// broadcast onward (row_bcast:15 into rows 1 and 3, row_bcast:31 into rows 2
// and 3). Lanes a shift leaves without a source add the 0 they start from.
__device__ __forceinline__ float wave_cumsum(float v) {
  v += dpp_mov<0x111>(v);   // row_shr:1
  v += dpp_mov<0x112>(v);   // row_shr:2
  v += dpp_mov<0x114>(v);   // row_shr:4
  v += dpp_mov<0x118>(v);   // row_shr:8
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xA, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x143, 0xC, 0xF, false));
  return v;
}
// lane i's value of v (i wave-uniform)
__device__ __forceinline__ float lane_val(float v, int i) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));
  v = fmaxf(v, dpp_mov<0x4E>(v));
  v = fmaxf(v, dpp_mov<0x124>(v));
  v = fmaxf(v, dpp_mov<0x128>(v));
  return fmaxf(fmaxf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)),
                     __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16))),
               fmaxf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32)),
                     __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48))));
}

}  // namespace tppsd
