// Internal helpers shared by the HIP sources of libsckv.so (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "../../include/sckv.h"

#define SCKV_INF_VU 0x7fffffff

namespace sckv {

// ---------------------------------------------------------------------------
// host side: error reporting
// ---------------------------------------------------------------------------
void set_error(const std::string& msg);
void clear_error();
int fail(int code, const std::string& msg);
int hip_check(hipError_t e, const char* what);

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline int elem_bytes(sckv_dtype dt) { return dt == SCKV_F32 ? 4 : 2; }
inline bool valid_dtype(int dt) { return dt == SCKV_F32 || dt == SCKV_BF16; }
inline bool supported_d(int d) { return d == 64 || d == 80; }

// ---------------------------------------------------------------------------
// device side
// ---------------------------------------------------------------------------
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// round-to-nearest-even fp32 -> bf16 (hardware conversion on gfx950)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
// two fp32 -> two bf16 (RNE) in one v_cvt_pk_bf16_f32; lo in bits 0..15
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// 16-byte piece of a row as floats (8 for bf16, 4 for f32)
template <typename T> struct Piece;
template <> struct Piece<uint16_t> {
  static constexpr int E = 8;
  __device__ __forceinline__ static void unpack(const u32x4& w, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) { f[2 * i] = bf16_lo(w[i]); f[2 * i + 1] = bf16_hi(w[i]); }
  }
  __device__ __forceinline__ static u32x4 pack(const float* f) {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(f[2 * i], f[2 * i + 1]);
    return w;
  }
};
template <> struct Piece<float> {
  static constexpr int E = 4;
  __device__ __forceinline__ static void unpack(const u32x4& w, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(w[i]);
  }
  __device__ __forceinline__ static u32x4 pack(const float* f) {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = __float_as_uint(f[i]);
    return w;
  }
};

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// 2^x with the hardware instruction; results below 2^-126 flush to zero,
// which is what a softmax weight of that size contributes anyway
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ds_read_b64_tr_b16 (gfx950): inside each group of 16 lanes, lane i gets
// element e = (the 4 halves at lane 4e + i/4's address)[i % 4]
__device__ __forceinline__ s16x4 lds_read_tr16(const void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(const_cast<void*>(p)));
}

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }

// wait until every outstanding vector-memory load of this wave has returned
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// cross-lane moves inside a row of 16 lanes (DPP; no LDS traffic)
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL,
                                                               0xf, 0xf, false));
}
constexpr int DPP_QUAD_XOR1 = 0xb1;      // quad_perm [1,0,3,2]
constexpr int DPP_QUAD_XOR2 = 0x4e;      // quad_perm [2,3,0,1]
constexpr int DPP_ROW_MIRROR = 0x140;    // lane i <- lane 15-i within a row
constexpr int DPP_ROW_HALF_MIRROR = 0x141;  // lane i <- lane 7-i within a half row

// sum over aligned groups of GRP lanes (8, 16 or 32); every lane gets the sum
template <int GRP>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(GRP == 8 || GRP == 16 || GRP == 32, "group size");
  x += dpp_mov<DPP_QUAD_XOR1>(x);
  x += dpp_mov<DPP_QUAD_XOR2>(x);
  x += dpp_mov<DPP_ROW_HALF_MIRROR>(x);
  if constexpr (GRP >= 16) x += dpp_mov<DPP_ROW_MIRROR>(x);
  if constexpr (GRP >= 32) x += __shfl_xor(x, 16, 64);
  return x;
}

__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0)); }

// number of set bits of a 64-bit wave mask strictly below this lane
__device__ __forceinline__ int mask_rank(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

}  // namespace sckv
