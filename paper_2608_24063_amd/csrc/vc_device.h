// vc_device.h -- gfx950 device helpers for the PruneKV kernels: bf16 vector
// types, the 16x16x32 bf16 MFMA, wave64 shuffles and the XCD-aware block
// remap.  Internal to libviscache.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

// Pointers the kernels read from the plan are generic; accesses through them
// compile to flat instructions, which on gfx9 also count against the LDS wait
// counter and so stall every LDS read behind in-flight global loads.  All
// global memory traffic goes through these global-address-space views.
#define VC_GLOBAL __attribute__((address_space(1)))

template <typename T>
__device__ __forceinline__ const VC_GLOBAL T *gp(const T *p) {
  return (const VC_GLOBAL T *)p;
}
template <typename T>
__device__ __forceinline__ VC_GLOBAL T *gp(T *p) {
  return (VC_GLOBAL T *)p;
}
// 16- and 8-byte global loads / stores at element pointer p.
template <typename T>
__device__ __forceinline__ u32x4 ld16(const T *p) {
  return *reinterpret_cast<const VC_GLOBAL u32x4 *>(gp(p));
}
template <typename T>
__device__ __forceinline__ u32x2 ld8(const T *p) {
  return *reinterpret_cast<const VC_GLOBAL u32x2 *>(gp(p));
}
template <typename T>
__device__ __forceinline__ void st16(T *p, u32x4 v) {
  *reinterpret_cast<VC_GLOBAL u32x4 *>(gp(p)) = v;
}
template <typename T>
__device__ __forceinline__ void st8(T *p, u32x2 v) {
  *reinterpret_cast<VC_GLOBAL u32x2 *>(gp(p)) = v;
}
template <typename T>
__device__ __forceinline__ T ldg(const T *p) {
  return *gp(p);
}
template <typename T>
__device__ __forceinline__ void stg(T *p, T v) {
  *gp(p) = v;
}
// float2 is a class type that cannot be accessed through an address-space
// qualified reference; move it as two 32-bit words.
__device__ __forceinline__ float2 ldg(const float2 *p) {
  const u32x2 v = ld8(p);
  return make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
}
__device__ __forceinline__ void stg(float2 *p, float2 v) {
  st8(p, u32x2{__float_as_uint(v.x), __float_as_uint(v.y)});
}
constexpr int kXcds = 8;  // MI355X: 8 accelerator complex dies, 32 CUs each

// D = A(16x32) * B(32x16) + C on the matrix cores.  Lane l holds row l%16 of A
// and column l%16 of B, each with the 8 k-elements of lane group l/16; D comes
// back with column l%16 and rows 4*(l/16)+i in element i.  Callers pick the
// same k-element order for A and B, so the order itself is free.
__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ u32x4 as_u32x4(bf16x8 v) { return __builtin_bit_cast(u32x4, v); }

// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Round a float to bf16 precision and return it as float.
__device__ __forceinline__ float round_bf16(float x) {
  return __uint_as_float(pack_bf16(x, 0.f) << 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <typename T>
__device__ __forceinline__ T shfl_xor(T v, int mask) {
  return __shfl_xor(v, mask, 64);
}

// Exchanges between lanes i and i ^ 16 / i ^ 32 that need no lane-index
// register (the generic shuffle keeps per-lane indices live across loops):
// an LDS swizzle swaps the 16-lane groups of each 32-lane half, and gfx950's
// v_permlane32_swap swaps the two halves, so max / sum over the pair i,
// i ^ 32 come out in every lane.
__device__ __forceinline__ float swap16(float x) {
  return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), 0x401F));  // and 0x1F, xor 0x10
}
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Inclusive prefix sum over the 64 lanes of a wave (DPP: shifts within rows
// of 16 lanes, then row broadcasts).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

// Block index remapped so that consecutive logical indices land on the same
// XCD: the hardware deals workgroups round-robin over the 8 XCDs, and each XCD
// has its own L2.  Logical blocks [x*per, (x+1)*per) run on XCD x.
__device__ __forceinline__ uint32_t xcd_block(uint32_t bid, uint32_t nblocks) {
  uint32_t per = nblocks / kXcds, rem = nblocks % kXcds;
  uint32_t x = bid % kXcds, slot = bid / kXcds;
  // XCDs [0, rem) receive per+1 blocks, the others per.
  uint32_t base = x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per;
  return base + slot;
}

}  // namespace vc
