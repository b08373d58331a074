// Device-side building blocks shared by the libcats kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cats {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaveSize = 64;

// Weight element types.  bf16 is carried as its raw 16-bit pattern; it is
// widened to fp32 exactly by placing the bits in the upper half of a word.
struct wbf16 {};
struct wf32 {};

template <typename WT> struct wtraits;
template <> struct wtraits<wbf16> {
  typedef uint16_t elem;
  static constexpr int VEC = 8;  // elements per 16-byte vector
};
template <> struct wtraits<wf32> {
  typedef float elem;
  static constexpr int VEC = 4;
};

// Byte offset that lies outside every buffer the kernels address: a
// buffer load at (a sum of at most two of) these offsets returns zeros and
// moves no data.  Buffers are limited to kBufMaxBytes so that a valid offset
// plus one kOOB never wraps back into range.
constexpr uint32_t kOOB = 0x40000000u;
constexpr uint64_t kBufMaxBytes = 0x40000000ull;

// Buffer resource over [base, base + bytes) for raw (stride 0) loads; the
// last word is the gfx9-family default format.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// 16-byte load through a buffer resource.  Out-of-range offsets read as
// zero without touching memory, which predicates a load without a branch:
// every load instruction then executes on every path, so the compiler can
// count outstanding loads exactly and keep prefetches in flight.  The
// non-temporal policy keeps the one-shot weight stream from evicting
// reusable lines (x, partial sums) from L2 and the MALL.
__device__ __forceinline__ u32x4 ld_buf16_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 2 /* nt */);
}

__device__ __forceinline__ u32x4 ld_buf16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}

// Device-coherent 16-byte load and store (cache policy sc1): they reach the
// memory level shared by every XCD, so blocks on different XCDs can exchange
// data within one kernel without a cache-wide write-back or invalidation.
constexpr int kCachePolicySc1 = 16;

__device__ __forceinline__ u32x4 ld_buf16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kCachePolicySc1);
}

__device__ __forceinline__ void st_buf16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)off, 0, kCachePolicySc1);
}

__device__ __forceinline__ u32x4 zero_u32x4() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return z;
}

// Widen one 16-byte vector of weights to fp32.
template <typename WT> __device__ __forceinline__ void widen(const u32x4& v, float* f);

template <> __device__ __forceinline__ void widen<wbf16>(const u32x4& v, float* f) {
  // little endian: element 2i is the low half of word i
  f[0] = __uint_as_float(v.x << 16);
  f[1] = __uint_as_float(v.x & 0xffff0000u);
  f[2] = __uint_as_float(v.y << 16);
  f[3] = __uint_as_float(v.y & 0xffff0000u);
  f[4] = __uint_as_float(v.z << 16);
  f[5] = __uint_as_float(v.z & 0xffff0000u);
  f[6] = __uint_as_float(v.w << 16);
  f[7] = __uint_as_float(v.w & 0xffff0000u);
}

template <> __device__ __forceinline__ void widen<wf32>(const u32x4& v, float* f) {
  f[0] = __uint_as_float(v.x);
  f[1] = __uint_as_float(v.y);
  f[2] = __uint_as_float(v.z);
  f[3] = __uint_as_float(v.w);
}

// DPP row permutation of a float (GFX9 encodings).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

__device__ __forceinline__ float lane_f32(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Sum over the 64 lanes of a wave; needs all lanes active.  Within each row
// of 16 lanes: swap neighbours, swap pairs, mirror halves, mirror the row
// (quad_perm [1,0,3,2], [2,3,0,1], row_half_mirror, row_mirror).  Each lane
// adds the same two operands as its partner at every stage, so all 16 lanes
// of a row hold the bitwise-identical row sum; the four row sums are then
// read out and added in a fixed order.  The result is uniform and does not
// depend on scheduling.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32<0xb1>(v);
  v += dpp_f32<0x4e>(v);
  v += dpp_f32<0x141>(v);
  v += dpp_f32<0x140>(v);
  return (lane_f32(v, 0) + lane_f32(v, 16)) + (lane_f32(v, 32) + lane_f32(v, 48));
}

// Make a value that is equal on all lanes visibly uniform to the compiler,
// so branches on it become scalar branches.
__device__ __forceinline__ float uniform_f32(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

__device__ __forceinline__ uint32_t uniform_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

// bf16 bit pattern nearest to f (ties to even); NaN stays a quiet NaN.
// x = bf16(x) + bf16(x - bf16(x)) holds 16 of fp32's 24 significand bits,
// and a bf16 weight times either part is exact in fp32: the split the
// matrix-core paths use for fp32 inputs.
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rne = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  return ((u & 0x7fffffffu) > 0x7f800000u) ? ((u >> 16) | 0x40u) : rne;
}

// SiLU(z) = z / (1 + e^{-z}).  For z below about -88 e^{-z} overflows to
// +inf and the result is -0, whose magnitude 0 is masked by any t > 0.
__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

}  // namespace cats
