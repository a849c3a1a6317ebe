// Device-side helpers shared by the gfx950 kernels of the probe forward.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sp {

// Context length of sequence b, clamped to [0, max_seq_len].
__device__ __forceinline__ int clamp_len(const int* seq_lens, int b, int max_seq_len) {
  int n = seq_lens[b];
  return n < 0 ? 0 : (n > max_seq_len ? max_seq_len : n);
}


typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
// Running-max start value: finite, so exp2(start - m) is 0 rather than NaN.
constexpr float kNegBig = -1.0e30f;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(f16 x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }  // RNE
template <> __device__ __forceinline__ f16 from_f32<f16>(float x) { return (f16)x; }     // RNE

// Two bf16 values packed in a dword -> the same two values as fp16.  Exact for
// magnitudes in fp16's normal range [2^-14, 65504]; larger ones saturate, smaller
// ones become fp16 subnormals (round toward zero).
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t v) {
  const float lo = __builtin_bit_cast(float, v << 16);
  const float hi = __builtin_bit_cast(float, v & 0xffff0000u);
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo, hi));
}
__device__ __forceinline__ uint4 bf16x8_to_f16x8(uint4 v) {
  return make_uint4(bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y), bf16x2_to_f16x2(v.z),
                    bf16x2_to_f16x2(v.w));
}
__device__ __forceinline__ u32x4 bf16x8_to_f16x8(u32x4 v) {
  return u32x4{bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y), bf16x2_to_f16x2(v.z), bf16x2_to_f16x2(v.w)};
}
__device__ __forceinline__ uint2 bf16x4_to_f16x4(uint2 v) {
  return make_uint2(bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y));
}

// 16-byte global load / store.
__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }

// Streaming (non-temporal) loads for data read exactly once, such as the KV
// cache: they do not displace reusable lines in the caches.
__device__ __forceinline__ uint4 ld16_stream(const void* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ u32x4 ld16v_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x4 ld16v(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ u32x2 ld8v(const void* p) { return *reinterpret_cast<const u32x2*>(p); }
__device__ __forceinline__ uint2 ld8_stream(const void* p) {
  const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
  return make_uint2(v.x, v.y);
}

__device__ __forceinline__ f16x8 as_f16x8(uint4 v) { return __builtin_bit_cast(f16x8, v); }
__device__ __forceinline__ f16x4 as_f16x4(uint2 v) { return __builtin_bit_cast(f16x4, v); }

// D(16x16, fp32) += A(16x32, fp16) * B(32x16, fp16).
// Lane l holds A[l%16][8(l/16) .. 8(l/16)+7], B[8(l/16) .. +7][l%16];
// D lane l holds rows 4(l/16) + r, r = 0..3, of column l%16.
__device__ __forceinline__ f32x4 mfma16x16x32(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// The same two shapes with bf16 operands (identical lane layouts).
__device__ __forceinline__ f32x4 mfma16x16x32_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// D(16x16, fp32) += A(16x16, fp16) * B(16x16, fp16).
// Lane l holds A[l%16][4(l/16) .. 4(l/16)+3], B[4(l/16) .. +3][l%16]; D as above.
__device__ __forceinline__ f32x4 mfma16x16x16(f16x4 a, f16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Block-wide sum for blockDim.x == 256 (4 waves); `red` holds >= 4 floats.
__device__ __forceinline__ float block_sum_256(float v, float* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// ---------------------------------------------------------------- direct loads into LDS
// Direct global -> LDS load of 16 bytes per lane from base + lane_off (base
// uniform across the wave, in SGPRs): lane l's bytes land at wave_dst + 16 l
// (wave_dst uniform, in M0).  STREAM: non-temporal, for data read once (the KV
// cache); otherwise the lines stay cached for other workgroups (weights and
// activations of the projections).  Written as inline asm so that the compiler
// does not order later LDS reads after it with a full vmcnt(0): the kernel
// waits for these loads itself (wait_vmcnt, then lds_barrier).  The
// vector-memory counter retires in order, so loads the compiler does not count
// only make its own waits for other loads stricter.
template <bool STREAM = true>
__device__ __forceinline__ void ld16_to_lds(const void* base, uint32_t lane_off, u32x4* wave_dst) {
  const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) u32x4*)wave_dst;
  if (STREAM)
    asm volatile("global_load_lds_dwordx4 %0, %1 nt" : : "v"(lane_off), "s"(base), "{m0}"(lds) : "memory");
  else
    asm volatile("global_load_lds_dwordx4 %0, %1" : : "v"(lane_off), "s"(base), "{m0}"(lds) : "memory");
}

// s_waitcnt vmcnt(N) alone (expcnt and lgkmcnt left unconstrained).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// Workgroup barrier for LDS traffic: waits for this wave's LDS operations
// (lgkmcnt) but not for its outstanding global loads, so direct-to-LDS loads of
// later units stay in flight; the caller first waits (vmcnt) for those that must
// have landed.  The empty asm statements keep the compiler from moving memory
// accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt unconstrained
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace sp
