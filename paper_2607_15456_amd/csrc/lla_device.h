// Device-side helpers shared by the LLA HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lla {

constexpr int kPage = 64;      // tokens per cache page (feature-major inside a page)
constexpr int kWave = 64;      // CDNA wavefront width
constexpr int kMaxRank = 512;  // largest r_k / r_v accepted
constexpr int kMaxHead = 256;  // largest d_head accepted

typedef uint16_t bf16_t;  // bfloat16 storage

// ---- bf16 <-> fp32 -------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(bf16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// Round-to-nearest-even fp32 -> bf16; NaN stays NaN (quiet bit set).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

// Element access for the two input types.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kPer16B = 4;
  __device__ __forceinline__ static float get(const float* p, size_t i) { return p[i]; }
  __device__ __forceinline__ static void unpack(const uint4& v, float (&o)[4]) {
    o[0] = __uint_as_float(v.x); o[1] = __uint_as_float(v.y);
    o[2] = __uint_as_float(v.z); o[3] = __uint_as_float(v.w);
  }
};
template <> struct Elem<bf16_t> {
  static constexpr int kPer16B = 8;
  __device__ __forceinline__ static float get(const bf16_t* p, size_t i) { return bf16_to_f32(p[i]); }
  __device__ __forceinline__ static void unpack(const uint4& v, float (&o)[8]) {
    o[0] = bf16_lo(v.x); o[1] = bf16_hi(v.x); o[2] = bf16_lo(v.y); o[3] = bf16_hi(v.y);
    o[4] = bf16_lo(v.z); o[5] = bf16_hi(v.z); o[6] = bf16_lo(v.w); o[7] = bf16_hi(v.w);
  }
};

template <typename T> __device__ __forceinline__ void store_out(T* p, size_t i, float v);
template <> __device__ __forceinline__ void store_out<float>(float* p, size_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, size_t i, float v) {
  p[i] = f32_to_bf16(v);
}

__device__ __forceinline__ uint4 ld16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

// 16-byte load with the non-temporal cache policy ("nt"), for data a kernel
// reads exactly once: it then does not displace reusable lines in L2 / MALL.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_nt(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Waits until this wavefront's earlier global stores are acknowledged by L2.
// Split-K partials: every wavefront waits this way, then after a workgroup
// barrier one thread's agent-scope release (a single L2 write-back) publishes
// the whole workgroup's stores.  A workgroup-scope release alone does not wait
// for outstanding stores (all wavefronts of a workgroup share one compute
// unit), so without it a wavefront's stores could still be in flight when that
// write-back runs.
__device__ __forceinline__ void wait_stores_in_l2() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Workgroup coordinates (x, y = head) renumbered so that every workgroup of a
// head runs on one XCD: the linear workgroup i = x + gridDim.x * y is
// dispatched to XCD i % 8, so when the head count is a multiple of 8, XCD c
// takes heads c, c + 8, ... and its L2 holds only their up-projections
// (otherwise every XCD fetches every head's).  A bijection on the grid; other
// head counts, and on = false, keep the launch order (in which all heads of a
// sequence share one XCD: what a rotary key shared by the heads wants).
__device__ __forceinline__ void xcd_head_order(int& x, int& y, bool on) {
  const int gy = gridDim.y;
  if (!on || gy % 8) {
    x = blockIdx.x;
    y = blockIdx.y;
    return;
  }
  const int i = blockIdx.x + gridDim.x * blockIdx.y;
  const int j = i >> 3, hp = gy >> 3;
  y = (i & 7) + 8 * (j % hp);
  x = j / hp;
}

// ---- cross-lane ----------------------------------------------------------

__device__ __forceinline__ float xor_shfl(float v, int mask) { return __shfl_xor(v, mask, kWave); }

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// Cache slot of token position pos under a sink + window eviction budget (the
// window part is a ring after the sink slots); window 0 means no eviction.
__device__ __forceinline__ int ring_slot(int pos, int sink, int window) {
  return (window == 0 || pos < sink) ? pos : sink + (pos - sink) % window;
}

}  // namespace lla
