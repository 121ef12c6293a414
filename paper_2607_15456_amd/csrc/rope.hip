// Rotary embedding of the decoupled rotary branch (App. J "Absorbed
// attention": a NoPE content path plus a small explicit rotary branch, shared
// across loops for each token).  Half-split convention: feature i pairs with
// feature i + dr/2 and turns by the angle p * base^(-2i/dr).
//
// Keys are rotated once, when their token is written (the branch is shared by
// the loops, so there is one write per token); queries are rotated by the
// caller through lla_rope_rotate before the attention call.  The angle is
// formed and reduced to [-pi, pi] in double precision (positions reach 2^24
// and beyond) and its sine and cosine taken in fp32, about 1e-7 absolute.

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {

template <typename T>
__device__ __forceinline__ float load_elem(const void* p, size_t i) {
  return Elem<T>::get(static_cast<const T*>(p), i);
}

// The dr/2 inverse frequencies base^(-2i/dr), once per workgroup (double).
__device__ __forceinline__ void inv_freq_table(double* t, int dr, double base) {
  for (int i = threadIdx.x; i < dr / 2; i += blockDim.x) t[i] = pow(base, -2.0 * i / dr);
  __syncthreads();
}

// (cos, sin) of p * inv_freq: the angle is formed and reduced to [-pi, pi] in
// double (positions reach 2^24 and beyond), then evaluated in fp32.
__device__ __forceinline__ void rope_cs(int p, double inv_freq, float& c, float& s) {
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  const double ang = (double)p * inv_freq;
  const double r = ang - rint(ang * (1.0 / kTwoPi)) * kTwoPi;
  sincosf((float)r, &s, &c);
}

// One thread per (row, pair i): every head's row is its own thread, so the
// loads of a call are all in flight at once (a loop over the heads would wait
// on each head's load in turn, since the output may alias the input); the
// angle is recomputed per head, bit for bit the same.
// Write: row (b, m, g) of x [B][M][G][dr] is rotated at position pos0 + m and
// lands in that position's slot of the paged cache of (b, g).
template <typename T>
__global__ __launch_bounds__(256) void rope_write_kernel(RopeArgs a) {
  __shared__ double s_inv[LLA_MAX_ROPE / 2];
  inv_freq_table(s_inv, a.dr, a.base);
  const int half = a.dr / 2;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)a.B * a.M * a.G * half) return;
  const size_t row = idx / half;  // (b, m, g)
  const int i = (int)(idx - row * half);
  const int g = (int)(row % a.G);
  const size_t bm = row / a.G;
  const int m = (int)(bm % a.M), b = (int)(bm / a.M);
  const int pos = a.pos0 + m;
  const int slot = ring_slot(pos, a.sink, a.window);  // rotated at its true position, stored at its slot
  float c, s;
  rope_cs(pos, s_inv[i], c, s);
  const float x1 = load_elem<T>(a.x, row * a.dr + i), x2 = load_elem<T>(a.x, row * a.dr + i + half);
  T* y = static_cast<T*>(a.y);
  const size_t page = ((size_t)(b * a.G + g) * a.n_max + (size_t)(slot / kPage) * kPage) * a.dr;
  store_out(y, page + (size_t)i * kPage + slot % kPage, x1 * c - x2 * s);
  store_out(y, page + (size_t)(i + half) * kPage + slot % kPage, x2 * c + x1 * s);
}

// Rotate: row (b, g, m) of x [B][G][M][dr] at position (pos ? pos[b] : pos0) + m.
template <typename T>
__global__ __launch_bounds__(256) void rope_rotate_kernel(RopeArgs a) {
  __shared__ double s_inv[LLA_MAX_ROPE / 2];
  inv_freq_table(s_inv, a.dr, a.base);
  const int half = a.dr / 2;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)a.B * a.G * a.M * half) return;
  const size_t row = idx / half;  // (b, g, m)
  const int i = (int)(idx - row * half);
  const int m = (int)(row % a.M), b = (int)(row / ((size_t)a.G * a.M));
  const int pos = (a.pos ? a.pos[b] : a.pos0) + m;
  float c, s;
  rope_cs(pos, s_inv[i], c, s);
  const float x1 = load_elem<T>(a.x, row * a.dr + i), x2 = load_elem<T>(a.x, row * a.dr + i + half);
  T* y = static_cast<T*>(a.y);
  store_out(y, row * a.dr + i, x1 * c - x2 * s);
  store_out(y, row * a.dr + i + half, x2 * c + x1 * s);
}

dim3 grid_for(const RopeArgs& a) {
  const size_t n = (size_t)a.B * a.M * a.G * (a.dr / 2);
  return dim3((unsigned)((n + 255) / 256));
}

}  // namespace

hipError_t launch_rope_write(const RopeArgs& a, hipStream_t stream) {
  if (a.dtype == LLA_BF16)
    hipLaunchKernelGGL(rope_write_kernel<bf16_t>, grid_for(a), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(rope_write_kernel<float>, grid_for(a), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_rope_rotate(const RopeArgs& a, hipStream_t stream) {
  if (a.dtype == LLA_BF16)
    hipLaunchKernelGGL(rope_rotate_kernel<bf16_t>, grid_for(a), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(rope_rotate_kernel<float>, grid_for(a), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace lla
