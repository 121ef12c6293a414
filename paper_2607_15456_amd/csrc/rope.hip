// Rotary embedding of the decoupled rotary branch (App. J "Absorbed
// attention": a NoPE content path plus a small explicit rotary branch, shared
// across loops for each token).  Half-split convention: feature i pairs with
// feature i + dr/2 and turns by the angle p * base^(-2i/dr).
//
// Keys are rotated once, when their token is written (the branch is shared by
// the loops, so there is one write per token); queries are rotated by the
// caller through lla_rope_rotate before the attention call.  The angle is
// formed and reduced in double precision (positions reach 2^24 and beyond), so
// the only rounding that matters is the final one to the storage type.

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {

template <typename T>
__device__ __forceinline__ float load_elem(const void* p, size_t i) {
  return Elem<T>::get(static_cast<const T*>(p), i);
}

// (cos, sin) of p * base^(-2i/dr)
__device__ __forceinline__ void rope_cs(int p, int i, int dr, double base, float& c, float& s) {
  const double ang = (double)p * pow(base, -2.0 * i / dr);
  double sd, cd;
  sincos(ang, &sd, &cd);
  c = (float)cd;
  s = (float)sd;
}

// One thread per (row, pair).  Write: row (b, m, g) of x [B][M][G][dr] lands at
// position pos0 + m of the paged cache of (b, g).
template <typename T>
__global__ __launch_bounds__(256) void rope_write_kernel(RopeArgs a) {
  const int half = a.dr / 2;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t rows = (size_t)a.B * a.M * a.G;
  if (idx >= rows * half) return;
  const size_t row = idx / half;
  const int i = (int)(idx - row * half);
  const int g = (int)(row % a.G);
  const size_t bm = row / a.G;
  const int m = (int)(bm % a.M), b = (int)(bm / a.M);
  const int pos = a.pos0 + m;
  float c, s;
  rope_cs(pos, i, a.dr, a.base, c, s);
  const float x1 = load_elem<T>(a.x, row * a.dr + i), x2 = load_elem<T>(a.x, row * a.dr + i + half);
  const size_t page = ((size_t)(b * a.G + g) * a.n_max + (size_t)(pos / kPage) * kPage) * a.dr;
  T* y = static_cast<T*>(a.y);
  store_out(y, page + (size_t)i * kPage + pos % kPage, x1 * c - x2 * s);
  store_out(y, page + (size_t)(i + half) * kPage + pos % kPage, x2 * c + x1 * s);
}

// Rotate: row (b, g, m) of x [B][G][M][dr] at position (pos ? pos[b] : pos0) + m.
template <typename T>
__global__ __launch_bounds__(256) void rope_rotate_kernel(RopeArgs a) {
  const int half = a.dr / 2;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t rows = (size_t)a.B * a.G * a.M;
  if (idx >= rows * half) return;
  const size_t row = idx / half;
  const int i = (int)(idx - row * half);
  const int m = (int)(row % a.M);
  const int b = (int)(row / ((size_t)a.G * a.M));
  const int pos = (a.pos ? a.pos[b] : a.pos0) + m;
  float c, s;
  rope_cs(pos, i, a.dr, a.base, c, s);
  const float x1 = load_elem<T>(a.x, row * a.dr + i), x2 = load_elem<T>(a.x, row * a.dr + i + half);
  T* y = static_cast<T*>(a.y);
  store_out(y, row * a.dr + i, x1 * c - x2 * s);
  store_out(y, row * a.dr + i + half, x2 * c + x1 * s);
}

dim3 grid_for(const RopeArgs& a) {
  const size_t n = (size_t)a.B * a.G * a.M * (a.dr / 2);
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
