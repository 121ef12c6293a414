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

// One thread per (b, m, pair i) and chunk of CH heads (grid dimension y): the
// angle is shared by the heads of the row, so cos and sin are formed once per
// chunk.  A chunk's loads are all issued before any of its stores: the output
// may alias the input, so a load after a store would wait for it.  Large calls
// (prefill) take chunks of 8 heads, so the inverse-frequency table is built by
// few workgroups; small ones (a decode step's queries) one head per thread, so
// the call has enough threads.
// Write: row (b, m, g) of x [B][M][G][dr] is rotated at position pos0 + m and
// lands in that position's slot of the paged cache of (b, g).
template <typename T, int CH>
__global__ __launch_bounds__(256) void rope_write_kernel(RopeArgs a) {
  __shared__ double s_inv[LLA_MAX_ROPE / 2];
  inv_freq_table(s_inv, a.dr, a.base);
  const int half = a.dr / 2;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)a.B * a.M * half) return;
  const size_t bm = idx / half;
  const int i = (int)(idx - bm * half);
  const int m = (int)(bm % a.M), b = (int)(bm / a.M);
  const int pos = a.pos0 + m;
  const int slot = ring_slot(pos, a.sink, a.window);  // rotated at its true position, stored at its slot
  float c, s;
  rope_cs(pos, s_inv[i], c, s);
  T* y = static_cast<T*>(a.y);
  const int g0 = blockIdx.y * CH;
  float x1[CH], x2[CH];
#pragma unroll
  for (int u = 0; u < CH; ++u) {
    const size_t row = bm * a.G + min(g0 + u, a.G - 1);
    x1[u] = load_elem<T>(a.x, row * a.dr + i);
    x2[u] = load_elem<T>(a.x, row * a.dr + i + half);
  }
#pragma unroll
  for (int u = 0; u < CH; ++u) {
    const int g = g0 + u;
    if (g < a.G) {
      const size_t page = ((size_t)(b * a.G + g) * a.n_max + (size_t)(slot / kPage) * kPage) * a.dr;
      store_out(y, page + (size_t)i * kPage + slot % kPage, x1[u] * c - x2[u] * s);
      store_out(y, page + (size_t)(i + half) * kPage + slot % kPage, x2[u] * c + x1[u] * s);
    }
  }
}

// Rotate: row (b, g, m) of x [B][G][M][dr] at position (pos ? pos[b] : pos0) + m.
template <typename T, int CH>
__global__ __launch_bounds__(256) void rope_rotate_kernel(RopeArgs a) {
  __shared__ double s_inv[LLA_MAX_ROPE / 2];
  inv_freq_table(s_inv, a.dr, a.base);
  const int half = a.dr / 2;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)a.B * a.M * half) return;
  const size_t bm = idx / half;
  const int i = (int)(idx - bm * half);
  const int m = (int)(bm % a.M), b = (int)(bm / a.M);
  const int pos = (a.pos ? a.pos[b] : a.pos0) + m;
  float c, s;
  rope_cs(pos, s_inv[i], c, s);
  T* y = static_cast<T*>(a.y);
  const int g0 = blockIdx.y * CH;
  float x1[CH], x2[CH];
#pragma unroll
  for (int u = 0; u < CH; ++u) {
    const size_t row = ((size_t)b * a.G + min(g0 + u, a.G - 1)) * a.M + m;
    x1[u] = load_elem<T>(a.x, row * a.dr + i);
    x2[u] = load_elem<T>(a.x, row * a.dr + i + half);
  }
#pragma unroll
  for (int u = 0; u < CH; ++u) {
    if (g0 + u < a.G) {
      const size_t row = ((size_t)b * a.G + g0 + u) * a.M + m;
      store_out(y, row * a.dr + i, x1[u] * c - x2[u] * s);
      store_out(y, row * a.dr + i + half, x2[u] * c + x1[u] * s);
    }
  }
}

constexpr size_t kChunkedFrom = 65536;  // (b, m, pair) threads from which heads go 8 per thread
dim3 grid_for(const RopeArgs& a, int ch) {
  const size_t n = (size_t)a.B * a.M * (a.dr / 2);
  return dim3((unsigned)((n + 255) / 256), (unsigned)((a.G + ch - 1) / ch));
}


}  // namespace

hipError_t launch_rope_write(const RopeArgs& a, hipStream_t stream) {
  const bool chunked = (size_t)a.B * a.M * (a.dr / 2) >= kChunkedFrom;
  const int ch = chunked ? 8 : 1;
  if (a.dtype == LLA_BF16) {
    if (chunked) hipLaunchKernelGGL((rope_write_kernel<bf16_t, 8>), grid_for(a, ch), dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((rope_write_kernel<bf16_t, 1>), grid_for(a, ch), dim3(256), 0, stream, a);
  } else {
    if (chunked) hipLaunchKernelGGL((rope_write_kernel<float, 8>), grid_for(a, ch), dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((rope_write_kernel<float, 1>), grid_for(a, ch), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_rope_rotate(const RopeArgs& a, hipStream_t stream) {
  const bool chunked = (size_t)a.B * a.M * (a.dr / 2) >= kChunkedFrom;
  const int ch = chunked ? 8 : 1;
  if (a.dtype == LLA_BF16) {
    if (chunked) hipLaunchKernelGGL((rope_rotate_kernel<bf16_t, 8>), grid_for(a, ch), dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((rope_rotate_kernel<bf16_t, 1>), grid_for(a, ch), dim3(256), 0, stream, a);
  } else {
    if (chunked) hipLaunchKernelGGL((rope_rotate_kernel<float, 8>), grid_for(a, ch), dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((rope_rotate_kernel<float, 1>), grid_for(a, ch), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace lla
