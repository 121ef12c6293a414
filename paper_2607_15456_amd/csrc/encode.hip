// Encode / cache write (Sec. 3, Eq. 2): c = (x - mu) W_down for the M new
// tokens of every sequence, both axes, written into the paged latent cache.
//
// bf16: a dense contraction on MFMA.  Per (axis, head) the output is the
// r x (B*M) matrix C^T = W_down^T X^T - (W_down^T mu) 1^T, computed with
// v_mfma_f32_32x32x16_bf16 on 32-row x 32-token tiles:
//   A operand  = 32 rows of W_down^T (row-major [r][T*d], 8 contiguous k per lane),
//   B operand  = 32 tokens of x      (each token's T*d stack is contiguous),
//   accumulator column = one token, so the 32x32 fp32 tile maps straight onto
//   the feature-major cache page (one feature row of consecutive tokens).
// The mean is a second accumulator fed with mu as a broadcast B operand, so
// (x - mu) W_down is formed in fp32 without re-rounding x - mu to bf16.
// The pass reads x once (HBM-bound at the paper's ranks: about (r_k + r_v)/2
// flop per byte).
//
// fp32: a plain LDS-tiled VALU GEMM with the same output mapping.

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

constexpr int kEncWaves = 4;

// Cache index of (b, h, position pos, feature row) in the paged layout.
__device__ __forceinline__ size_t cache_index(int b, int h, int H, int n_max, int r, int pos,
                                              int row) {
  return ((size_t)(b * H + h) * n_max + (size_t)(pos / kPage) * kPage) * r + (size_t)row * kPage +
         (pos % kPage);
}

// grid: x = token-group blocks, y = row-tile blocks, z = axis * H + h
// wr = waves of a workgroup laid along rows (1, 2 or 4); the rest along tokens.
__global__ __launch_bounds__(kEncWaves * kWave) void encode_bf16_kernel(EncodeArgs a, int wr) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int axis = blockIdx.z / a.H, h = blockIdx.z - axis * a.H;
  const int r = a.r[axis], K = a.K;
  const int tg = blockIdx.x * (kEncWaves / wr) + wave / wr;
  const int rt = blockIdx.y * wr + wave % wr;
  const int TT = a.B * a.M;
  if (tg * 32 >= TT || rt * 32 >= r) return;

  const int col = lane & 31, half = lane >> 5;
  const int row_a = rt * 32 + col;  // A operand row (feature)
  const int tok_b = tg * 32 + col;  // B operand column (token)
  const bool row_ok = row_a < r, tok_ok = tok_b < TT;

  const bf16_t* w = static_cast<const bf16_t*>(a.wdt[axis]) + ((size_t)h * r + (row_ok ? row_a : 0)) * K;
  const bf16_t* x = static_cast<const bf16_t*>(a.x[axis]) + ((size_t)(tok_ok ? tok_b : 0) * a.H + h) * K;
  const bf16_t* mu = a.mu[axis] ? static_cast<const bf16_t*>(a.mu[axis]) + (size_t)h * K : nullptr;

  f32x16 acc = {0.f}, accm = {0.f};
  const uint4 zero = make_uint4(0, 0, 0, 0);
#pragma unroll 8
  for (int k0 = 0; k0 < K; k0 += 16) {
    const int k = k0 + half * 8;
    const uint4 av = row_ok ? ld16(w + k) : zero;
    const uint4 bv = tok_ok ? ld16(x + k) : zero;
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(av), as_bf16x8(bv), acc, 0, 0, 0);
    if (mu) {
      const uint4 mv = ld16(mu + k);
      accm = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(av), as_bf16x8(mv), accm, 0, 0, 0);
    }
  }
  if (!tok_ok) return;
  const int b = tok_b / a.M, pos = a.pos0 + (tok_b - b * a.M);
  bf16_t* c = static_cast<bf16_t*>(a.c[axis]);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int row = rt * 32 + 8 * (i / 4) + 4 * half + (i % 4);
    if (row < r) c[cache_index(b, h, a.H, a.n_max, r, pos, row)] = f32_to_bf16(acc[i] - accm[i]);
  }
}

// fp32: 16 tokens x 16 rows per workgroup, K staged through LDS in chunks of 64.
constexpr int kT = 16, kKC = 64;
__global__ __launch_bounds__(256) void encode_f32_kernel(EncodeArgs a) {
  __shared__ float s_x[kT][kKC + 1];
  __shared__ float s_w[kT][kKC + 1];
  const int axis = blockIdx.z / a.H, h = blockIdx.z - axis * a.H;
  const int r = a.r[axis], K = a.K, TT = a.B * a.M;
  if (blockIdx.y * kT >= r) return;
  const int tt = threadIdx.x / kT, rr = threadIdx.x % kT;
  const int tok = blockIdx.x * kT + tt, row = blockIdx.y * kT + rr;
  const float* x = static_cast<const float*>(a.x[axis]);
  const float* w = static_cast<const float*>(a.wdt[axis]) + (size_t)h * r * K;
  const float* mu = a.mu[axis] ? static_cast<const float*>(a.mu[axis]) + (size_t)h * K : nullptr;
  float acc = 0.f;
  for (int k0 = 0; k0 < K; k0 += kKC) {
    for (int e = threadIdx.x; e < kT * kKC; e += 256) {
      const int i = e / kKC, kk = e % kKC, k = k0 + kk;
      const int t = blockIdx.x * kT + i, ro = blockIdx.y * kT + i;
      float xv = 0.f;
      if (t < TT && k < K) xv = x[((size_t)t * a.H + h) * K + k] - (mu ? mu[k] : 0.f);
      s_x[i][kk] = xv;
      s_w[i][kk] = (ro < r && k < K) ? w[(size_t)ro * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < kKC; ++kk) acc = fmaf(s_x[tt][kk], s_w[rr][kk], acc);
    __syncthreads();
  }
  if (tok < TT && row < r) {
    const int b = tok / a.M, pos = a.pos0 + (tok - b * a.M);
    static_cast<float*>(a.c[axis])[cache_index(b, h, a.H, a.n_max, r, pos, row)] = acc;
  }
}

}  // namespace

hipError_t launch_encode(const EncodeArgs& a, hipStream_t stream) {
  const int TT = a.B * a.M;
  const int rmax = a.r[0] > a.r[1] ? a.r[0] : a.r[1];
  if (a.dtype == LLA_BF16) {
    const int tiles = (rmax + 31) / 32, groups = (TT + 31) / 32;
    const int wr = tiles >= 4 ? 4 : tiles >= 2 ? 2 : 1;
    dim3 grid((groups + kEncWaves / wr - 1) / (kEncWaves / wr), (tiles + wr - 1) / wr, 2 * a.H);
    hipLaunchKernelGGL(encode_bf16_kernel, grid, dim3(kEncWaves * kWave), 0, stream, a, wr);
  } else {
    dim3 grid((TT + kT - 1) / kT, (rmax + kT - 1) / kT, 2 * a.H);
    hipLaunchKernelGGL(encode_f32_kernel, grid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace lla
