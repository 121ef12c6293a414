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

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Per-axis fields selected without dynamic indexing (which would spill the
// argument struct to scratch).
template <typename T>
__device__ __forceinline__ T pick(const T (&v)[2], int axis) {
  const T v0 = v[0], v1 = v[1];  // values, so the select is not between two addresses
  return axis ? v1 : v0;
}

// Cache index of (b, h, slot pos, feature row): the paged feature-major layout,
// or (tm, the LLA-2D key cache) token-major rows of r features.
__device__ __forceinline__ size_t cache_index(int b, int h, int H, int n_max, int r, int pos,
                                              int row, bool tm = false) {
  if (tm) return ((size_t)(b * H + h) * n_max + pos) * r + row;
  return ((size_t)(b * H + h) * n_max + (size_t)(pos / kPage) * kPage) * r + (size_t)row * kPage +
         (pos % kPage);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kEncTok = 32;           // tokens per workgroup block
constexpr int kEncKC = 512;           // K elements staged per step
constexpr int kEncXS = kEncKC + 8;    // LDS row stride (elements): 1040 B, staggers banks
constexpr int kEncMaxTasks = 4;       // 16x16 output tiles per wavefront

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// One workgroup: 32 consecutive tokens (b, m flattened) x heads [h0, h1) x
// 16-row output tiles [rt0, rt1) of one axis.  x is streamed through
// double-buffered LDS one (head, 512-element K chunk) stage at a time: each
// wave-wide load reads one token's contiguous 1 KB, and the next stage's loads
// are in flight while the current stage is multiplied.  Each wavefront owns up
// to 4 (row tile, token tile) 16x16 accumulators (v_mfma_f32_16x16x32_bf16:
// A = 16 rows of W_down^T from L2, B = 16 tokens from LDS); a head's tiles
// are written to the feature-major cache pages after its last K chunk.
// grid: x = token blocks, y = head chunks, z = axis * nrc + row chunk
__global__ __launch_bounds__(256) void encode_bf16_kernel(EncodeArgs a, int heads_per_wg, int rt_per_wg,
                                                          int nrc) {
  __shared__ __attribute__((aligned(16))) bf16_t s_x[2][kEncTok * kEncXS];
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int axis = blockIdx.z / nrc, rc = blockIdx.z - axis * nrc;
  const int r = pick(a.r, axis), K = a.K, H = a.H;
  const int RT = (r + 15) / 16;
  const int rt0 = rc * rt_per_wg;
  if (rt0 >= RT) return;  // uniform over the workgroup
  const int rt1 = min(RT, rt0 + rt_per_wg);
  const int ntask = (rt1 - rt0) * 2;  // x 2 token tiles of 16
  const int h0 = blockIdx.y * heads_per_wg, h1 = min(H, h0 + heads_per_wg);
  const int TT = a.B * a.M;
  const int t0 = blockIdx.x * kEncTok;
  const int nkc = (K + kEncKC - 1) / kEncKC;
  const int nstage = (h1 - h0) * nkc;
  const bf16_t* xg = static_cast<const bf16_t*>(pick(a.x, axis));
  const bf16_t* wg = static_cast<const bf16_t*>(pick(a.wdt, axis));
  const bf16_t* mug = static_cast<const bf16_t*>(pick(a.mu, axis));

  uint4 rgs[8];
  auto stage_load = [&](int st) {
    const int h = h0 + st / nkc, k0 = (st % nkc) * kEncKC;
    const int cpt = min(kEncKC, K - k0) / 8;  // 16-byte chunks per token
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int c = tid + i * 256;
      if (c < kEncTok * cpt) {
        const int tok = c / cpt, part = c - tok * cpt, t = t0 + tok;
        // tokens past the last one re-read it: their output columns are never stored
        rgs[i] = ld16(xg + ((size_t)min(t, TT - 1) * H + h) * K + k0 + part * 8);
      }
    }
  };
  auto stage_store = [&](int st, int buf) {
    const int k0 = (st % nkc) * kEncKC;
    const int cpt = min(kEncKC, K - k0) / 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int c = tid + i * 256;
      if (c < kEncTok * cpt) {
        const int tok = c / cpt, part = c - tok * cpt;
        *reinterpret_cast<uint4*>(&s_x[buf][tok * kEncXS + part * 8]) = rgs[i];
      }
    }
  };

  f32x4 acc[kEncMaxTasks], accm[kEncMaxTasks];
#pragma unroll
  for (int u = 0; u < kEncMaxTasks; ++u) acc[u] = accm[u] = f32x4{0.f};
  const int li = lane & 15, lg = lane >> 4;

  stage_load(0);
  stage_store(0, 0);
  __syncthreads();
  for (int st = 0; st < nstage; ++st) {
    const int buf = st & 1;
    if (st + 1 < nstage) stage_load(st + 1);
    const int h = h0 + st / nkc, kc = st % nkc, k0 = kc * kEncKC;
    const int ks = min(kEncKC, K - k0) / 32;  // K-steps of 32 in this chunk
#pragma unroll
    for (int u = 0; u < kEncMaxTasks; ++u) {
      const int task = wave + 4 * u;
      if (task < ntask) {
        const int rt = rt0 + task / 2, tt = task % 2;
        const int row = rt * 16 + li;
        const bool row_ok = row < r;
        const bf16_t* wrow = wg + ((size_t)h * r + (row_ok ? row : 0)) * K + k0 + 8 * lg;
        const bf16_t* xrow = &s_x[buf][(tt * 16 + li) * kEncXS + 8 * lg];
        const bf16_t* mrow = mug ? mug + (size_t)h * K + k0 + 8 * lg : nullptr;
        // eight K-steps of W_down^T fragments in flight at once (with few
        // tokens the weights are the whole traffic, and a load per step
        // would expose the load latency sixteen times per chunk)
        for (int s0 = 0; s0 < ks; s0 += 8) {
          bf16x8 av[8];
#pragma unroll
          for (int j = 0; j < 8; ++j)
            av[j] = as_bf16x8(row_ok && s0 + j < ks ? ld16(wrow + 32 * (s0 + j)) : make_uint4(0, 0, 0, 0));
          if (s0 + 8 <= ks) {
            // a whole group: no guard per product (a guard there makes each
            // MFMA a block of its own, waiting on its own operand reads)
            if (mrow) {
              uint4 mv[8];
#pragma unroll
              for (int j = 0; j < 8; ++j) mv[j] = ld16(mrow + 32 * (s0 + j));
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                const bf16x8 bv = as_bf16x8(*reinterpret_cast<const uint4*>(xrow + 32 * (s0 + j)));
                acc[u] = mfma16(av[j], bv, acc[u]);
                accm[u] = mfma16(av[j], as_bf16x8(mv[j]), accm[u]);
              }
            } else {
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                const bf16x8 bv = as_bf16x8(*reinterpret_cast<const uint4*>(xrow + 32 * (s0 + j)));
                acc[u] = mfma16(av[j], bv, acc[u]);
              }
            }
          } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              if (s0 + j < ks) {
                const bf16x8 bv = as_bf16x8(*reinterpret_cast<const uint4*>(xrow + 32 * (s0 + j)));
                acc[u] = mfma16(av[j], bv, acc[u]);
                if (mrow) accm[u] = mfma16(av[j], as_bf16x8(ld16(mrow + 32 * (s0 + j))), accm[u]);
              }
            }
          }
        }
        if (kc == nkc - 1) {  // head done: write its tile, c = x W - mu W
          const int t = t0 + tt * 16 + li;
          if (t < TT) {
            const int b = t / a.M, pos = ring_slot(a.pos0 + (t - b * a.M), a.sink, a.window);
            bf16_t* c = static_cast<bf16_t*>(pick(a.c, axis));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int rr = rt * 16 + 4 * lg + e;
              if (rr < r) c[cache_index(b, h, H, a.n_max, r, pos, rr, axis == 0 && a.k_token_major)] = f32_to_bf16(acc[u][e] - accm[u][e]);
            }
          }
          acc[u] = accm[u] = f32x4{0.f};
        }
      }
    }
    if (st + 1 < nstage) stage_store(st + 1, buf ^ 1);
    __syncthreads();
  }
}

// Many new tokens at small ranks (a prefill's cache write, r <= 64, T*d = KS*32):
// the weights stay in registers and the tokens stream past them.  Grid:
// x = token ranges, y = head, z = axis.  Wavefront w owns 16-row tile rt of
// the head's W_down^T (its A fragments for the whole T*d held in KS registers
// of 16 bytes) and one or two 16-token tiles of every 32-token block; blocks
// of x are staged through double-buffered LDS with coalesced 1 KB loads.  The
// mean term W_down^T mu is one extra product per workgroup at the start.
template <int KS>
__global__ __launch_bounds__(256) void encode_stream_kernel(EncodeArgs a, int blocks_per_wg) {
  constexpr int K = KS * 32;
  constexpr int XS = K + 8;
  __shared__ __attribute__((aligned(16))) bf16_t s_x[2][kEncTok * XS];
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int axis = blockIdx.z, h = blockIdx.y, H = a.H;
  const int r = pick(a.r, axis);
  const int RT = r > 32 ? 4 : 2;           // 16-row tiles (rows >= r are zero)
  const int rt = wave % RT;
  const int ntt = RT == 4 ? 2 : 1;         // token tiles per wavefront
  const int tt0 = RT == 4 ? 0 : wave / 2;
  const int TT = a.B * a.M;
  const int nblk = (TT + kEncTok - 1) / kEncTok;
  const int b0 = blockIdx.x * blocks_per_wg, b1 = min(nblk, b0 + blocks_per_wg);
  if (b0 >= b1) return;
  const int li = lane & 15, lg = lane >> 4;
  const int row = rt * 16 + li;
  const bool row_ok = row < r;

  // resident A fragments of W_down^T rows [16 rt, 16 rt + 16)
  const bf16_t* wrow = static_cast<const bf16_t*>(pick(a.wdt, axis)) + ((size_t)h * r + (row_ok ? row : 0)) * K + 8 * lg;
  bf16x8 wf[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) wf[s] = as_bf16x8(row_ok ? ld16(wrow + 32 * s) : make_uint4(0, 0, 0, 0));
  f32x4 bmu = f32x4{0.f};
  if (pick(a.mu, axis)) {
    const bf16_t* mrow = static_cast<const bf16_t*>(pick(a.mu, axis)) + (size_t)h * K + 8 * lg;
#pragma unroll
    for (int s = 0; s < KS; ++s) bmu = mfma16(wf[s], as_bf16x8(ld16(mrow + 32 * s)), bmu);
  }

  const bf16_t* xg = static_cast<const bf16_t*>(pick(a.x, axis));
  constexpr int CPT = K / 8;                               // 16-byte chunks per token
  constexpr int NCH = (kEncTok * CPT + 255) / 256;         // chunks per thread per block
  uint4 rgs[NCH];
  auto load_blk = [&](int blk) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + i * 256;
      if (c < kEncTok * CPT) {
        const int tok = c / CPT, part = c - tok * CPT, t = blk * kEncTok + tok;
        // tokens past the last one re-read it: their output columns are never stored;
        // x is read once (non-temporal: 210 -> 192 us on the 4 x 8192-token write)
        rgs[i] = ld16_nt(xg + ((size_t)min(t, TT - 1) * H + h) * K + part * 8);
      }
    }
  };
  auto store_blk = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + i * 256;
      if (c < kEncTok * CPT) {
        const int tok = c / CPT, part = c - tok * CPT;
        *reinterpret_cast<uint4*>(&s_x[buf][tok * XS + part * 8]) = rgs[i];
      }
    }
  };

  bf16_t* cout = static_cast<bf16_t*>(pick(a.c, axis));
  load_blk(b0);
  store_blk(0);
  __syncthreads();
  for (int blk = b0; blk < b1; ++blk) {
    const int buf = (blk - b0) & 1;
    if (blk + 1 < b1) load_blk(blk + 1);
    for (int u = 0; u < ntt; ++u) {
      const int tt = tt0 + u;
      const bf16_t* xrow = &s_x[buf][(tt * 16 + li) * XS + 8 * lg];
      f32x4 acc = f32x4{0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s)
        acc = mfma16(wf[s], as_bf16x8(*reinterpret_cast<const uint4*>(xrow + 32 * s)), acc);
      const int t = blk * kEncTok + tt * 16 + li;
      if (t < TT) {
        const int b = t / a.M, pos = ring_slot(a.pos0 + (t - b * a.M), a.sink, a.window);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rr = rt * 16 + 4 * lg + e;
          if (rr < r) cout[cache_index(b, h, H, a.n_max, r, pos, rr, axis == 0 && a.k_token_major)] = f32_to_bf16(acc[e] - bmu[e]);
        }
      }
    }
    if (blk + 1 < b1) store_blk(buf ^ 1);
    __syncthreads();
  }
}

// Few new tokens (a decode step writes one per sequence): the weights are the
// whole traffic, so every W_down^T element is read once and nothing waits on
// more than one round of loads.  Workgroup = 32 rows of one (axis, head) x 32
// tokens; wavefront w computes the 16x16 tile (row tile w % 2, token tile
// w / 2) with both operands loaded straight from global memory, sixteen
// K-steps of A and B fragments in flight at once (no LDS, no barrier).
// With a long K (the LLA-2D stack) the K-steps are split over ksplit
// workgroups per tile so the weights spread over the whole machine; each
// writes its fp32 partial tile and encode_reduce_kernel (the next launch)
// adds them and writes the cache.
// grid: x = 32-token blocks, y = 32-row chunks of axis k then axis v,
// z = head * ksplit + K-split
__global__ __launch_bounds__(256) void encode_few_kernel(EncodeArgs a, int nrc_k) {
  constexpr int CH = 16;  // K-steps per round of loads
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int axis = blockIdx.y >= (unsigned)nrc_k ? 1 : 0;
  const int rc = blockIdx.y - axis * nrc_k;
  const int split = blockIdx.z % a.ksplit, h = blockIdx.z / a.ksplit, H = a.H, K = a.K;
  const int r = pick(a.r, axis);
  const int li = lane & 15, lg = lane >> 4;
  const int row = rc * 32 + (wave & 1) * 16 + li;
  const int TT = a.B * a.M;
  const int tcol = blockIdx.x * 32 + (wave >> 1) * 16 + li;  // token of this lane's B column
  const bool row_ok = row < r, tok_ok = tcol < TT;
  const bf16_t* wrow = static_cast<const bf16_t*>(pick(a.wdt, axis)) + ((size_t)h * r + (row_ok ? row : 0)) * K + 8 * lg;
  const bf16_t* xrow = static_cast<const bf16_t*>(pick(a.x, axis)) + ((size_t)(tok_ok ? tcol : 0) * H + h) * K + 8 * lg;
  const bf16_t* mrow = pick(a.mu, axis) ? static_cast<const bf16_t*>(pick(a.mu, axis)) + (size_t)h * K + 8 * lg : nullptr;
  const uint4 zero = make_uint4(0, 0, 0, 0);
  const int per = (K / 32 + a.ksplit - 1) / a.ksplit;  // K-steps of this split: [sb, se)
  const int sb = split * per, se = min(K / 32, sb + per);
  f32x4 acc = f32x4{0.f}, accm = f32x4{0.f};
  for (int s0 = sb; s0 < se; s0 += CH) {
    bf16x8 wf[CH], xf[CH], mf[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const bool in = s0 + j < se;
      wf[j] = as_bf16x8(row_ok && in ? ld16(wrow + 32 * (s0 + j)) : zero);
      xf[j] = as_bf16x8(tok_ok && in ? ld16(xrow + 32 * (s0 + j)) : zero);
      mf[j] = as_bf16x8(mrow && in ? ld16(mrow + 32 * (s0 + j)) : zero);
    }
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      acc = mfma16(wf[j], xf[j], acc);
      if (mrow) accm = mfma16(wf[j], mf[j], accm);
    }
  }
  acc -= accm;
  if (a.ksplit > 1) {  // partial tile; encode_reduce_kernel adds the splits
    const size_t unit = ((size_t)h * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
    *reinterpret_cast<f32x4*>(a.part + (unit * a.ksplit + split) * 1024 + tid * 4) = acc;
    return;
  }
  // output tile: lane (li, lg) holds rows 4 lg .. 4 lg + 3 of token column li
  const int t = blockIdx.x * 32 + (wave >> 1) * 16 + li;
  if (t < TT) {
    const int b = t / a.M, pos = ring_slot(a.pos0 + (t - b * a.M), a.sink, a.window);
    bf16_t* c = static_cast<bf16_t*>(pick(a.c, axis));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int rr = rc * 32 + (wave & 1) * 16 + 4 * lg + e;
      if (rr < r) c[cache_index(b, h, H, a.n_max, r, pos, rr, axis == 0 && a.k_token_major)] = f32_to_bf16(acc[e]);
    }
  }
}

// Prefill-sized writes over a long stack (the LLA-2D down-projection, K =
// T*H*d = 8192 values into r = 288 / 480): 2 r flops per byte of x, a
// compute-bound GEMM.  A workgroup of 8 wavefronts takes 256 tokens x 96 rows
// of one axis; both operands are staged through double-buffered LDS in K-chunks
// of 64 (two further chunks in flight in registers), and wavefront w computes
// tokens 32w .. 32w + 31 x all 96 rows on v_mfma_f32_32x32x16_bf16:
//   keys   (token-major cache): D = C^T (M = row, N = token), a lane holds
//          4-row runs of one token;
//   values (feature-major pages): D = C (M = token, N = row).
// The row blocks of one token block are dispatched back to back on one XCD
// (workgroup i runs on XCD i % 8), so its x chunks come from that XCD's L2
// after the first read.  With a mean, wavefronts 0 .. 2 also form W_down^T mu
// for one 32-row tile each (mu as a broadcast operand), shared through LDS.
constexpr int kGTok = 256, kGRow = 96, kGKC = 64, kGS = kGKC + 8;
constexpr int kGTS = kGTok + 8;  // row stride (bf16) of the epilogue's output tile in LDS
constexpr int kGThreads = 512;

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// AXIS: 0 keys, 1 values.  TM: the output cache is token-major (the LLA-2D key
// cache); the products then hold rows in a lane's registers (one token per
// lane), stored as 8 bytes of 4 consecutive features.  Otherwise a lane's
// register groups hold 4 consecutive tokens of one row, and the tile reaches
// the feature-major pages through LDS as whole 128-byte page rows.
template <int AXIS, bool TM>
__device__ __forceinline__ void encode_gemm_body(const EncodeArgs& a, int tb, int rb, int h0, int nh,
                                                 bf16_t (*s_x)[kGTok * kGS], bf16_t (*s_w)[kGRow * kGS],
                                                 float* s_mu, bf16_t* s_t) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane & 31, g = lane >> 5;
  constexpr int axis = AXIS;
  const int row0 = rb * kGRow;
  const int r = pick(a.r, axis), K = a.K, H = a.H;
  const int TT = a.B * a.M, t0 = tb * kGTok;
  const bf16_t* xg = static_cast<const bf16_t*>(pick(a.x, axis));
  const bf16_t* wg = static_cast<const bf16_t*>(pick(a.wdt, axis));
  // The workgroup walks heads h0 .. h0 + nh - 1 as one stream of K-chunks
  // (chunk q: head h0 + q / nkc, K offset (q % nkc) * kGKC), so the loads of a
  // head's first chunks are in flight while the previous head finishes.
  const int nkc = K / kGKC, total = nh * nkc;

  // staging: x chunk = 256 tokens x 64 (4 chunks of 16 bytes per thread),
  // W chunk = 96 rows x 64 (768 chunks: threads 0 .. 255 take two)
  uint4 sxa[4], swa[2], sxb[4], swb[2];  // two register sets, named at compile time
  auto load = [&](int q, uint4 (&sx)[4], uint4 (&sw)[2]) {
    const int hq = q / nkc, hh = h0 + hq, k0 = (q - hq * nkc) * kGKC;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + i * kGThreads, tok = c >> 3, part = c & 7, t = t0 + tok;
      sx[i] = ld16(xg + ((size_t)(t < TT ? t : TT - 1) * H + hh) * K + k0 + 8 * part);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * kGThreads, row = row0 + (c >> 3), part = c & 7;
      sw[i] = ld16(wg + ((size_t)hh * r + (row < r ? row : r - 1)) * K + k0 + 8 * part);
    }
  };
  auto store = [&](const uint4 (&sx)[4], const uint4 (&sw)[2], int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + i * kGThreads, tok = c >> 3, part = c & 7;
      *reinterpret_cast<uint4*>(&s_x[buf][tok * kGS + 8 * part]) = t0 + tok < TT ? sx[i] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * kGThreads, rr = c >> 3, part = c & 7;
      if (c < kGRow * 8)
        *reinterpret_cast<uint4*>(&s_w[buf][rr * kGS + 8 * part]) = row0 + rr < r ? sw[i] : make_uint4(0, 0, 0, 0);
    }
  };

  f32x16 acc[3], accm = f32x16{0.f};
#pragma unroll
  for (int rt = 0; rt < 3; ++rt) acc[rt] = f32x16{0.f};
  const bool mu = pick(a.mu, axis) != nullptr;  // uniform
  const bf16_t* mug = mu ? static_cast<const bf16_t*>(pick(a.mu, axis)) + 8 * g : nullptr;

  auto chunk = [&](int q, int buf) {
    const bf16_t* xs = &s_x[buf][(32 * wave + col) * kGS + 8 * g];
    const bf16_t* ws = &s_w[buf][col * kGS + 8 * g];
#pragma unroll
    for (int s = 0; s < kGKC / 16; ++s) {
      const bf16x8 xo = as_bf16x8(*reinterpret_cast<const uint4*>(xs + 16 * s));
#pragma unroll
      for (int rt = 0; rt < 3; ++rt) {
        const bf16x8 wo = as_bf16x8(*reinterpret_cast<const uint4*>(ws + 32 * rt * kGS + 16 * s));
        acc[rt] = TM ? mfma32(wo, xo, acc[rt]) : mfma32(xo, wo, acc[rt]);
      }
    }
    // the mean's products in one block after the chunk's (a guard inside the
    // K-step loop made each of them a block of its own)
    if (mu && wave < 3) {
      uint4 wm[kGKC / 16], mo[kGKC / 16];
#pragma unroll
      for (int s = 0; s < kGKC / 16; ++s) {
        wm[s] = *reinterpret_cast<const uint4*>(ws + 32 * wave * kGS + 16 * s);
        mo[s] = ld16(mug + (size_t)(h0 + q / nkc) * K + (q % nkc) * kGKC + 16 * s);
      }
#pragma unroll
      for (int s = 0; s < kGKC / 16; ++s) accm = mfma32(as_bf16x8(wm[s]), as_bf16x8(mo[s]), accm);
    }
  };

  // head hh done: the mean's products to LDS, the tile to the cache, then the
  // accumulators cleared for the next head
  auto finish = [&](int hh_) {
    // Opaque copies: the epilogue's row and token bookkeeping is then formed
    // here, per head, instead of being hoisted out of the head loop, where it
    // would hold registers across every chunk.
    int hh = hh_, r = pick(a.r, axis), row0 = rb * kGRow, t0 = tb * kGTok;
    asm volatile("" : "+s"(hh), "+s"(r), "+s"(row0), "+s"(t0));
    if (mu) {
      // accm (M = row of tile `wave`, N = any column): rows 8(q/4) + 4g + q%4
      if (wave < 3 && col == 0) {
#pragma unroll
        for (int q = 0; q < 16; ++q) s_mu[32 * wave + 8 * (q / 4) + 4 * g + q % 4] = accm[q];
      }
      __syncthreads();
    }

    bf16_t* cout = static_cast<bf16_t*>(pick(a.c, axis));
    if constexpr (TM) {
      // lane (token col, half g), register q of row tile rt: row 32 rt + 8(q/4) + 4g + q%4
      const int t = t0 + 32 * wave + col;
      if (t < TT) {
        const int b = t / a.M, pos = ring_slot(a.pos0 + (t - b * a.M), a.sink, a.window);
#pragma unroll
        for (int rt = 0; rt < 3; ++rt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int rl = 32 * rt + 8 * i + 4 * g, row = row0 + rl;  // first of 4 consecutive rows
            if (row + 3 < r) {
              // token-major cache: the 4 rows are contiguous, 8-byte aligned (r_k % 32 == 0)
              const uint32_t lo = uint32_t(f32_to_bf16(acc[rt][4 * i] - (mu ? s_mu[rl] : 0.f))) |
                                  (uint32_t(f32_to_bf16(acc[rt][4 * i + 1] - (mu ? s_mu[rl + 1] : 0.f))) << 16);
              const uint32_t hi = uint32_t(f32_to_bf16(acc[rt][4 * i + 2] - (mu ? s_mu[rl + 2] : 0.f))) |
                                  (uint32_t(f32_to_bf16(acc[rt][4 * i + 3] - (mu ? s_mu[rl + 3] : 0.f))) << 16);
              *reinterpret_cast<uint2*>(&cout[cache_index(b, hh, H, a.n_max, r, pos, row, true)]) = make_uint2(lo, hi);
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (row + e < r)
                  cout[cache_index(b, hh, H, a.n_max, r, pos, row + e, true)] =
                      f32_to_bf16(acc[rt][4 * i + e] - (mu ? s_mu[rl + e] : 0.f));
            }
          }
      }
    } else {
      // lane (row col of tile rt, half g), register q: token 32 wave + 8(q/4) + 4g + q%4,
      // so registers 4i .. 4i + 3 are 4 consecutive tokens of one feature row.
      // The tile goes through LDS as [row][token] bf16, then runs of 8 threads
      // store a row's 64 tokens of one page as 128 contiguous bytes (16 bytes
      // each) when the slots are 8 consecutive positions of one sequence (no
      // ring, a position a multiple of 8), else one element at a time.
#pragma unroll
      for (int rt = 0; rt < 3; ++rt) {
        const int rl = 32 * rt + col;
        const float m = mu ? s_mu[rl] : 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t lo = uint32_t(f32_to_bf16(acc[rt][4 * i] - m)) |
                              (uint32_t(f32_to_bf16(acc[rt][4 * i + 1] - m)) << 16);
          const uint32_t hi = uint32_t(f32_to_bf16(acc[rt][4 * i + 2] - m)) |
                              (uint32_t(f32_to_bf16(acc[rt][4 * i + 3] - m)) << 16);
          *reinterpret_cast<uint2*>(&s_t[rl * kGTS + 32 * wave + 8 * i + 4 * g]) = make_uint2(lo, hi);
        }
      }
      __syncthreads();
      constexpr int kItems = kGRow * (kGTok / 8) / kGThreads;  // 16-byte pieces per thread
#pragma unroll
      for (int k = 0; k < kItems; ++k) {
        const int item = tid + k * kGThreads, rl = item / (kGTok / 8), grp = item % (kGTok / 8);
        const int row = row0 + rl;
        if (row >= r) continue;
        const uint4 v = *reinterpret_cast<const uint4*>(&s_t[rl * kGTS + 8 * grp]);
        const int t = t0 + 8 * grp;  // first token of the piece
        const int b = t / a.M, m0 = t - b * a.M, p = a.pos0 + m0;
        if (a.window == 0 && t + 7 < TT && m0 + 7 < a.M && (p & 7) == 0) {
          *reinterpret_cast<uint4*>(&cout[cache_index(b, hh, H, a.n_max, r, p, row)]) = v;
        } else {
          const bf16_t* e8 = reinterpret_cast<const bf16_t*>(&v);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int te = t + e;
            if (te < TT) {
              const int be = te / a.M, pos = ring_slot(a.pos0 + (te - be * a.M), a.sink, a.window);
              cout[cache_index(be, hh, H, a.n_max, r, pos, row)] = e8[e];
            }
          }
        }
      }
    }
#pragma unroll
    for (int rt = 0; rt < 3; ++rt) acc[rt] = f32x16{0.f};
    accm = f32x16{0.f};
  };

  // set a holds even chunks, set b odd ones; chunk q is in LDS buffer q % 2
  // (nkc is even whenever a workgroup takes more than one head, so every head
  // starts on set a).  Each head's last chunk is followed, after the barrier,
  // by its epilogue; the barriers of the next head's chunks order its use of
  // LDS against the next epilogue.
  load(0, sxa, swa);
  load(total > 1 ? 1 : 0, sxb, swb);
  store(sxa, swa, 0);
  __syncthreads();
  for (int hq = 0; hq < nh; ++hq) {
    const int qe = (hq + 1) * nkc;  // end of this head's chunks
    for (int q = hq * nkc; q < qe; q += 2) {
      load(min(q + 2, total - 1), sxa, swa);
      chunk(q, 0);
      if (q + 1 < total) store(sxb, swb, 1);
      __syncthreads();
      if (q + 1 < qe) {
        load(min(q + 3, total - 1), sxb, swb);
        chunk(q + 1, 1);
        if (q + 2 < total) store(sxa, swa, 0);
        __syncthreads();
      }
    }
    finish(h0 + hq);
  }
}

// Both axes in one launch (1024 equal workgroups for the 2D prompt write of
// 4 x 8192 tokens: four full rounds of the machine).  XCD-aware order: the
// j-th workgroup of XCD x takes token block x + 8 (j / nrb) and row block
// j % nrb (the row blocks of axis k, then those of axis v).
__global__ __launch_bounds__(kGThreads) __attribute__((amdgpu_waves_per_eu(2)))
void encode_gemm_kernel(EncodeArgs a, int nrb_k, int nrb, int ntb, int hpw) {
  __shared__ __attribute__((aligned(16))) bf16_t s_x[2][kGTok * kGS];
  __shared__ __attribute__((aligned(16))) bf16_t s_w[2][kGRow * kGS];
  __shared__ float s_mu[kGRow];
  __shared__ __attribute__((aligned(16))) bf16_t s_t[kGRow * kGTS];  // epilogue tile (feature-major outputs)
  const int xcd = blockIdx.x % 8, j = blockIdx.x / 8;
  const int tb = xcd + 8 * (j / nrb), rb = j % nrb;
  if (tb >= ntb) return;  // padding of the grid to whole rounds of 8 token blocks
  const int h0 = blockIdx.y * hpw, nh = min(hpw, a.H - h0);  // a run of heads
  if (rb >= nrb_k)
    encode_gemm_body<1, false>(a, tb, rb - nrb_k, h0, nh, s_x, s_w, s_mu, s_t);
  else if (a.k_token_major)
    encode_gemm_body<0, true>(a, tb, rb, h0, nh, s_x, s_w, s_mu, s_t);
  else
    encode_gemm_body<0, false>(a, tb, rb, h0, nh, s_x, s_w, s_mu, s_t);
}

// Second launch of a split write: tile unit (grid x, y, z as the split launch
// with z = head) adds its ksplit fp32 partials in split order and writes the
// cache exactly as the unsplit path does.
__global__ __launch_bounds__(256) void encode_reduce_kernel(EncodeArgs a, int nrc_k) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int axis = blockIdx.y >= (unsigned)nrc_k ? 1 : 0;
  const int rc = blockIdx.y - axis * nrc_k;
  const int h = blockIdx.z, H = a.H, r = pick(a.r, axis), TT = a.B * a.M;
  const int li = lane & 15, lg = lane >> 4;
  const size_t unit = ((size_t)h * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
  const float* part = a.part + unit * a.ksplit * 1024 + tid * 4;
  constexpr int kPre = 32;  // partials in flight at once
  f32x4 v[kPre];
#pragma unroll
  for (int s = 0; s < kPre; ++s)
    v[s] = s < a.ksplit ? *reinterpret_cast<const f32x4*>(part + (size_t)s * 1024) : f32x4{0.f};
  f32x4 acc = f32x4{0.f};
#pragma unroll
  for (int s = 0; s < kPre; ++s) acc += v[s];
  const int t = blockIdx.x * 32 + (wave >> 1) * 16 + li;
  if (t < TT) {
    const int b = t / a.M, pos = ring_slot(a.pos0 + (t - b * a.M), a.sink, a.window);
    bf16_t* c = static_cast<bf16_t*>(pick(a.c, axis));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int rr = rc * 32 + (wave & 1) * 16 + 4 * lg + e;
      if (rr < r) c[cache_index(b, h, H, a.n_max, r, pos, rr, axis == 0 && a.k_token_major)] = f32_to_bf16(acc[e]);
    }
  }
}

// fp32: 16 tokens x 16 rows per workgroup, K staged through LDS in chunks of 64.
constexpr int kT = 16, kKC = 64;
__global__ __launch_bounds__(256) void encode_f32_kernel(EncodeArgs a) {
  __shared__ float s_x[kT][kKC + 1];
  __shared__ float s_w[kT][kKC + 1];
  const int axis = blockIdx.z / a.H, h = blockIdx.z - axis * a.H;
  const int r = pick(a.r, axis), K = a.K, TT = a.B * a.M;
  if (blockIdx.y * kT >= r) return;
  const int tt = threadIdx.x / kT, rr = threadIdx.x % kT;
  const int tok = blockIdx.x * kT + tt, row = blockIdx.y * kT + rr;
  const float* x = static_cast<const float*>(pick(a.x, axis));
  const float* w = static_cast<const float*>(pick(a.wdt, axis)) + (size_t)h * r * K;
  const float* mu = pick(a.mu, axis) ? static_cast<const float*>(pick(a.mu, axis)) + (size_t)h * K : nullptr;
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
    const int b = tok / a.M, pos = ring_slot(a.pos0 + (tok - b * a.M), a.sink, a.window);
    static_cast<float*>(pick(a.c, axis))[cache_index(b, h, a.H, a.n_max, r, pos, row, axis == 0 && a.k_token_major)] = acc;
  }
}

}  // namespace

static int gemm_heads_per_wg(int H, int blocks, int nkc) {
  if (nkc % 2) return 1;  // a run of heads needs every head to start on the same register set
  const int hpw = (int)((int64_t)H * blocks / 1024);
  return hpw < 1 ? 1 : hpw > H ? H : hpw;
}

int encode_ksplit(int TT, int K) {
  if (TT > 64 || K < 2048) return 1;
  const int s = K / 512;  // 16 K-steps (one round of loads) per split
  return s > 32 ? 32 : s;
}

size_t encode_ws_bytes(int B, int M, int H, int K, int r_k, int r_v) {
  const int TT = B * M, ks = encode_ksplit(TT, K);
  if (ks == 1) return 0;
  const size_t units = (size_t)((TT + kEncTok - 1) / kEncTok) * ((r_k + 31) / 32 + (r_v + 31) / 32) * H;
  return units * ks * 1024 * sizeof(float);
}

hipError_t launch_encode(const EncodeArgs& a, hipStream_t stream) {
  const int TT = a.B * a.M;
  const int rmax = a.r[0] > a.r[1] ? a.r[0] : a.r[1];
  if (a.dtype == LLA_BF16) {
    // Many tokens: a workgroup streams all heads of its 32 tokens (one
    // contiguous region of x).  Fewer tokens: one head and two row tiles per
    // workgroup, so the weights spread over the machine.
    const int blocks = (TT + kEncTok - 1) / kEncTok;
    if (TT <= 64) {  // a decode step's writes: weights read once, one round of loads
      const int nrc_k = (a.r[0] + 31) / 32, nrc_v = (a.r[1] + 31) / 32;
      dim3 grid(blocks, nrc_k + nrc_v, a.H * a.ksplit);
      hipLaunchKernelGGL(encode_few_kernel, grid, dim3(256), 0, stream, a, nrc_k);
      if (a.ksplit > 1)
        hipLaunchKernelGGL(encode_reduce_kernel, dim3(blocks, nrc_k + nrc_v, a.H), dim3(256), 0, stream, a, nrc_k);
      return hipGetLastError();
    }
    if (blocks >= 256 && rmax <= 64 && (a.K == 512 || a.K == 256)) {
      // prefill-sized write: resident weights, streamed tokens; ~2 workgroups per CU
      const int per_head = 2 * a.H;
      int wgx = (2 * device_cu_count() + per_head - 1) / per_head;
      if (wgx > blocks) wgx = blocks;
      const int bpw = (blocks + wgx - 1) / wgx;
      dim3 grid((blocks + bpw - 1) / bpw, a.H, 2);
      if (a.K == 512)
        hipLaunchKernelGGL((encode_stream_kernel<16>), grid, dim3(256), 0, stream, a, bpw);
      else
        hipLaunchKernelGGL((encode_stream_kernel<8>), grid, dim3(256), 0, stream, a, bpw);
      return hipGetLastError();
    }
    if (TT >= kGTok && a.K % kGKC == 0 && (a.K >= 2048 || rmax > 64)) {
      // prefill-sized write over a long stack (the LLA-2D down-projection), or
      // at ranks above the streaming kernel's (the per-head tiers): a GEMM
      // tiled for the MFMAs, x re-read from L2 per row block
      const int ntb = (TT + kGTok - 1) / kGTok, ntb8 = (ntb + 7) / 8 * 8;
      const int nrb_k = (a.r[0] + kGRow - 1) / kGRow, nrb = nrb_k + (a.r[1] + kGRow - 1) / kGRow;
      // heads per workgroup: as many as keep at least 1024 workgroups (four
      // rounds of the machine), so short stacks (per-head writes) do not pay
      // the pipeline fill and the epilogue per head on their own
      const int hpw = gemm_heads_per_wg(a.H, nrb * ntb8, a.K / kGKC);
      hipLaunchKernelGGL(encode_gemm_kernel, dim3(nrb * ntb8, (a.H + hpw - 1) / hpw), dim3(kGThreads), 0, stream, a,
                         nrb_k, nrb, ntb, hpw);
      return hipGetLastError();
    }
    const int heads_per_wg = blocks >= 256 ? a.H : 1;
    const int rtmax = (rmax + 15) / 16;
    const int rt_per_wg = blocks >= 256 ? (rtmax < 8 ? rtmax : 8) : 2;
    const int nrc = (rtmax + rt_per_wg - 1) / rt_per_wg;
    dim3 grid(blocks, (a.H + heads_per_wg - 1) / heads_per_wg, 2 * nrc);
    hipLaunchKernelGGL(encode_bf16_kernel, grid, dim3(256), 0, stream, a, heads_per_wg, rt_per_wg, nrc);
  } else {
    dim3 grid((TT + kT - 1) / kT, (rmax + kT - 1) / kT, 2 * a.H);
    hipLaunchKernelGGL(encode_f32_kernel, grid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace lla
