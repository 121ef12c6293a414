// LLA-2D causal prefill at loop l (Sec. 3 "The LLA-2D variant (loop x head)";
// App. J "Per-head LLA versus LLA-2D at inference": either variant may take
// the full-memory path that materialises K/V or attend over the latents).
//
// With one latent per token for all heads the ranks exceed d_head (288 / 480
// against 128 at the 21.33x operating point), so the absorbed form would cost
// 2 (r_k + r_v) flops per causal score, against 2 d_head (r_k + r_v) per key
// and head to rebuild K and V once plus 4 d_head per score to attend over them.
// For a prompt of M new tokens that is about 3x fewer flops from M ~ 128 on,
// so this path rebuilds:
//
//   recon2d_kernel:  K_h = C_k U_{k,h}^T and V_h = C_v U_{v,h}^T (Eq. 3 with the
//                    (l, h) slice of W_up) for every cached token n < p0 + M,
//                    rounded to fp16, into a caller-owned workspace;
//   flash2d_kernel:  causal attention of the M queries of every head over its
//                    rebuilt K_h, V_h (d_head = 128), online softmax over
//                    64-key pages, then out = O / l + mu_v.
//
// mu_k is not added: q . mu_k is the same for every key and cancels in the
// softmax.  mu_v is added to the normalised output (the weights sum to 1).
//
// The attention's products run on fp16 MFMAs (the same rate as bf16 on this
// chip): the bf16 query converts to fp16 exactly, and the rebuilt K and V and
// the softmax weights keep 11 significant bits instead of bf16's 8, so the
// rounding of these intermediates stays well inside the bf16 error budget even
// for peaked rows.  Values beyond fp16's range (65504) become infinite and the
// output is then not finite.
//
// Workspace layouts, chosen so that every MFMA operand of the attention is one
// 16-byte LDS read:
//   kh [B][H][nk][128]            keys token-major (a key's 128 features contiguous)
//   vt [B][H][nk/64][128][64]     values feature-major per 64-key page; inside each
//                                 16-key block the keys are stored in the order
//                                 0-3, 8-11, 4-7, 12-15 (the order in which a
//                                 32x32 accumulator hands its rows to a lane half)
// with nk = p0 + M rounded up to a page; tokens n >= p0 + M are written as 0.

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kD = 128;            // d_head of both kernels
constexpr int kThreads = 256;      // 4 wavefronts
constexpr int kRTok = 128;         // tokens per rebuild workgroup (two pages)
constexpr int kQBlock = 256;       // queries per attention workgroup (32 per wavefront)
constexpr int kFThreads = 512;     // attention workgroup: 8 wavefronts
constexpr float kLazy = 8.0f;      // raise the running max only when it grows by more than this (log2)

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f16x8 as_f16x8(uint4 v) { return __builtin_bit_cast(f16x8, v); }
__device__ __forceinline__ f32x16 mfma_h(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
// two fp32 values as bf16 (output) or fp16 (rebuilt K / V), round to nearest even
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return uint32_t(f32_to_bf16(lo)) | (uint32_t(f32_to_bf16(hi)) << 16);
}
__device__ __forceinline__ uint32_t pack2h(float lo, float hi) {
  const _Float16 a = (_Float16)lo, b = (_Float16)hi;
  return uint32_t(__builtin_bit_cast(uint16_t, a)) | (uint32_t(__builtin_bit_cast(uint16_t, b)) << 16);
}
typedef short i16x4 __attribute__((ext_vector_type(4)));
// ds_read_b64_tr_b16: each 16-lane group reads a 16 x 4 block of 16-bit values
// (lane L: 4 consecutive elements at its address) and lane L receives element
// L % 4 of the lanes 4 e + L / 4, e = 0..3
__device__ __forceinline__ uint2 lds_tr16(const bf16_t* p) {
  return __builtin_bit_cast(uint2,
                            __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p)));
}

// max over both halves of the wavefront (lane i and lane i ^ 32)
__device__ __forceinline__ float half_swap_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_swap_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---------------------------------------------------------------------------
// Rebuild.  One workgroup = 128 tokens of one sequence, every head: the latent
// tile is staged once in LDS token-major (a token's r features contiguous) and
// wavefront w computes features 32w .. 32w + 31 of every head, with that
// head's up-projection rows as the other operand (16-byte loads).
//   keys:   D = K^T (M = feature, N = token, K = latent feature j), so a lane
//           holds 4-feature runs of one token (8-byte stores);
//   values: D = V (M = token, N = feature), so a lane holds the tokens
//           16 b + 8 g .. + 7 of the permuted order of one feature (16-byte stores).
// ---------------------------------------------------------------------------
template <int N>
struct IntC {
  static constexpr int value = N;
};

// Feature-major pages (the values; the per-head caches below) are staged as
// they are, 16-byte chunks of 8 tokens of one feature, with the chunk index of
// rows 4k+2, 4k+3 XORed with 4; ds_read_b64_tr_b16 then hands each lane one
// token's 4 consecutive features, the MFMA operand layout.  Both the staging
// stores and the transposed reads are free of bank conflicts.  (The keys are
// token-major already and are staged row by row.)
template <int AXIS, int KS>  // AXIS 0: keys, 1: values; KS = r / 16
__global__ __launch_bounds__(kThreads) void recon2d_kernel(Prefill2dArgs a) {
  constexpr int R = KS * 16;
  constexpr int TOK = kRTok;           // tokens per workgroup
  constexpr bool FM = AXIS == 1;       // the latents arrive as feature-major pages
  constexpr int CS = R + 8;  // token-major LDS row stride (bf16): 16-byte reads of 16 rows hit distinct banks
  constexpr int LDS = FM ? (TOK / kPage) * R * kPage : TOK * CS;
  __shared__ __attribute__((aligned(16))) bf16_t s_c[LDS];

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane & 31, g = lane >> 5;
  const int b = blockIdx.y, n0 = blockIdx.x * TOK;
  const int nvalid = a.p0 + a.M;  // tokens that hold latents; the rest are rebuilt as 0
  const int H = a.H;
  constexpr int rr = R;  // the cache's rank (row pitch of its pages)

  // ---- latent tile, zero past nvalid (and past rr) ----
  if constexpr (!FM) {
    const bf16_t* src = static_cast<const bf16_t*>(a.ck) + (size_t)b * a.n_max * R;
    constexpr int C8 = R / 8;
    for (int e = tid; e < TOK * C8; e += kThreads) {
      const int n = e / C8, c8 = e - n * C8;
      const uint4 v = n0 + n < nvalid ? ld16(src + (size_t)(n0 + n) * R + 8 * c8) : make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4*>(&s_c[n * CS + 8 * c8]) = v;
    }
  } else {
    // chunk e: page pg, feature row j, 8-token chunk c (consecutive e are
    // consecutive 16 bytes of the cache)
    const bf16_t* src = static_cast<const bf16_t*>(a.cv) + (size_t)b * a.n_max * rr;
    for (int e = tid; e < TOK / kPage * R * 8; e += kThreads) {
      const int pg = e / (R * 8), rem = e - pg * (R * 8), j = rem >> 3, c = rem & 7;
      const int nb = n0 + pg * kPage + 8 * c;  // first token of the chunk
      uint4 v = make_uint4(0, 0, 0, 0);
      if (nb < nvalid && j < rr) {
        v = ld16(src + (size_t)(n0 / kPage + pg) * kPage * rr + (size_t)j * kPage + 8 * c);
        const int nv = nvalid - nb;  // tokens of the chunk that hold latents
        if (nv < 8) {
          auto keep = [nv](int i) { return nv > 2 * i + 1 ? 0xffffffffu : nv > 2 * i ? 0x0000ffffu : 0u; };
          v.x &= keep(0);
          v.y &= keep(1);
          v.z &= keep(2);
          v.w &= keep(3);
        }
      }
      *reinterpret_cast<uint4*>(&s_c[(pg * R + j) * kPage + ((c ^ (((j >> 1) & 1) << 2)) << 3)]) = v;
    }
  }
  __syncthreads();

  // The latent operand of K-step s for 32-token tile nt: lane (col, g) gets
  // features 16 s + 8 g .. + 7 of token 32 nt + col.  Transposed reads: lane
  // (x16, th) of a 16-lane group addresses feature row 16 s + 8 g + x16 / 4
  // (+ 4 for the second read) and tokens 16 th + 4 (x16 % 4) .. + 3 of its tile.
  const int x16 = lane & 15, th = (lane >> 4) & 1, sw1 = (x16 >> 3) & 1;
  const int troff = (8 * g + (x16 >> 2)) * kPage + ((2 * th + ((x16 & 3) >> 1)) << 3) + 4 * (x16 & 1);
  auto lat_op = [&](int nt, int s) -> bf16x8 {
    if constexpr (!FM) {
      return as_bf16x8(*reinterpret_cast<const uint4*>(&s_c[(32 * nt + col) * CS + 16 * s + 8 * g]));
    } else {
      const bf16_t* p = s_c + (nt >> 1) * R * kPage + troff + ((4 * ((nt & 1) ^ sw1)) << 3) + 16 * s * kPage;
      const uint2 r0 = lds_tr16(p), r1 = lds_tr16(p + 4 * kPage);
      return as_bf16x8(make_uint4(r0.x, r0.y, r1.x, r1.y));
    }
  };

  const bf16_t* U = static_cast<const bf16_t*>(AXIS == 0 ? a.uk : a.uv);
  const int ntile = min(TOK, a.nk - n0) / 32;  // 32-token tiles of this workgroup inside nk
  // up-projection rows 32 wave + col of head h as K-step operands
  auto load_u = [&](int h, uint4 (&u)[KS]) {
    const bf16_t* row = U + ((size_t)h * kD + 32 * wave + col) * R + 8 * g;
#pragma unroll
    for (int s = 0; s < KS; ++s) u[s] = ld16(row + 16 * s);
  };
  uint4 ua[KS];
  // NT = the workgroup's token tiles, a compile-time count so the product loop
  // has no branches (a guard per product had split every MFMA into a block of
  // its own, each waiting on its own LDS read)
  auto head = [&](int h, const uint4 (&u)[KS], auto ntc) {
    constexpr int NT = decltype(ntc)::value;
    f32x16 acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x16{0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const bf16x8 c = lat_op(nt, s);
        acc[nt] = AXIS == 0 ? mfma(as_bf16x8(u[s]), c, acc[nt]) : mfma(c, as_bf16x8(u[s]), acc[nt]);
      }
    }
    const size_t bh = (size_t)b * H + h;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (AXIS == 0) {
        // lane (token col, half g), register r: feature 32 wave + 8 (r/4) + 4 g + r%4
        uint16_t* dst = static_cast<uint16_t*>(a.kh) + (bh * a.nk + n0 + 32 * nt + col) * kD + 32 * wave + 4 * g;
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4)
          *reinterpret_cast<uint2*>(dst + 8 * c4) =
              make_uint2(pack2h(acc[nt][4 * c4], acc[nt][4 * c4 + 1]), pack2h(acc[nt][4 * c4 + 2], acc[nt][4 * c4 + 3]));
      } else {
        // lane (feature col, half g), registers 8 blk .. 8 blk + 7: tokens at
        // permuted positions 16 blk + 8 g .. + 7 of the tile's 32
        const int tok0 = n0 + 32 * nt;
        uint16_t* dst = static_cast<uint16_t*>(a.vt) +
                      ((bh * (a.nk / kPage) + tok0 / kPage) * kD + 32 * wave + col) * kPage + tok0 % kPage + 8 * g;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
          const f32x16& x = acc[nt];
          const int r0 = 8 * blk;
          *reinterpret_cast<uint4*>(dst + 16 * blk) =
              make_uint4(pack2h(x[r0], x[r0 + 1]), pack2h(x[r0 + 2], x[r0 + 3]), pack2h(x[r0 + 4], x[r0 + 5]),
                         pack2h(x[r0 + 6], x[r0 + 7]));
        }
      }
    }
  };
  // every operand load of a head is issued before its first product, so the
  // products of the early K-steps overlap the later loads
  for (int h = 0; h < H; ++h) {
    load_u(h, ua);
    switch (ntile) {  // uniform; 2 or 4 (the key count is a multiple of 64)
      case 4: head(h, ua, IntC<4>{}); break;
      case 2: head(h, ua, IntC<2>{}); break;
      default: break;
    }
  }
}

// ---------------------------------------------------------------------------
// Per-head rebuild over a run of pages.  One workgroup = one (b, h) and up to
// `ppw` consecutive 64-token pages: the head's up-projection rows are loaded
// into registers once, and while one page's products run from LDS the next
// page's latents are already in flight into registers.  Staging, operand
// reads (ds_read_b64_tr_b16) and outputs are those of the per-head
// recon2d_kernel above.
// ---------------------------------------------------------------------------
template <int AXIS, int KS>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void recon_ph_kernel(Prefill2dArgs a, int ppw) {
  constexpr int R = KS * 16;
  constexpr int CPT = (R * 8 + kThreads - 1) / kThreads;  // 16-byte chunks of a page per thread
  __shared__ __attribute__((aligned(16))) bf16_t s_c[R * kPage];

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane & 31, g = lane >> 5;
  const int bh = blockIdx.y, h = bh % a.H;
  const int nvalid = a.p0 + a.M;
  const int rr = AXIS == 0 ? a.rk : a.rv;
  const int pg0 = blockIdx.x * ppw, pg1 = min(pg0 + ppw, a.nk / kPage);
  const bf16_t* src = static_cast<const bf16_t*>(AXIS == 0 ? a.ck : a.cv) + (size_t)bh * a.n_max * rr;

  // this thread's chunks of a page: chunk e = tid + 256 i is feature row e / 8,
  // tokens 8 (e % 8) .. + 7
  uint4 stg[CPT];
  auto gload = [&](int pg) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int e = tid + i * kThreads, j = e >> 3, c = e & 7;
      const int nb = pg * kPage + 8 * c;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (e < R * 8 && j < rr && nb < nvalid) {
        v = ld16(src + (size_t)pg * kPage * rr + (size_t)j * kPage + 8 * c);
        const int nv = nvalid - nb;
        if (nv < 8) {
          auto keep = [nv](int q) { return nv > 2 * q + 1 ? 0xffffffffu : nv > 2 * q ? 0x0000ffffu : 0u; };
          v.x &= keep(0);
          v.y &= keep(1);
          v.z &= keep(2);
          v.w &= keep(3);
        }
      }
      stg[i] = v;
    }
  };
  auto lstore = [&]() {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int e = tid + i * kThreads, j = e >> 3, c = e & 7;
      if (e < R * 8) *reinterpret_cast<uint4*>(&s_c[j * kPage + ((c ^ (((j >> 1) & 1) << 2)) << 3)]) = stg[i];
    }
  };
  const int x16 = lane & 15, th = (lane >> 4) & 1, sw1 = (x16 >> 3) & 1;
  const int troff = (8 * g + (x16 >> 2)) * kPage + ((2 * th + ((x16 & 3) >> 1)) << 3) + 4 * (x16 & 1);
  auto lat_op = [&](int nt, int s) -> bf16x8 {  // token tile nt (0, 1) of the staged page
    const bf16_t* p = s_c + troff + ((4 * (nt ^ sw1)) << 3) + 16 * s * kPage;
    const uint2 r0 = lds_tr16(p), r1 = lds_tr16(p + 4 * kPage);
    return as_bf16x8(make_uint4(r0.x, r0.y, r1.x, r1.y));
  };
  // up-projection rows 32 wave + col of head h (features past rr are zero)
  uint4 ua[KS];
  {
    const bf16_t* row = static_cast<const bf16_t*>(AXIS == 0 ? a.uk : a.uv) + ((size_t)h * kD + 32 * wave + col) * rr + 8 * g;
#pragma unroll
    for (int s = 0; s < KS; ++s) ua[s] = 16 * s + 8 * g < rr ? ld16(row + 16 * s) : make_uint4(0, 0, 0, 0);
  }
  if (pg0 < pg1) gload(pg0);
  for (int pg = pg0; pg < pg1; ++pg) {
    lstore();
    __syncthreads();
    if (pg + 1 < pg1) gload(pg + 1);  // in flight during this page's products
    f32x16 acc[2] = {f32x16{0.f}, f32x16{0.f}};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const bf16x8 c = lat_op(nt, s);
        acc[nt] = AXIS == 0 ? mfma(as_bf16x8(ua[s]), c, acc[nt]) : mfma(c, as_bf16x8(ua[s]), acc[nt]);
      }
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int tok0 = pg * kPage + 32 * nt;
      if (AXIS == 0) {
        // lane (token col, half g), register r: feature 32 wave + 8 (r/4) + 4 g + r%4
        uint16_t* dst = static_cast<uint16_t*>(a.kh) + ((size_t)bh * a.nk + tok0 + col) * kD + 32 * wave + 4 * g;
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4)
          *reinterpret_cast<uint2*>(dst + 8 * c4) =
              make_uint2(pack2h(acc[nt][4 * c4], acc[nt][4 * c4 + 1]), pack2h(acc[nt][4 * c4 + 2], acc[nt][4 * c4 + 3]));
      } else {
        // lane (feature col, half g), registers 8 blk .. + 7: tokens at permuted
        // positions 16 blk + 8 g .. + 7 of the tile
        uint16_t* dst = static_cast<uint16_t*>(a.vt) +
                        (((size_t)bh * (a.nk / kPage) + pg) * kD + 32 * wave + col) * kPage + 32 * nt + 8 * g;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
          const f32x16& x = acc[nt];
          const int r0 = 8 * blk;
          *reinterpret_cast<uint4*>(dst + 16 * blk) =
              make_uint4(pack2h(x[r0], x[r0 + 1]), pack2h(x[r0 + 2], x[r0 + 3]), pack2h(x[r0 + 4], x[r0 + 5]),
                         pack2h(x[r0 + 6], x[r0 + 7]));
        }
      }
    }
    __syncthreads();  // the page's LDS tile is read by every wavefront before the next is stored
  }
}

// ---------------------------------------------------------------------------
// Attention.  One workgroup = 8 wavefronts x 32 queries of one (b, h); keys in
// 64-token pages staged in LDS (K token-major, V feature-major) once for the 8
// wavefronts, two pages in flight in registers.  Products (v_mfma_f32_32x32x16_f16), transposed so each
// accumulator feeds the next product with no lane exchange:
//   S^T  (M = key, N = query, K = feature): A = K tile rows,  B = the query (registers)
//   O^T += (M = feature, N = query, K = key): A = V^T tile rows, B = P from S^T
// A 32x32 accumulator gives lane (q + 32 g), register r the row 8(r/4) + 4g + r%4
// of column q: registers 8u .. 8u + 7 of a key tile are the keys
// 16u + 8(e/4) + 4g + e%4, e < 8, which the permuted V^T rows hold contiguously.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kFThreads) __attribute__((amdgpu_waves_per_eu(2)))
void flash2d_kernel(Prefill2dArgs a) {
  constexpr int KS = kD / 16;       // K-steps of the score product
  constexpr int KST = kD + 8;       // K tile row stride (fp16 elements)
  constexpr int VST = kPage + 8;    // V^T tile row stride (fp16 elements)
  constexpr int KTILE = kPage * KST, VTILE = kD * VST;
  constexpr int CH = kPage * kD / 8 / kFThreads;  // 16-byte chunks per thread per page and axis (2)
  __shared__ __attribute__((aligned(16))) uint16_t s_k[2 * KTILE];  // fp16
  __shared__ __attribute__((aligned(16))) uint16_t s_v[2 * VTILE];

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane & 31, g = lane >> 5;
  const int bh = blockIdx.x, h = bh % a.H;
  const int M = a.M, p0 = a.p0;
  const int nqb = (M + kQBlock - 1) / kQBlock;
  const int qb = nqb - 1 - (int)blockIdx.y;  // heaviest (latest) query blocks first
  const int q0 = qb * kQBlock, qw0 = q0 + 32 * wave;
  const int myq = qw0 + col;
  const bool q_ok = myq < M, wave_live = qw0 < M;
  const int qlast_w = min(qw0 + 31, M - 1);
  const int kmax = p0 + min(q0 + kQBlock, M);  // keys [0, kmax) matter to the workgroup
  const int npages = (kmax + kPage - 1) / kPage;

  // ---- page staging: both pages are 16 KB contiguous in the workspace ----
  const uint16_t* kbase = static_cast<const uint16_t*>(a.kh) + (size_t)bh * a.nk * kD;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.vt) + (size_t)bh * a.nk * kD;
  uint4 stk[2][CH], stv[2][CH];
  auto load_page = [&](int pg, int set) {
    const uint16_t* kp = kbase + (size_t)pg * kPage * kD;
    const uint16_t* vp = vbase + (size_t)pg * kPage * kD;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      stk[set][c] = ld16(kp + 8 * (tid + c * kFThreads));
      stv[set][c] = ld16(vp + 8 * (tid + c * kFThreads));
    }
  };
  auto store_page = [&](int set, int buf) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int ch = tid + c * kFThreads;
      *reinterpret_cast<uint4*>(&s_k[buf * KTILE + (ch >> 4) * KST + 8 * (ch & 15)]) = stk[set][c];
      *reinterpret_cast<uint4*>(&s_v[buf * VTILE + (ch >> 3) * VST + 8 * (ch & 7)]) = stv[set][c];
    }
  };

  load_page(0, 0);
  load_page(min(1, npages - 1), 1);
  // the query as the score product's B operand: lane (q, g), K-step s = features
  // 16s + 8g .. + 7, scaled by scale * log2(e) and rounded to fp16, so the score
  // product yields base-2 logits
  const float qs = a.qscale;
  f16x8 qop[KS];
  {
    const bf16_t* qrow = static_cast<const bf16_t*>(a.q) + ((size_t)bh * M + (q_ok ? myq : 0)) * kD + 8 * g;
    uint4 raw[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) raw[s] = ld16(qrow + 16 * s);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      float x[8];
      Elem<bf16_t>::unpack(raw[s], x);
#pragma unroll
      for (int e = 0; e < 8; ++e) qop[s][e] = (_Float16)(x[e] * qs);
    }
  }
  // One more K-step carries the running max: A holds 1 in feature 0 for every
  // key, B holds -m in feature 0 for the lane's query, so the score products
  // yield s - m directly.  m is kept representable in fp16 (every raise rounds
  // it), which makes the shift exact and the rescale exp2(m_old - m_new) exact.
  const f16x8 a_one = {(_Float16)(g == 0 ? 1.f : 0.f), 0, 0, 0, 0, 0, 0, 0};
  store_page(0, 0);
  __syncthreads();

  f32x16 oacc[kD / 32];
#pragma unroll
  for (int t = 0; t < kD / 32; ++t) oacc[t] = f32x16{0.f};
  float m_run = 0.f, l_lane = 0.f;  // the first page always raises m
  const int qpos = p0 + myq;

  auto page = [&](int p, auto bufc) {
    constexpr int buf = decltype(bufc)::value;
    // set buf held page p (already in LDS); page p + 2 goes into it (near the
    // end the last page is re-read, so every wait is for exactly one page)
    load_page(min(p + 2, npages - 1), buf);
    const int key0 = p * kPage;
    if (wave_live && key0 <= p0 + qlast_w) {
      const bool diag = key0 + kPage - 1 > p0 + qw0;
      const uint16_t* kt_row = s_k + buf * KTILE + col * KST + 8 * g;
      const uint16_t* vt_row = s_v + buf * VTILE + col * VST + 8 * g;
      // all of the page's operand fragments are read from LDS ahead of their
      // products (scheduling fences keep them there): the 16 K fragments before
      // the score products, which then issue back to back, and the 16 V fragments
      // right after them, so the value reads overlap the score products and the
      // softmax (1.314 -> 1.281 ms per call on 4 x 8192 tokens, 16 heads)
      uint4 kop[KS][2];
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) kop[s][kt] = *reinterpret_cast<const uint4*>(kt_row + 32 * kt * KST + 16 * s);
      __builtin_amdgcn_sched_barrier(0);
      const f16x8 b_m = {(_Float16)(g == 0 ? -m_run : 0.f), 0, 0, 0, 0, 0, 0, 0};
      f32x16 sc[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) sc[kt] = mfma_h(a_one, b_m, f32x16{0.f});
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) sc[kt] = mfma_h(as_f16x8(kop[s][kt]), qop[s], sc[kt]);
      uint4 vop[2][kD / 32][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int t = 0; t < kD / 32; ++t)
#pragma unroll
          for (int u = 0; u < 2; ++u)
            vop[kt][t][u] = *reinterpret_cast<const uint4*>(vt_row + 32 * t * VST + 32 * kt + 16 * u);
      __builtin_amdgcn_sched_barrier(0);
      const int lim = qpos - key0 - 4 * g;
      if (__builtin_expect(diag, 0)) {
        // key 32kt + 8(r/4) + 4g + r%4 of the page is visible iff 32kt + 8(r/4) + r%4 <= lim
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (32 * kt + 8 * (r / 4) + (r % 4) > lim) sc[kt][r] = neg_inf();
      }
      // page maximum of the lane's query: four max3 chains, then the other lane half
      float m0 = fmaxf(fmaxf(sc[0][0], sc[0][1]), sc[0][2]), m1 = fmaxf(fmaxf(sc[0][8], sc[0][9]), sc[0][10]);
      float m2 = fmaxf(fmaxf(sc[1][0], sc[1][1]), sc[1][2]), m3 = fmaxf(fmaxf(sc[1][8], sc[1][9]), sc[1][10]);
#pragma unroll
      for (int r = 3; r < 7; r += 2) {
        m0 = fmaxf(fmaxf(m0, sc[0][r]), sc[0][r + 1]);
        m1 = fmaxf(fmaxf(m1, sc[0][8 + r]), sc[0][9 + r]);
        m2 = fmaxf(fmaxf(m2, sc[1][r]), sc[1][r + 1]);
        m3 = fmaxf(fmaxf(m3, sc[1][8 + r]), sc[1][9 + r]);
      }
      m0 = fmaxf(fmaxf(m0, sc[0][7]), fmaxf(m1, sc[0][15]));
      m2 = fmaxf(fmaxf(m2, sc[1][7]), fmaxf(m3, sc[1][15]));
      const float mx = half_swap_max(fmaxf(m0, m2));  // page max of s - m
      // raise the running max on the first page, then only when a score
      // exceeds it by more than 2^kLazy (the weights stay below 2^kLazy)
      const bool raise = mx > kLazy || p == 0;
      if (__builtin_expect(__builtin_amdgcn_ballot_w64(raise) != 0, 0)) {
        if (raise) {
          const float m_new = (float)(_Float16)(m_run + mx);
          const float delta = m_new - m_run;  // exact: both are fp16 values
          const float alpha = p == 0 ? 0.f : __builtin_amdgcn_exp2f(-delta);
#pragma unroll
          for (int t = 0; t < kD / 32; ++t) oacc[t] *= alpha;
          l_lane *= alpha;
#pragma unroll
          for (int kt = 0; kt < 2; ++kt) sc[kt] -= delta;
          m_run = m_new;
        }
      }
      // one branch-free block: the second half's exponentials can issue
      // between the first half's value products
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        f16x8 pop[2];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            pop[u][e] = (_Float16)__builtin_amdgcn_exp2f(sc[kt][8 * u + e]);  // exp2(-inf) = 0
        // the normaliser sums the fp16 weights the value product uses, two per
        // v_dot2_f32_f16 against (1, 1) with fp32 accumulation
        const f16x2 ones = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int e = 0; e < 8; e += 2)
            l_lane = __builtin_amdgcn_fdot2(f16x2{pop[u][e], pop[u][e + 1]}, ones, l_lane, false);
#pragma unroll
        for (int t = 0; t < kD / 32; ++t)
#pragma unroll
          for (int u = 0; u < 2; ++u)
            oacc[t] = mfma_h(as_f16x8(vop[kt][t][u]), pop[u], oacc[t]);
      }
    }
    if (p + 1 < npages) store_page(buf ^ 1, buf ^ 1);
    __syncthreads();
  };
  for (int p = 0; p < npages; p += 2) {
    page(p, IntC<0>{});
    if (p + 1 < npages) page(p + 1, IntC<1>{});
  }

  // ---- epilogue: out = O / l + mu_v ----
  if (!wave_live) return;
  const float inv_l = 1.0f / half_swap_sum(l_lane);
  const bf16_t* muv = a.muv ? static_cast<const bf16_t*>(a.muv) + (size_t)h * kD : nullptr;
  const size_t orow = ((size_t)bh * M + myq) * kD;
  if (!q_ok) return;
#pragma unroll
  for (int t = 0; t < kD / 32; ++t) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i0 = 32 * t + 8 * c + 4 * g;
      const uint2 mw = muv ? *reinterpret_cast<const uint2*>(muv + i0) : make_uint2(0, 0);
      const float v0 = fmaf(oacc[t][4 * c + 0], inv_l, bf16_lo(mw.x));
      const float v1 = fmaf(oacc[t][4 * c + 1], inv_l, bf16_hi(mw.x));
      const float v2 = fmaf(oacc[t][4 * c + 2], inv_l, bf16_lo(mw.y));
      const float v3 = fmaf(oacc[t][4 * c + 3], inv_l, bf16_hi(mw.y));
      if (a.out_dtype == LLA_F32)
        *reinterpret_cast<float4*>(static_cast<float*>(a.out) + orow + i0) = make_float4(v0, v1, v2, v3);
      else
        *reinterpret_cast<uint2*>(static_cast<bf16_t*>(a.out) + orow + i0) = make_uint2(pack2(v0, v1), pack2(v2, v3));
    }
  }
}

template <int AXIS, int KS>
hipError_t launch_recon(const Prefill2dArgs& a, hipStream_t stream) {
  const dim3 grid((a.nk + kRTok - 1) / kRTok, a.B);
  hipLaunchKernelGGL((recon2d_kernel<AXIS, KS>), grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <int AXIS>
hipError_t launch_recon_r(const Prefill2dArgs& a, int r, hipStream_t stream) {
  switch (r / 16) {
#define LLA_R(ks) \
  case ks: return launch_recon<AXIS, ks>(a, stream);
    LLA_R(1) LLA_R(2) LLA_R(3) LLA_R(4) LLA_R(5) LLA_R(6) LLA_R(7) LLA_R(8)
    LLA_R(9) LLA_R(10) LLA_R(11) LLA_R(12) LLA_R(13) LLA_R(14) LLA_R(15) LLA_R(16)
    LLA_R(17) LLA_R(18) LLA_R(19) LLA_R(20) LLA_R(21) LLA_R(22) LLA_R(23) LLA_R(24)
    LLA_R(25) LLA_R(26) LLA_R(27) LLA_R(28) LLA_R(29) LLA_R(30) LLA_R(31) LLA_R(32)
#undef LLA_R
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

size_t prefill_2d_ws_bytes(int B, int H, int n_keys) {
  const size_t nk = ((size_t)n_keys + kPage - 1) / kPage * kPage;
  return 2 * (size_t)B * H * nk * kD * sizeof(bf16_t);
}

hipError_t launch_prefill_2d(const Prefill2dArgs& a, hipStream_t stream) {
  hipError_t e = launch_recon_r<0>(a, a.rk, stream);
  if (e != hipSuccess) return e;
  e = launch_recon_r<1>(a, a.rv, stream);
  if (e != hipSuccess) return e;
  const dim3 grid(a.B * a.H, (a.M + kQBlock - 1) / kQBlock);
  hipLaunchKernelGGL(flash2d_kernel, grid, dim3(kFThreads), 0, stream, a);
  return hipGetLastError();
}

template <int AXIS>
hipError_t launch_recon_ph(const Prefill2dArgs& a, int r, hipStream_t stream) {
  // pages per workgroup: about 2048 workgroups over the (b, h) pages, 1 to 8 pages each
  const int pages = a.nk / kPage;
  const long total = (long)pages * a.B * a.H;
  int ppw = (int)(total / 2048);
  ppw = ppw < 1 ? 1 : ppw > 8 ? 8 : ppw;
  const dim3 grid((pages + ppw - 1) / ppw, a.B * a.H);
  switch ((r + 15) / 16) {
#define LLA_R(ks) \
  case ks: hipLaunchKernelGGL((recon_ph_kernel<AXIS, ks>), grid, dim3(kThreads), 0, stream, a, ppw); break;
    LLA_R(1) LLA_R(2) LLA_R(3) LLA_R(4) LLA_R(5) LLA_R(6) LLA_R(7) LLA_R(8)
    LLA_R(9) LLA_R(10) LLA_R(11) LLA_R(12) LLA_R(13) LLA_R(14) LLA_R(15) LLA_R(16)
    LLA_R(17) LLA_R(18) LLA_R(19) LLA_R(20) LLA_R(21) LLA_R(22) LLA_R(23) LLA_R(24)
    LLA_R(25) LLA_R(26) LLA_R(27) LLA_R(28) LLA_R(29) LLA_R(30) LLA_R(31) LLA_R(32)
#undef LLA_R
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_prefill_rebuild(const Prefill2dArgs& a, hipStream_t stream) {
  hipError_t e = launch_recon_ph<0>(a, a.rk, stream);
  if (e != hipSuccess) return e;
  e = launch_recon_ph<1>(a, a.rv, stream);
  if (e != hipSuccess) return e;
  const dim3 grid(a.B * a.H, (a.M + kQBlock - 1) / kQBlock);
  hipLaunchKernelGGL(flash2d_kernel, grid, dim3(kFThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace lla
