// LLA-2D decode (Sec. 3 "The LLA-2D variant (loop x head)"): one latent per
// token and layer reconstructs all H heads, so the H queries of a sequence
// share every latent read.  Absorbed form (App. J "Absorbed attention"), per
// head h of loop l:
//   q~_h = U_{k,l,h}^T q_h,  s_h[n] = q~_h . c_k[n],  p_h = softmax(s_h),
//   z_h = sum_n p_h[n] c_v[n],  o_h = U_{v,l,h} z_h + mu_{v,l,h}.
// Scores and values are two small-N GEMMs per page of 64 tokens (N = H = 16
// heads), on v_mfma_f32_16x16x32_bf16:
//   S^T [tokens x heads] = C_k [tokens x r_k] . Q~^T    A: 8 consecutive features of
//                                                        one token (token-major key cache)
//   Z^T [features x heads] += C_v^T [features x tokens] . P^T
//                                                        A: 8 consecutive tokens of one
//                                                        feature (paged feature-major values)
// so both operands load straight from the caches with 16-byte loads.  In a
// 16x16 accumulator lane (col + 16g) holds rows 4g..4g+3 of column col: the
// column is a head, so the running max and the rescale of Z are lane-local.
// Q~ enters as hi + lo bf16 terms (about 16 significant bits in the scores).
//
// Three launches: absorb (Q~ for every (b, h) into the workspace), scan (each
// workgroup one sequence and a range of pages; 4 wavefronts each score one
// 16-token tile of a page and each accumulate a quarter of Z's feature tiles;
// softmax partials to the workspace), merge (per (b, h): combine the partials,
// o = U_v z / l + mu_v).

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kHeads2d = 16;  // the N of every product: one column per head
constexpr int kScanWaves = 4;
constexpr float kLazy2d = 8.0f;  // raise the running max only when it grows by more than this (log2)

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

typedef __amdgpu_buffer_rsrc_t BufRsrc;
__device__ __forceinline__ BufRsrc make_rsrc(const void* base, size_t bytes) {
  const int n = bytes >= 0xffffffffull ? -1 : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}
__device__ __forceinline__ uint4 buf_ld16(BufRsrc r, int voff, int soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// ---- absorb: Q~[b][h][j] = qscale * sum_i U_k[h][i][j] q[b][h][i] ----
// One v_mfma_f32_32x32x16_bf16 chain per wavefront computes a 32 (features j)
// x 32 (sequences b) tile of Q~^T over K = d:  A = U_k^T (LDS, transposed on
// the way in), B = q rows (16-byte global loads).  A 32x32 accumulator gives
// lane (c + 32 g), register r the element [8 (r/4) + 4 g + r%4][c], so each
// lane stores runs of 4 consecutive features of one sequence.  Outputs are
// stored as hi and lo bf16 terms ([B][2][H][r_k]), the form the scan takes.
// grid (H, ceil(r_k / 128), ceil(B / 32)); wavefront w covers features
// 128 blockIdx.y + 32 w.
typedef float f32x16 __attribute__((ext_vector_type(16)));
template <int N>
struct KSteps {
  static constexpr int value = N;
};
constexpr int kAbsJ = 128, kAbsB = 32;
__global__ __launch_bounds__(256) void absorb2d_kernel(Decode2dArgs a) {
  constexpr int US = kMaxHead + 8;  // transposed U_k row stride (bf16)
  __shared__ __attribute__((aligned(16))) bf16_t s_ut[kAbsJ * US];
  const int h = blockIdx.x, j0 = blockIdx.y * kAbsJ, b0 = blockIdx.z * kAbsB;
  const int d = a.d, rk = a.rk, nj = min(kAbsJ, rk - j0);  // nj: a multiple of 32
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int c = lane & 31, g = lane >> 5;
  const bf16_t* uk = static_cast<const bf16_t*>(a.uk) + (size_t)h * d * rk + j0;
  const bf16_t* qrow = static_cast<const bf16_t*>(a.q) + ((size_t)(b0 + c) * a.H + h) * d;
  const bool q_ok = b0 + c < a.B;
  // U_k[h][2p .. 2p+1][j0 + 8c .. +7] -> s_ut[8c + x][2p .. 2p+1] as one dword per
  // x; item e = (c, p) with p fastest, so a wavefront's LDS writes fall on
  // consecutive dwords.  All loads first.
  constexpr int kU = kMaxHead / 2 * kAbsJ / 8 / 256;
  const int np = d / 2, nitems = np * (nj / 8);
  uint4 xu[kU][2];
#pragma unroll
  for (int k = 0; k < kU; ++k) {
    const int e = tid + 256 * k, c = e / np, p = e - c * np;
    const bf16_t* src = uk + (size_t)(2 * p) * rk + 8 * c;
    xu[k][0] = e < nitems ? *reinterpret_cast<const uint4*>(src) : uint4{0, 0, 0, 0};
    xu[k][1] = e < nitems ? *reinterpret_cast<const uint4*>(src + rk) : uint4{0, 0, 0, 0};
  }
  uint4 xq[kMaxHead / 16];  // B fragments: q[b][16 t + 8 g .. +7]
#pragma unroll
  for (int t = 0; t < kMaxHead / 16; ++t)
    xq[t] = (q_ok && 16 * t < d) ? *reinterpret_cast<const uint4*>(qrow + 16 * t + 8 * g) : uint4{0, 0, 0, 0};
#pragma unroll
  for (int k = 0; k < kU; ++k) {
    const int e = tid + 256 * k, c = e / np, p = e - c * np;
    if (e < nitems) {
      const uint32_t r0[4] = {xu[k][0].x, xu[k][0].y, xu[k][0].z, xu[k][0].w};
      const uint32_t r1[4] = {xu[k][1].x, xu[k][1].y, xu[k][1].z, xu[k][1].w};
      uint32_t* dst = reinterpret_cast<uint32_t*>(s_ut) + (8 * c) * (US / 2) + p;
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        dst[(2 * x) * (US / 2)] = (r0[x] & 0xffffu) | (r1[x] << 16);
        dst[(2 * x + 1) * (US / 2)] = (r0[x] >> 16) | (r1[x] & 0xffff0000u);
      }
    }
  }
  __syncthreads();
  if (32 * wave >= nj) return;
  f32x16 acc = f32x16{0.f};
  const bf16_t* ua = &s_ut[(32 * wave + c) * US + 8 * g];
  // the K-step count as a compile-time parameter (d / 16, dispatched once), so
  // the chain has no branch per product
  auto chain = [&](auto ktc) {
    constexpr int KT = decltype(ktc)::value;
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(ua + 16 * t));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, __builtin_bit_cast(bf16x8, xq[t]), acc, 0, 0, 0);
    }
  };
  switch (d / 32) {  // d_head: a multiple of 32 up to 256
    case 1: chain(KSteps<2>{}); break;
    case 2: chain(KSteps<4>{}); break;
    case 3: chain(KSteps<6>{}); break;
    case 4: chain(KSteps<8>{}); break;
    case 5: chain(KSteps<10>{}); break;
    case 6: chain(KSteps<12>{}); break;
    case 7: chain(KSteps<14>{}); break;
    default: chain(KSteps<16>{}); break;
  }
  if (!q_ok) return;
  const size_t plane = (size_t)kHeads2d * rk;
  bf16_t* out = a.qt + (size_t)(b0 + c) * 2 * plane + (size_t)h * rk + j0 + 32 * wave + 4 * g;
#pragma unroll
  for (int m = 0; m < 4; ++m) {  // registers 4m .. 4m+3: features 8m + 4g .. +3
    uint32_t hi[2], lo[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const float x0 = acc[4 * m + 2 * e] * a.qscale, x1 = acc[4 * m + 2 * e + 1] * a.qscale;
      const __bf16 h0 = (__bf16)x0, h1 = (__bf16)x1;
      hi[e] = (uint32_t)__builtin_bit_cast(bf16_t, h0) | ((uint32_t)__builtin_bit_cast(bf16_t, h1) << 16);
      lo[e] = (uint32_t)__builtin_bit_cast(bf16_t, (__bf16)(x0 - (float)h0)) |
              ((uint32_t)__builtin_bit_cast(bf16_t, (__bf16)(x1 - (float)h1)) << 16);
    }
    *reinterpret_cast<uint2*>(out + 8 * m) = uint2{hi[0], hi[1]};
    *reinterpret_cast<uint2*>(out + plane + 8 * m) = uint2{lo[0], lo[1]};
  }
}

// ---- scan: one sequence b, pages [pb, pe); partials (m, l, z) per head ----
// Two page streams per workgroup: wavefronts 4 s .. 4 s + 3 (stream s) take the
// pages pb + s, pb + s + 2, ...; each stream keeps its own softmax state and
// the two are combined on chip at the end, so a split costs one partial.
// VT: value feature tiles (16 features each) per wavefront; KS: score K-steps of 32 features.
constexpr int kStreams = 2;
constexpr int kScanThreads = kStreams * kScanWaves * kWave;
template <int KS, int VT>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(2)))
void scan2d_kernel(Decode2dArgs a) {
  constexpr int PS = kPage + 8;  // P row stride (bf16): [head][token]
  constexpr int QS = KS * 32 + 8;  // Q~ row stride (bf16): rows hi 0..15, lo 16..31
  // Q~ during the loop; stream 1's z tiles for the final combine afterwards
  constexpr int kQBytes = 2 * kHeads2d * QS * 2, kXBytes = kScanWaves * VT * 4 * kWave * 4;
  __shared__ __attribute__((aligned(16))) char s_raw[kQBytes > kXBytes ? kQBytes : kXBytes];
  __shared__ __attribute__((aligned(16))) bf16_t s_p[kStreams][2][kHeads2d * PS];
  __shared__ float s_max[kStreams][kScanWaves][kHeads2d];
  __shared__ float s_l[kStreams][kScanWaves][kHeads2d];
  __shared__ float s_m1[kHeads2d];
  bf16_t* s_q = reinterpret_cast<bf16_t*>(s_raw);

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int stream = wave / kScanWaves, sw = wave % kScanWaves;  // stream, wavefront in it
  const int col = lane & 15, g = lane >> 4;  // col: token row (A) / head column (B, D)
  const int split = blockIdx.x, b = blockIdx.y;
  const int rk = a.rk, rv = a.rv;
  const int N = a.ctx_len ? a.ctx_len[b] : a.n_ctx;
  const bool bad = (N < 1) || (N > a.n_ctx);
  const int pages = bad ? 0 : (N + kPage - 1) / kPage;
  const int per = (pages + a.splits - 1) / a.splits;
  const int pb = min(pages, split * per), pe = min(pages, pb + per);

  // key rows: token-major [n_max][r_k]; value pages: [n_max/64][r_v][64]
  const BufRsrc ksrc = make_rsrc(static_cast<const bf16_t*>(a.ck) + (size_t)b * a.n_max * rk,
                                 (size_t)a.n_max * rk * 2);
  const BufRsrc vsrc = make_rsrc(static_cast<const bf16_t*>(a.cv) + (size_t)b * a.n_max * rv,
                                 (size_t)a.n_max * rv * 2);
  const int vtiles = rv / 16;
  // A fragments: keys of token 16*sw + col, features 32 s + 8 g; values of
  // feature 16 t + col, tokens 32 u + 8 g.  The per-lane part of each address is
  // one register; the step, tile and page parts are uniform (scalar offset).
  const int k_lane = ((sw * 16 + col) * rk + 8 * g) * 2;
  const int v_lane = (col * kPage + 8 * g) * 2;
  const int ks = rk / 32;  // K-steps in use (r_k is a multiple of 32)
  // every lane issues every load (steps past r_k re-read the last one and are
  // not multiplied), so the waits count loads exactly
  auto kload = [&](uint4 (&kf)[KS], int page) {
#pragma unroll
    for (int s = 0; s < KS; ++s)
      kf[s] = buf_ld16(ksrc, k_lane, __builtin_amdgcn_readfirstlane(page * kPage * rk * 2 + min(s, ks - 1) * 64));
  };
  auto vload = [&](uint4 (&vf)[VT][2], int page) {
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      const int tile = min(sw + kScanWaves * t, vtiles - 1);  // tiles past r_v re-read the last one
      const int soff = __builtin_amdgcn_readfirstlane((page * rv + tile * 16) * kPage * 2);
#pragma unroll
      for (int u = 0; u < 2; ++u) vf[t][u] = buf_ld16(vsrc, v_lane + 64 * u, soff);
    }
  };
  // The first page's loads go out before Q~ is staged (they do not depend on
  // it); afterwards a page's keys are requested as soon as the previous
  // page's scores have consumed the key registers, its values once the
  // previous page's value products are issued.
  uint4 kf[KS], vf[VT][2];
  if (pb + stream < pe) {
    kload(kf, pb + stream);
    vload(vf, pb + stream);
  }

  // Q~ of the 16 heads (hi and lo planes from the absorb launch) -> LDS
  {
    constexpr int kPer = (4 * KS * 32 + kScanThreads - 1) / kScanThreads;
    const int row8 = rk / 8, n16 = 4 * rk;  // 16-byte chunks: per row, in all 32 rows
    const uint4* src = reinterpret_cast<const uint4*>(a.qt + (size_t)b * 2 * kHeads2d * rk);
    uint4 x[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = tid + k * kScanThreads;
      x[k] = e < n16 ? src[e] : uint4{0, 0, 0, 0};
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = tid + k * kScanThreads;
      if (e < n16) {
        const int row = e / row8;
        *reinterpret_cast<uint4*>(&s_q[row * QS + 8 * (e - row * row8)]) = x[k];
      }
    }
    // zero columns r_k .. 32 KS - 1 (the unused K-steps multiply them)
    const int pad8 = (KS * 32 - rk) / 8;
    for (int e = tid; e < 2 * kHeads2d * pad8; e += kScanThreads) {
      const int row = e / pad8;
      *reinterpret_cast<uint4*>(&s_q[row * QS + rk + 8 * (e - row * pad8)]) = uint4{0, 0, 0, 0};
    }
  }
  __syncthreads();

  f32x4 zacc[VT];
#pragma unroll
  for (int t = 0; t < VT; ++t) zacc[t] = f32x4{0.f};
  float m_run = neg_inf(), l_run = 0.f;  // of head `col` (same in all 4 lane groups)

  // One page in flight per wavefront; the other stream covers part of the
  // latency.  A stream without a page this round still meets the barriers.
  int pbuf = 0;
  const int rounds = (pe - pb + kStreams - 1) / kStreams;
  for (int it = 0; it < rounds; ++it) {
    const int p = pb + kStreams * it + stream;
    const bool act = p < pe;  // uniform over the stream
    const bool more = p + kStreams < pe;
    f32x4 sc = f32x4{0.f};
    if (act) {
      // ---- S^T tile: tokens 16 sw .. +15 of the page x 16 heads ----
      int qo = col * QS + 8 * g;
      asm volatile("" : "+v"(qo));  // re-read Q~ from LDS every page rather than pin it in registers
#pragma unroll
      for (int s = 0; s < KS; ++s) {  // steps past r_k meet zero Q~ columns: no branch
        const bf16x8 bq = as_bf16x8(*reinterpret_cast<const uint4*>(&s_q[qo + 32 * s]));
        const bf16x8 bl = as_bf16x8(*reinterpret_cast<const uint4*>(&s_q[qo + kHeads2d * QS + 32 * s]));
        sc = mfma16(as_bf16x8(kf[s]), bq, sc);
        sc = mfma16(as_bf16x8(kf[s]), bl, sc);
      }
      if (more) kload(kf, p + kStreams);
      // tokens beyond the context (the last page) score -inf
      const int tok0 = p * kPage + sw * 16 + 4 * g;
      float mx = neg_inf();
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (tok0 + r >= N) sc[r] = neg_inf();
        mx = fmaxf(mx, sc[r]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      if (lane < 16) s_max[stream][sw][col] = mx;
    }
    __syncthreads();
    if (act) {
      const float pm = fmaxf(fmaxf(s_max[stream][0][col], s_max[stream][1][col]),
                             fmaxf(s_max[stream][2][col], s_max[stream][3][col]));
      // lazy running max: raised on the first page and when the page exceeds it by > 2^kLazy2d
      if (m_run == neg_inf() || pm > m_run + kLazy2d) {
        const float alpha = m_run == neg_inf() ? 0.f : __builtin_amdgcn_exp2f(m_run - pm);
        l_run *= alpha;
#pragma unroll
        for (int t = 0; t < VT; ++t) zacc[t] *= alpha;
        m_run = pm;
      }
      float pr[4], ls = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pr[r] = __builtin_amdgcn_exp2f(sc[r] - m_run);
        ls += pr[r];
      }
      ls += __shfl_xor(ls, 16, kWave);
      ls += __shfl_xor(ls, 32, kWave);
      l_run += ls;  // this wave's 16 tokens; the waves' sums are added at the end
      uint2 w;
      w.x = (uint32_t)__builtin_bit_cast(bf16_t, (__bf16)pr[0]) | ((uint32_t)__builtin_bit_cast(bf16_t, (__bf16)pr[1]) << 16);
      w.y = (uint32_t)__builtin_bit_cast(bf16_t, (__bf16)pr[2]) | ((uint32_t)__builtin_bit_cast(bf16_t, (__bf16)pr[3]) << 16);
      *reinterpret_cast<uint2*>(&s_p[stream][pbuf][col * PS + sw * 16 + 4 * g]) = w;
    }
    __syncthreads();
    if (act) {
      // ---- Z^T += C_v^T P^T for this wave's feature tiles ----
      // Branch-free: value slots past the context may hold anything, so the
      // tokens at or beyond N are masked to zero (all-ones masks before the
      // last page); tiles past r_v are multiplied too and never stored.
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const bf16x8 bp = as_bf16x8(*reinterpret_cast<const uint4*>(&s_p[stream][pbuf][col * PS + 32 * u + 8 * g]));
        const int nv = N - (p * kPage + 32 * u + 8 * g);
        uint32_t keep[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) keep[i] = nv > 2 * i + 1 ? 0xffffffffu : nv > 2 * i ? 0x0000ffffu : 0u;
#pragma unroll
        for (int t = 0; t < VT; ++t) {
          const uint4 v = uint4{vf[t][u].x & keep[0], vf[t][u].y & keep[1], vf[t][u].z & keep[2], vf[t][u].w & keep[3]};
          zacc[t] = mfma16(as_bf16x8(v), bp, zacc[t]);
        }
      }
      if (more) vload(vf, p + kStreams);
    }
    pbuf ^= 1;
  }

  // ---- combine the two streams, then the partial (m, l, z) of this split ----
  if (lane < 16) s_l[stream][sw][col] = l_run;
  __syncthreads();  // every wave is past its last read of Q~: s_raw now holds stream 1's tiles
  float* s_x = reinterpret_cast<float*>(s_raw);
  if (stream == 1) {
#pragma unroll
    for (int t = 0; t < VT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) s_x[((sw * VT + t) * 4 + r) * kWave + lane] = zacc[t][r];
    if (sw == 0 && lane < 16) s_m1[col] = m_run;
  }
  __syncthreads();
  if (stream == 1) return;
  const float m1 = s_m1[col], mm = fmaxf(m_run, m1);
  const float w0 = m_run == neg_inf() ? 0.f : __builtin_amdgcn_exp2f(m_run - mm);
  const float w1 = m1 == neg_inf() ? 0.f : __builtin_amdgcn_exp2f(m1 - mm);
  const size_t pbase = (((size_t)b * a.splits + split) * kHeads2d + col) * (size_t)(rv + 2);
  if (sw == 0 && lane < 16) {
    a.part[pbase] = mm;
    a.part[pbase + 1] = w0 * (s_l[0][0][col] + s_l[0][1][col] + s_l[0][2][col] + s_l[0][3][col]) +
                        w1 * (s_l[1][0][col] + s_l[1][1][col] + s_l[1][2][col] + s_l[1][3][col]);
  }
#pragma unroll
  for (int t = 0; t < VT; ++t) {
    const int tile = sw + kScanWaves * t;
    if (tile < vtiles) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        a.part[pbase + 2 + tile * 16 + 4 * g + r] = w0 * zacc[t][r] + w1 * s_x[((sw * VT + t) * 4 + r) * kWave + lane];
    }
  }
}

// ---- merge: per (head h, two sequences), combine the splits and apply U_v ----
// The loads that depend on nothing (the U_v rows this thread multiplies, the
// split statistics, the z partials) are all issued first, so a workgroup pays
// about one memory latency; U_v is read once for both sequences.
// U_v layout over a wavefront: lane (r8 = lane / 8, c8 = lane % 8) takes rows
// 8 (wave + 4 k) + r8 and 16-byte chunks c8 + 8 m, so one load instruction
// reads 8 whole 128-byte row segments; the 8 lanes of a row add their parts
// with three shuffles.  z feature tid + 256 m.
constexpr int kMergeB = 1;   // sequences per workgroup
constexpr int kMergeR = 4;   // U_v rows per thread held (d <= 128)
constexpr int kMergeC = 8;   // U_v chunks per row and thread held (r_v <= 512)
constexpr int kMergeM = 2;   // z features per thread held (r_v <= 512)
constexpr int kMergeS = 16;  // splits held
__global__ __launch_bounds__(256) void merge2d_kernel(Decode2dArgs a) {
  __shared__ float s_z[kMergeB][LLA_MAX_RANK_2D];
  __shared__ float s_w[kMergeB][LLA_MAX_SPLITS];
  __shared__ float s_inv[kMergeB];
  const int h = blockIdx.x, b0 = blockIdx.y * kMergeB, rv = a.rv, d = a.d, S = a.splits;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int nb = min(kMergeB, a.B - b0);
  const size_t sstride = (size_t)kHeads2d * (rv + 2);
  auto part_of = [&](int bb) { return a.part + ((size_t)(b0 + bb) * S * kHeads2d + h) * (size_t)(rv + 2); };
  const bf16_t* uv = static_cast<const bf16_t*>(a.uv) + (size_t)h * d * rv;
  const int n8 = rv / 8, r8 = lane >> 3, c8 = lane & 7;
  auto row_of = [&](int k) { return 8 * (wave + 4 * k) + r8; };
  // 1) U_v chunks
  uint4 w[kMergeR][kMergeC];
#pragma unroll
  for (int k = 0; k < kMergeR; ++k)
#pragma unroll
    for (int m = 0; m < kMergeC; ++m) {
      const int row = row_of(k), cj = c8 + 8 * m;
      w[k][m] = (row < d && cj < n8) ? *reinterpret_cast<const uint4*>(uv + (size_t)row * rv + 8 * cj)
                                     : uint4{0, 0, 0, 0};
    }
  // 2) split statistics: wave bb, lane s
  float ms = neg_inf(), ls = 0.f;
  if (wave < nb && lane < S) {
    ms = part_of(wave)[lane * sstride];
    ls = part_of(wave)[lane * sstride + 1];
  }
  // 3) z partials
  float zp[kMergeB][kMergeM][kMergeS];
#pragma unroll
  for (int bb = 0; bb < kMergeB; ++bb)
#pragma unroll
    for (int m = 0; m < kMergeM; ++m)
#pragma unroll
      for (int s = 0; s < kMergeS; ++s) {
        const int j = tid + 256 * m;
        zp[bb][m][s] = (bb < nb && j < rv && s < S) ? part_of(bb)[s * sstride + 2 + j] : 0.f;
      }
  const bf16_t* muv = a.muv ? static_cast<const bf16_t*>(a.muv) + (size_t)h * d : nullptr;

  // split weights of sequence `wave` (one wavefront each)
  if (wave < nb) {
    float m = ms;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) m = fmaxf(m, __shfl_xor(m, off, kWave));
    const float wt = ms == neg_inf() ? 0.f : __builtin_amdgcn_exp2f(ms - m);
    float l = wt * ls;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) l += __shfl_xor(l, off, kWave);
    if (lane < S) s_w[wave][lane] = wt;
    if (lane == 0) s_inv[wave] = 1.0f / l;
  }
  __syncthreads();
#pragma unroll
  for (int bb = 0; bb < kMergeB; ++bb) {
    if (bb >= nb) break;
#pragma unroll
    for (int m = 0; m < kMergeM; ++m) {
      const int j = tid + 256 * m;
      float z = 0.f;
#pragma unroll
      for (int s = 0; s < kMergeS; ++s)
        if (s < S) z = fmaf(s_w[bb][s], zp[bb][m][s], z);
      for (int s = kMergeS; s < S; ++s)
        if (j < rv) z = fmaf(s_w[bb][s], part_of(bb)[s * sstride + 2 + j], z);
      if (j < rv) s_z[bb][j] = z * s_inv[bb];
    }
    for (int j = tid + 256 * kMergeM; j < rv; j += 256) {  // r_v > 512
      float z = 0.f;
      for (int s = 0; s < S; ++s) z = fmaf(s_w[bb][s], part_of(bb)[s * sstride + 2 + j], z);
      s_z[bb][j] = z * s_inv[bb];
    }
  }
  __syncthreads();
  // o[b][row] = sum_j U_v[row][j] z[b][j] (+ mu_v)
  auto fma8 = [&](float (&acc)[kMergeB], uint4 v, int cj) {
#pragma unroll
    for (int bb = 0; bb < kMergeB; ++bb) {
      const float* z = &s_z[bb][8 * cj];
      float x = acc[bb];
      x = fmaf(bf16_lo(v.x), z[0], x);
      x = fmaf(bf16_hi(v.x), z[1], x);
      x = fmaf(bf16_lo(v.y), z[2], x);
      x = fmaf(bf16_hi(v.y), z[3], x);
      x = fmaf(bf16_lo(v.z), z[4], x);
      x = fmaf(bf16_hi(v.z), z[5], x);
      x = fmaf(bf16_lo(v.w), z[6], x);
      x = fmaf(bf16_hi(v.w), z[7], x);
      acc[bb] = x;
    }
  };
  auto finish = [&](float (&acc)[kMergeB], int row) {
#pragma unroll
    for (int bb = 0; bb < kMergeB; ++bb) {
      float x = acc[bb];
      x += __shfl_xor(x, 1, kWave);
      x += __shfl_xor(x, 2, kWave);
      x += __shfl_xor(x, 4, kWave);
      if (row < d && c8 == 0 && bb < nb) {
        const int b = b0 + bb;
        const int N = a.ctx_len ? a.ctx_len[b] : a.n_ctx;
        float v = x + (muv ? bf16_to_f32(muv[row]) : 0.f);
        if (N < 1 || N > a.n_ctx) v = __builtin_nanf("");
        const size_t o = ((size_t)b * a.H + h) * d + row;
        if (a.out_dtype == LLA_F32)
          static_cast<float*>(a.out)[o] = v;
        else
          static_cast<bf16_t*>(a.out)[o] = f32_to_bf16(v);
      }
    }
  };
#pragma unroll
  for (int k = 0; k < kMergeR; ++k) {
    const int row = row_of(k);
    if (8 * (wave + 4 * k) >= d) break;  // uniform
    float acc[kMergeB] = {};
#pragma unroll
    for (int m = 0; m < kMergeC; ++m)
      if (c8 + 8 * m < n8) fma8(acc, w[k][m], c8 + 8 * m);
    for (int cj = c8 + 8 * kMergeC; cj < n8; cj += 8)  // r_v > 512
      if (row < d) fma8(acc, *reinterpret_cast<const uint4*>(uv + (size_t)row * rv + 8 * cj), cj);
    finish(acc, row);
  }
  for (int k = kMergeR; 8 * (wave + 4 * k) < d; ++k) {  // d > 128
    const int row = row_of(k);
    float acc[kMergeB] = {};
    for (int cj = c8; cj < n8; cj += 8)
      if (row < d) fma8(acc, *reinterpret_cast<const uint4*>(uv + (size_t)row * rv + 8 * cj), cj);
    finish(acc, row);
  }
}

template <int KS, int VT>
void launch_scan(const Decode2dArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((scan2d_kernel<KS, VT>), dim3(a.splits, a.B), dim3(kScanThreads), 0, stream, a);
}

}  // namespace

int decode_2d_splits(int B, int n_ctx) {
  const int pages = (n_ctx + kPage - 1) / kPage;
  int s = (device_cu_count() + B - 1) / B;  // about one (two-stream) workgroup per compute unit
  if (s > pages) s = pages;
  if (s > LLA_MAX_SPLITS) s = LLA_MAX_SPLITS;
  return s < 1 ? 1 : s;
}

hipError_t launch_decode_2d(const Decode2dArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(absorb2d_kernel, dim3(a.H, (a.rk + kAbsJ - 1) / kAbsJ, (a.B + kAbsB - 1) / kAbsB),
                     dim3(256), 0, stream, a);
  // K-steps of 32 key features; value tiles of 16 features spread over the 4 wavefronts
  const int ks = a.rk / 32, vt = (a.rv / 16 + kScanWaves - 1) / kScanWaves;
  const int vtb = vt <= 2 ? 2 : vt <= 4 ? 4 : vt <= 8 ? 8 : 16;
  const int ksb = ks <= 4 ? 4 : ks <= 8 ? 8 : ks == 9 ? 9 : ks <= 12 ? 12 : ks <= 16 ? 16 : 32;
#define LLA_SCAN(K, V) \
  if (ksb == K && vtb == V) launch_scan<K, V>(a, stream);
  LLA_SCAN(4, 2) LLA_SCAN(4, 4) LLA_SCAN(4, 8) LLA_SCAN(4, 16)
  LLA_SCAN(8, 2) LLA_SCAN(8, 4) LLA_SCAN(8, 8) LLA_SCAN(8, 16)
  LLA_SCAN(9, 2) LLA_SCAN(9, 4) LLA_SCAN(9, 8) LLA_SCAN(9, 16)
  LLA_SCAN(12, 2) LLA_SCAN(12, 4) LLA_SCAN(12, 8) LLA_SCAN(12, 16)
  LLA_SCAN(16, 2) LLA_SCAN(16, 4) LLA_SCAN(16, 8) LLA_SCAN(16, 16)
  LLA_SCAN(32, 2) LLA_SCAN(32, 4) LLA_SCAN(32, 8) LLA_SCAN(32, 16)
#undef LLA_SCAN
  hipLaunchKernelGGL(merge2d_kernel, dim3(a.H, (a.B + kMergeB - 1) / kMergeB), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace lla
