// Causal prefill attention at loop l over the paged latent cache, bf16 inputs
// on MFMA, absorbed form (App. J "Absorbed attention"):
//   Q~ = Q U_k (scale * log2 e folded in),  S = Q~ C_k^T (key n <= query pos),
//   P = softmax(S) row-wise (online over 64-token pages),  Z = P C_v,
//   O = (Z / l) U_v^T + mu_v.
// The paper's two-pass decoder re-forwards the prompt with attention over the
// reconstructed cache (App. A); this kernel is that attention read straight
// from the latents.
//
// One workgroup = 8 wavefronts x 32 queries of one (b, h).  Every product is
// a v_mfma_f32_32x32x16_bf16 and is computed transposed so that each
// accumulator's registers feed the next product's B operand with no
// cross-lane movement:
//   D1 = Q~^T   (M = feature j, N = query, K = d)     A: U_k^T (LDS)      B: Q rows (global)
//   D2 = S^T    (M = key n,     N = query, K = j)     A: K tile (LDS, token-major)  B: D1 (fp16)
//   D3 = Z^T   += (M = j,       N = query, K = key)   A: V tile (LDS, feature-major) B: P from D2
//   D4 = O^T    (M = out i,     N = query, K = j)     A: U_v (LDS)        B: D3 / l
// A 32x32 accumulator gives lane (q + 32g), register r the element
// [8(r/4) + 4g + r%4][q]: every register of a lane belongs to the lane's
// query q, so the softmax state (running max, rescaling) is lane-local.  The
// K index of the next product is enumerated in that same order: K-step t,
// lane half g, element e stands for index 16t + 8(e/4) + 4g + e%4, which is
// exactly registers 8(t%2) + e of accumulator tile t/2.
// The denominator l comes out of the value product: the padded V tile carries
// a row of ones at feature r_v, so Z^T[r_v][q] = sum_n p[q][n].
// With the decoupled rotary branch (App. J), the rotary key rows follow the r_k
// content rows in the score tile and the rotated query part follows Q~'s, so
// the same products add q_r . k_r to every score.
// The score, value and output products run on v_mfma_f32_32x32x16_f16 (the
// bf16 rate): Q~, the softmax weights and Z / l enter them in fp16, and the
// key and value pages and U_v are converted from bf16 to fp16 (exact) as they
// are staged, so these intermediates keep 11 significant bits rather than
// bf16's 8, in one product per K-step (a two-term bf16 split of Q~ needs two).
// Latents or U_v entries beyond fp16's range (65504) would make the output
// non-finite.
// The running max enters the score product through a padding feature (S - m
// comes out of the MFMAs), and is only raised when a page exceeds it by more
// than 2^8 (lazy rescale), so most pages cost
// half a max3, one exp2 and half a packed conversion per score.  This file is
// compiled without NaN semantics: scores are either finite or -inf (masked),
// so max needs no NaN canonicalisation.
// K/V pages are staged cooperatively into double-buffered LDS tiles (the K
// page transposed to token-major on the way); the global loads of the two
// following pages are in flight while the current page is computed.

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kPWaves = 8;
constexpr int kPThreads = kPWaves * kWave;
constexpr int kQBlock = kPWaves * 32;  // queries per workgroup
constexpr int kMaxDPrefill = 128;
constexpr float kLazy = 8.0f;          // rescale only when the max grows by more than this (log2)
constexpr uint16_t kOneH = 0x3C00;     // 1.0 in fp16

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Raw buffer resource (gfx9 family word 3) over one contiguous region; loads
// take a per-lane offset and a wave-uniform (scalar) offset.
typedef __amdgpu_buffer_rsrc_t BufRsrc;
__device__ __forceinline__ BufRsrc make_rsrc(const void* base, size_t bytes) {
  const int n = bytes >= 0xffffffffull ? -1 : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}
__device__ __forceinline__ uint4 buf_ld16(BufRsrc r, int voff, int soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ uint16_t buf_ld2(BufRsrc r, int voff, int soff) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma_h(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ uint16_t f16_bits(float x) { return __builtin_bit_cast(uint16_t, (_Float16)x); }
// Two floats to two fp16 (round to nearest even) in one v_cvt_pk_f16_f32; written
// out because the compiler splits a packed conversion whose halves are stored
// separately back into two single conversions.
__device__ __forceinline__ uint32_t cvt_pk_f16(float lo, float hi) {
  uint32_t r;
  asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(r) : "v"(lo), "v"(hi));
  return r;
}

// A/B operand for K-step ordering 16t + 8(e/4) + 4g + e%4 read from an LDS row:
// elements [base + 4g .. +3] and [base + 8 + 4g .. +3].
__device__ __forceinline__ bf16x8 lds_pair(const bf16_t* row, int base, int g) {
  const uint2 lo = *reinterpret_cast<const uint2*>(row + base + 4 * g);
  const uint2 hi = *reinterpret_cast<const uint2*>(row + base + 8 + 4 * g);
  return as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
}

// Registers 8h..8h+7 of an accumulator, scaled, as a bf16 operand.
__device__ __forceinline__ bf16x8 to_operand(const f32x16& acc, int h, float scale) {
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (__bf16)(acc[8 * h + e] * scale);
  return o;
}

// The same in fp16 (11 significant bits).
__device__ __forceinline__ f16x8 to_operand_h(const f32x16& acc, int h, float scale) {
  f16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (_Float16)(acc[8 * h + e] * scale);
  return o;
}

// Waves per SIMD the register budget is sized for: the smallest tiles fit
// four (<= 128 VGPRs), the others two.
constexpr int prefill_occupancy(int rkp, int rvp) { return rkp + rvp <= 64 ? 4 : 2; }

// max over both halves of the wavefront (lane i and lane i ^ 32)
__device__ __forceinline__ float half_swap_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

template <int N>
struct IntC {
  static constexpr int value = N;
};

template <int RKP, int RVP>
__global__ __launch_bounds__(kPThreads) __attribute__((amdgpu_waves_per_eu(prefill_occupancy(RKP, RVP))))
void prefill_bf16_kernel(PrefillArgs a) {
  constexpr int KS = RKP / 16;        // K-steps of the score product (over features)
  constexpr int QT = RKP / 32;        // accumulator tiles of Q~^T
  constexpr int ZT = RVP / 32;        // accumulator tiles of Z^T
  constexpr int ZK = RVP / 16;        // K-steps of the output product
  constexpr int CKS = RKP + 4;        // token-major K tile row stride (elements)
  constexpr int CVS = kPage + 4;      // feature-major V tile row stride (elements)
  constexpr int UKS = kMaxDPrefill + 8;
  constexpr int UVS = RVP + 4;
  constexpr int KTILE = kPage * CKS, VTILE = RVP * CVS;

  __shared__ __attribute__((aligned(16))) bf16_t s_ukt[RKP * UKS];
  __shared__ __attribute__((aligned(16))) uint16_t s_uv[kMaxDPrefill * UVS];  // fp16
  __shared__ __attribute__((aligned(16))) uint16_t s_ck[2 * KTILE];  // fp16 key tiles
  __shared__ __attribute__((aligned(16))) uint16_t s_cv[2 * VTILE];  // fp16 value tiles

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane & 31, g = lane >> 5;
  const int bh = blockIdx.x;
  const int h = bh % a.H;
  const int nqb = (a.M + kQBlock - 1) / kQBlock;
  const int qb = nqb - 1 - (int)blockIdx.y;  // heaviest (latest) query blocks first
  const int d = a.d, rk = a.rk, rv = a.rv, M = a.M, p0 = a.p0;
  const int rke = rk + a.dr;  // score features: r_k content, then the rotary branch
  const int q0 = qb * kQBlock;
  const int qw0 = q0 + wave * 32;
  const int myq = qw0 + col;
  const bool q_ok = myq < M;
  const bool wave_live = qw0 < M;
  const int qlast_w = min(qw0 + 31, M - 1);                    // last query of this wave
  const int kmax = p0 + min(q0 + kQBlock, M);                  // keys [0, kmax) matter to the block
  const int npages = (kmax + kPage - 1) / kPage;

  // ---- constant LDS: U_k^T and U_v (zero padded), padding of the page tiles ----
  // K feature RKP - 1 is 1 for every key (it carries the running max, below);
  // K features r_k .. RKP - 2 are 0.  V row r_v is all ones (the denominator),
  // V rows past it are 0.
  // Thread (tj, ti) = (tid % 32, tid / 32) fills feature columns j = tj + 32 jj
  // and rows i = ti + TI k (TI = threads / 32) of U_k^T (transposed) and U_v; features past r are
  // zero.  The LDS offsets are compile-time apart, the global reads are buffer
  // loads with the row offset in a scalar register, and all of a column's
  // loads are issued before its stores.
  {
    const int tj = tid & 31, ti = tid >> 5;
    constexpr int TI = kPThreads / 32;  // row stride (d_head is a multiple of 32, so of TI)
    const BufRsrc uks = make_rsrc(static_cast<const bf16_t*>(a.uk) + (size_t)h * d * rk, (size_t)d * rk * 2);
    const BufRsrc uvs = make_rsrc(static_cast<const bf16_t*>(a.uv) + (size_t)h * d * rv, (size_t)d * rv * 2);
    constexpr int KR = kMaxDPrefill / TI;  // rows per thread
#pragma unroll
    for (int jj = 0; jj < RKP / 32; ++jj) {
      const int j = tj + 32 * jj;
      uint16_t w[KR];
#pragma unroll
      for (int k = 0; k < KR; ++k) w[k] = 0;
      if (j < rk) {
#pragma unroll
        for (int k = 0; k < KR; ++k)
          if (TI * k < d) w[k] = buf_ld2(uks, (ti * rk + j) * 2, __builtin_amdgcn_readfirstlane(TI * k * rk * 2));
      }
#pragma unroll
      for (int k = 0; k < KR; ++k)
        if (TI * k < d) s_ukt[j * UKS + ti + TI * k] = w[k];
    }
#pragma unroll
    for (int jj = 0; jj < RVP / 32; ++jj) {
      const int j = tj + 32 * jj;
      uint16_t w[KR];
#pragma unroll
      for (int k = 0; k < KR; ++k) w[k] = 0;
      if (j < rv) {
#pragma unroll
        for (int k = 0; k < KR; ++k)
          if (TI * k < d) w[k] = buf_ld2(uvs, (ti * rv + j) * 2, __builtin_amdgcn_readfirstlane(TI * k * rv * 2));
      }
#pragma unroll
      for (int k = 0; k < KR; ++k)
        if (TI * k < d) s_uv[(ti + TI * k) * UVS + j] = f16_bits(bf16_to_f32(w[k]));  // exact
    }
  }
  // page-tile padding of both buffers: K columns r_k..RKP-1 of every token row
  // (at most 32 of them, RKP - 32 <= r_k), V rows r_v..RVP-1 (16-byte stores)
  {
    const int n = tid & (kPage - 1);
    for (int j = rke + (tid >> 6); j < RKP; j += kPThreads / kPage) {
      const uint16_t v = (j == RKP - 1) ? kOneH : uint16_t(0);
      s_ck[n * CKS + j] = v;
      s_ck[KTILE + n * CKS + j] = v;
    }
  }
  for (int e = tid; e < 2 * 32 * 8; e += kPThreads) {
    const int buf = e >> 8, j = rv + ((e >> 3) & 31), n8 = e & 7;
    const uint32_t f = (j == rv) ? 0x3C003C00u : 0u;  // two fp16 ones, or zeros
    if (j < RVP) *reinterpret_cast<uint4*>(&s_cv[buf * VTILE + j * CVS + 8 * n8]) = make_uint4(f, f, f, f);
  }

  // ---- page staging ----
  // A page of one axis is r feature rows of 128 contiguous bytes, so chunk ch
  // (16 bytes, feature row ch/8, tokens 8(ch%8)..+7) sits at byte 16 ch of the
  // page: buffer loads with the page offset in a scalar register and a fixed
  // lane offset.  K chunks are transposed into the token-major tile on the way
  // (8 two-byte LDS stores); V chunks are copied into the feature-major tile.
  constexpr int CHK = ((RKP - 1) * 8 + kPThreads - 1) / kPThreads;  // r_k <= RKP - 1
  constexpr int CHV = ((RVP - 1) * 8 + kPThreads - 1) / kPThreads;  // r_v <= RVP - 1
  const size_t unit = (size_t)bh;
  const BufRsrc ksrc = make_rsrc(static_cast<const bf16_t*>(a.ck) + unit * (size_t)a.n_max * rk,
                                 (size_t)a.n_max * rk * 2);
  const BufRsrc vsrc = make_rsrc(static_cast<const bf16_t*>(a.cv) + unit * (size_t)a.n_max * rv,
                                 (size_t)a.n_max * rv * 2);
  const int kpage_b = kPage * rk * 2, vpage_b = kPage * rv * 2;
  const int nkch = rke * 8, nvch = rv * 8, ncch = rk * 8;  // K chunks: content, then rotary
  // rotary keys: chunk ch >= r_k * 8 is chunk ch - r_k * 8 of the rotary page
  // (feature row r_k + (ch - r_k * 8) / 8 of the score tile)
  const bool rope = a.dr > 0;
  const BufRsrc rsrc = make_rsrc(rope ? static_cast<const bf16_t*>(a.rc) +
                                            ((size_t)(bh / a.H) * a.Hr + (a.Hr == 1 ? 0 : h)) * (size_t)a.n_max * a.dr
                                      : static_cast<const bf16_t*>(a.ck),
                                 (size_t)a.n_max * a.dr * 2);
  const int rpage_b = kPage * a.dr * 2;
  int kdst[CHK], vdst[CHV];  // LDS element offsets of this thread's chunks inside a tile
#pragma unroll
  for (int c = 0; c < CHK; ++c) {
    const int ch = tid + c * kPThreads;
    kdst[c] = (ch & 7) * 8 * CKS + (ch >> 3);
  }
#pragma unroll
  for (int c = 0; c < CHV; ++c) {
    const int ch = tid + c * kPThreads;
    vdst[c] = (ch >> 3) * CVS + (ch & 7) * 8;
  }
  // Two register sets: page p + 2 is in flight while page p + 1 waits in
  // registers and page p is computed from LDS.  Every lane issues every load
  // (lanes past the last chunk re-read chunk 0 and drop it), so the wait for
  // one page never covers the next page's loads.
  uint4 stk[2][CHK], stv[2][CHV];
  auto load_page = [&](int pg, int set) {
#pragma unroll
    for (int c = 0; c < CHK; ++c) {
      const int ch = tid + c * kPThreads;
      stk[set][c] = buf_ld16(ksrc, ch < ncch ? ch * 16 : 0, __builtin_amdgcn_readfirstlane(pg * kpage_b));
      if (rope) {
        const uint4 w = buf_ld16(rsrc, ch >= ncch && ch < nkch ? (ch - ncch) * 16 : 0,
                                 __builtin_amdgcn_readfirstlane(pg * rpage_b));
        if (ch >= ncch) stk[set][c] = w;
      }
    }
#pragma unroll
    for (int c = 0; c < CHV; ++c) {
      const int ch = tid + c * kPThreads;
      stv[set][c] = buf_ld16(vsrc, ch < nvch ? ch * 16 : 0, __builtin_amdgcn_readfirstlane(pg * vpage_b));
    }
  };
  auto store_page = [&](int pg, int set, uint16_t* tk, uint16_t* tv) {
#pragma unroll
    for (int c = 0; c < CHK; ++c) {
      const int ch = tid + c * kPThreads;
      if (ch < nkch) {
        // keys: bf16 -> fp16 (exact within fp16's range), transposed to token-major
        float v[8];
        Elem<bf16_t>::unpack(stk[set][c], v);
        // packed conversions (round to nearest even); the high halves are stored
        // straight from the packed register
        uint16_t* dst = tk + kdst[c];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const uint32_t w = cvt_pk_f16(v[e], v[e + 1]);
          dst[e * CKS] = (uint16_t)w;
          dst[(e + 1) * CKS] = (uint16_t)(w >> 16);
        }
      }
    }
    const bool last = (pg + 1) * kPage > kmax;  // tokens past the last key are zeroed
#pragma unroll
    for (int c = 0; c < CHV; ++c) {
      const int ch = tid + c * kPThreads;
      if (ch < nvch) {
        uint4 w = stv[set][c];
        if (last) {
          // keep tokens n0 + e < kmax: dword i holds tokens 2i (low half) and 2i + 1
          const int nv = kmax - (pg * kPage + (ch & 7) * 8);
          auto keep = [nv](int i) {
            return nv > 2 * i + 1 ? 0xffffffffu : nv > 2 * i ? 0x0000ffffu : 0u;
          };
          w.x &= keep(0);
          w.y &= keep(1);
          w.z &= keep(2);
          w.w &= keep(3);
        }
        // bf16 -> fp16 (exact within fp16's range); masked tokens stay 0
        float x[8];
        Elem<bf16_t>::unpack(w, x);
        f16x8 hx;
#pragma unroll
        for (int e = 0; e < 8; ++e) hx[e] = (_Float16)x[e];
        const uint4 hw = __builtin_bit_cast(uint4, hx);
        uint16_t* dst = tv + vdst[c];
        *reinterpret_cast<uint2*>(dst) = make_uint2(hw.x, hw.y);
        *reinterpret_cast<uint2*>(dst + 4) = make_uint2(hw.z, hw.w);
      }
    }
  };

  load_page(0, 0);
  load_page(min(1, npages - 1), 1);
  __syncthreads();  // constant LDS written
  store_page(0, 0, s_ck, s_cv);

  // ---- D1 = Q~^T for this wave's 32 queries ----
  f16x8 qop[KS];  // Q~ in fp16
  {
    f32x16 d1[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) d1[t] = f32x16{0.f};
    const bf16_t* qrow = static_cast<const bf16_t*>(a.q) + (unit * M + (q_ok ? myq : 0)) * d;
    uint4 bq[kMaxDPrefill / 16];  // the whole query row in flight at once
#pragma unroll
    for (int s = 0; s < kMaxDPrefill / 16; ++s)
      bq[s] = (q_ok && s < d / 16) ? ld16(qrow + 16 * s + 8 * g) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int s = 0; s < kMaxDPrefill / 16; ++s) {
      if (s < d / 16) {
#pragma unroll
        for (int t = 0; t < QT; ++t) {
          const bf16x8 au = as_bf16x8(*reinterpret_cast<const uint4*>(&s_ukt[(32 * t + col) * UKS + 16 * s + 8 * g]));
          d1[t] = mfma(au, as_bf16x8(bq[s]), d1[t]);
        }
      }
    }
    if (rope && q_ok) {  // the (already rotated) rotary query part fills features r_k .. rke - 1
      const bf16_t* qrr = static_cast<const bf16_t*>(a.qr) + (unit * M + myq) * a.dr;
#pragma unroll
      for (int t = 0; t < QT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int f = 32 * t + 8 * (r / 4) + 4 * g + (r % 4);
          if (f >= rk && f < rke) d1[t][r] += bf16_to_f32(qrr[f - rk]);
        }
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qop[ks] = to_operand_h(d1[ks / 2], ks % 2, a.qscale);
  }
  __syncthreads();  // page 0 staged

  // ---- online softmax over the key pages ----
  // The running max rides in the score product itself: K feature RKP - 1 is 1
  // for every key and the same feature of Q~ (K-step KS - 1, element 7 of the
  // upper lane half) holds negm = -m in fp16, so the MFMAs yield S - m
  // directly.  negm is the exact value the product uses.
  f32x16 zacc[ZT];
#pragma unroll
  for (int t = 0; t < ZT; ++t) zacc[t] = f32x16{0.f};
  float negm = 0.f;
  const int qpos = p0 + myq;  // absolute position of this lane's query

  auto page = [&](int p, auto bufc) {
    constexpr int buf = decltype(bufc)::value;
    // set buf held page p, already in LDS; near the end the last page is
    // re-read rather than branching, so the wait below is always for one page
    load_page(min(p + 2, npages - 1), buf);
    const int key0 = p * kPage;
    if (wave_live && key0 <= p0 + qlast_w) {
      const bool diag = key0 + kPage - 1 > p0 + qw0;
      const uint16_t* ktile = s_ck + buf * KTILE + col * CKS;
      const bf16_t* vtile = reinterpret_cast<const bf16_t*>(s_cv) + buf * VTILE + col * CVS;  // fp16 bits
      // Both 32-key halves are scored up front (the second half's MFMAs run
      // while the first half's softmax is on the VALU); each half is then
      // its own online-softmax step.
      // All K operands of the page are read from LDS before the first score
      // MFMA, the V operands right after the last one: their latency is
      // covered by the MFMAs instead of stalling each product.
      f16x8 ak[2][KS];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          ak[kt][ks] = __builtin_bit_cast(f16x8, lds_pair(reinterpret_cast<const bf16_t*>(ktile) + 32 * kt * CKS,
                                                          16 * ks, g));
      __builtin_amdgcn_sched_barrier(0);
      f32x16 sc[2] = {f32x16{0.f}, f32x16{0.f}};
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          sc[kt] = mfma_h(ak[kt][ks], qop[ks], sc[kt]);
        }
      f16x8 av[ZT][4];
#pragma unroll
      for (int t = 0; t < ZT; ++t)
#pragma unroll
        for (int u = 0; u < 4; ++u) av[t][u] = __builtin_bit_cast(f16x8, lds_pair(vtile + 32 * t * CVS, 16 * u, g));
      __builtin_amdgcn_sched_barrier(0);
      const int lim = qpos - key0 - 4 * g;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        f32x16& v = sc[kt];
        if (__builtin_expect(diag, 0)) {
          // key 32kt + 8(r/4) + 4g + r%4 of the page is visible iff 32kt + 8(r/4) + r%4 <= lim
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (32 * kt + 8 * (r / 4) + (r % 4) > lim) v[r] = neg_inf();
        }
        // row max of the half: two max3 chains of eight scores
        float m0 = fmaxf(fmaxf(v[0], v[1]), v[2]), m1 = fmaxf(fmaxf(v[8], v[9]), v[10]);
        m0 = fmaxf(fmaxf(m0, v[3]), v[4]);
        m1 = fmaxf(fmaxf(m1, v[11]), v[12]);
        m0 = fmaxf(fmaxf(m0, v[5]), v[6]);
        m1 = fmaxf(fmaxf(m1, v[13]), v[14]);
        float mx = fmaxf(fmaxf(m0, v[7]), fmaxf(m1, v[15]));
        mx = half_swap_max(mx);
        // Raise the running max on the first half-page, and later only when a
        // score exceeds it by more than 2^kLazy.
        const bool first = (p == 0 && kt == 0);
        const bool raise = first || mx > kLazy;
        if (__builtin_expect(__builtin_amdgcn_ballot_w64(raise) != 0, 0)) {
          // new fold value -(m + mx) in fp16; lanes that do not raise keep theirs
          const _Float16 t16 = (_Float16)(negm - mx);
          const float delta = raise ? (float)t16 - negm : 0.f;
          if (!first) {
            const float alpha = __builtin_amdgcn_exp2f(delta);
#pragma unroll
            for (int t = 0; t < ZT; ++t) zacc[t] *= alpha;
          }
          // the scores not yet exponentiated were computed with the old fold
#pragma unroll
          for (int k2 = kt; k2 < 2; ++k2) sc[k2] += delta;
          negm += delta;
          const bool put = raise && g == 1;
          qop[KS - 1][7] = put ? t16 : qop[KS - 1][7];
        }
        // P as the value product's B operands: K-step u = registers 8(u%2).. of this half
        f16x8 pop[2];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int e = 0; e < 8; ++e) pop[u][e] = (_Float16)__builtin_amdgcn_exp2f(v[8 * u + e]);
#pragma unroll
        for (int t = 0; t < ZT; ++t)
#pragma unroll
          for (int u = 0; u < 2; ++u)
            zacc[t] = mfma_h(av[t][2 * kt + u], pop[u], zacc[t]);
      }
    }
    if (p + 1 < npages) store_page(p + 1, buf ^ 1, s_ck + (buf ^ 1) * KTILE, s_cv + (buf ^ 1) * VTILE);
    __syncthreads();
  };
  for (int p = 0; p < npages; p += 2) {
    page(p, IntC<0>{});
    if (p + 1 < npages) page(p + 1, IntC<1>{});
  }

  // ---- epilogue: l from the ones row, O^T = U_v (Z / l)^T + mu_v ----
  if (!wave_live) return;
  float lsum = 0.f;
  {
    const int t = rv / 32, rr = rv % 32;
    const int gl = (rr / 4) % 2, reg = 4 * (rr / 8) + rr % 4;
#pragma unroll
    for (int tt = 0; tt < ZT; ++tt)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (tt == t && r == reg && g == gl) lsum = zacc[tt][r];
    lsum += xor_shfl(lsum, 32);
  }
  const float inv_l = 1.0f / lsum;
  f16x8 zop[ZK];
#pragma unroll
  for (int ks = 0; ks < ZK; ++ks) zop[ks] = to_operand_h(zacc[ks / 2], ks % 2, inv_l);
  const bf16_t* muv = a.muv ? static_cast<const bf16_t*>(a.muv) + (size_t)h * d : nullptr;
  const size_t orow = (unit * M + myq) * (size_t)d;
  for (int it = 0; it < d / 32; ++it) {
    f32x16 o = f32x16{0.f};
    const bf16_t* urow = reinterpret_cast<const bf16_t*>(&s_uv[(32 * it + col) * UVS]);  // fp16 bits
#pragma unroll
    for (int ks = 0; ks < ZK; ++ks) o = mfma_h(__builtin_bit_cast(f16x8, lds_pair(urow, 16 * ks, g)), zop[ks], o);
    if (q_ok) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int i0 = 32 * it + 8 * c + 4 * g;
        const uint2 mw = muv ? *reinterpret_cast<const uint2*>(muv + i0) : make_uint2(0, 0);
        float v[4];
        v[0] = o[4 * c + 0] + bf16_lo(mw.x);
        v[1] = o[4 * c + 1] + bf16_hi(mw.x);
        v[2] = o[4 * c + 2] + bf16_lo(mw.y);
        v[3] = o[4 * c + 3] + bf16_hi(mw.y);
        if (a.out_dtype == LLA_F32) {
          *reinterpret_cast<float4*>(static_cast<float*>(a.out) + orow + i0) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          bf16_t* op = static_cast<bf16_t*>(a.out) + orow + i0;
#pragma unroll
          for (int e = 0; e < 4; ++e) op[e] = f32_to_bf16(v[e]);
        }
      }
    }
  }
}

template <int RKP, int RVP>
hipError_t launch_t(const PrefillArgs& a, hipStream_t stream) {
  const int nqb = (a.M + kQBlock - 1) / kQBlock;
  dim3 grid(a.B * a.H, nqb);
  hipLaunchKernelGGL((prefill_bf16_kernel<RKP, RVP>), grid, dim3(kPThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_prefill_bf16(const PrefillArgs& a, hipStream_t stream) {
  // K features padded past r_k + d_rope (room for the running-max feature
  // RKP - 1); V features padded past r_v (room for the ones row)
  const int rke = a.rk + a.dr;
  const int rkp = rke < 32 ? 32 : rke < 64 ? 64 : 96;
  const int rvp = a.rv < 32 ? 32 : a.rv < 64 ? 64 : 96;
  switch (rkp * 1000 + rvp) {
    case 32032: return launch_t<32, 32>(a, stream);
    case 32064: return launch_t<32, 64>(a, stream);
    case 32096: return launch_t<32, 96>(a, stream);
    case 64032: return launch_t<64, 32>(a, stream);
    case 64064: return launch_t<64, 64>(a, stream);
    case 64096: return launch_t<64, 96>(a, stream);
    case 96032: return launch_t<96, 32>(a, stream);
    case 96064: return launch_t<96, 64>(a, stream);
    default: return launch_t<96, 96>(a, stream);
  }
}

}  // namespace lla
