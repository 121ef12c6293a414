// Loop-l decode attention over the paged latent cache, absorbed form
// (App. J "Absorbed attention"): scores q~ . c_k[n] with q~ = U_k^T q, online
// softmax, z = sum_n a_n c_v[n], out = U_v z + mu_v.  K and V are never
// materialised.
//
// The pass is HBM-bound (about one flop per latent byte), so the kernel is
// built around the load stream.  A cache page holds 64 tokens feature-major:
// one feature row of the page is 128 contiguous bytes (bf16), and one 16-byte
// load covers EPL = 8 consecutive tokens of one feature.  A wavefront works on
// groups of PPG = 8 pages (512 tokens):
//   * K phase -- lane (pg, ts) owns tokens ts*8..ts*8+7 of page pg of the
//     group and walks every feature row j, accumulating q~_j * c_k[j][tokens]
//     (q~_j is an LDS broadcast).  Each wave-wide load reads one 128-byte row
//     segment of each of the 8 pages; the lane ends with 8 complete scores,
//     so no cross-lane reduction and no redundant exp is needed.
//   * softmax -- one wave-wide max per group, running max m and sum l; the z
//     accumulators are rescaled only when m grows.
//   * V phase -- the probabilities go through a per-wave LDS buffer, and lane
//     (rg, ts) owns feature rows j = k*8 + rg and token slice ts of each page:
//     zacc[k] += sum over its 8 tokens of p_n c_v[j][n]; the reduction over
//     token slices is deferred to the end of the scan.
// Fewer 8-page groups than wavefronts (HALF: short contexts, and contexts
// split over many workgroups): the K phase takes groups of 4 pages and each
// wave-wide load covers two feature rows (lanes 32..63 take the odd row); one
// lane swap then sums the two halves of every score.  All wavefronts stream
// with full 16-byte loads, and a group's K phase has half as many dependent
// load batches.
// The waves of a workgroup interleave groups and merge their (m, l, z) in LDS.
// When the context is split over several workgroups (split-K), each writes its
// merged partial to the workspace and the last to arrive (an agent-scope
// atomic counter, one L2 write-back per workgroup) merges all partials and
// runs the value epilogue out = U_v (z / l) + mu_v; the counter is left at
// zero.
//
// With the decoupled rotary branch (App. J: a small explicit rotary key per
// token, shared across loops), the rotated query part joins q~ and the rotary
// key rows are scanned right after the r_k content rows, in the same batches.
//
// The prologue (q~ = U_k^T q) and the epilogue (U_v z) read the loop-l
// up-projections with vector loads and reduce in a fixed order, so results
// are bitwise reproducible.
//
// The same kernel serves the fp32 causal prefill: M queries per (b, h), query m
// attending positions [0, p0 + m], one workgroup per query.

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {


template <int BYTES> struct VecT;
template <> struct VecT<16> { typedef uint4 type; };
template <> struct VecT<8> { typedef uint2 type; };
template <> struct VecT<4> { typedef uint32_t type; };
template <> struct VecT<2> { typedef uint16_t type; };

// Load VW consecutive elements (VW * sizeof(T) bytes, naturally aligned) as floats.
template <typename T, int VW>
__device__ __forceinline__ void load_vec(const T* p, float (&o)[VW]) {
  typedef typename VecT<VW * sizeof(T)>::type V;
  const V v = *reinterpret_cast<const V*>(p);
  const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
  for (int i = 0; i < VW; ++i) o[i] = Elem<T>::get(e, i);
}

// q~[j] = qscale * sum_i U_k[i][j] q[i].  Thread f -> (column chunk jc of VW
// columns, row block ib); row-block partials are summed in a fixed order.
template <typename T, int VW, int kThreads>
__device__ void absorb_query(const T* uk, int d, int rk, float qscale, const float* s_q,
                             float* s_part, float* s_qt) {
  const int nch = rk / VW;
  const int rb = nch >= kThreads ? 1 : kThreads / nch;
  for (int f = threadIdx.x; f < nch * rb; f += kThreads) {
    const int jc = f % nch, ib = f / nch;
    float acc[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) acc[e] = 0.f;
#pragma unroll 8
    for (int i = ib; i < d; i += rb) {
      float u[VW];
      load_vec<T, VW>(uk + (size_t)i * rk + jc * VW, u);
      const float qi = s_q[i];
#pragma unroll
      for (int e = 0; e < VW; ++e) acc[e] = fmaf(u[e], qi, acc[e]);
    }
#pragma unroll
    for (int e = 0; e < VW; ++e) s_part[ib * rk + jc * VW + e] = acc[e];
  }
  __syncthreads();
  for (int j = threadIdx.x; j < rk; j += kThreads) {
    float s = 0.f;
    for (int ib = 0; ib < rb; ++ib) s += s_part[ib * rk + j];
    s_qt[j] = s * qscale;
  }
  __syncthreads();
}

// q~[j] = qscale * sum_i U_k[i][j] q[i], with each thread reading the q
// entries of its rows straight from memory (no wait between the q and U_k
// loads) and at most 8 row blocks, so the final fixed-order sum is short.
template <typename T, int VW, int kThreads>
__device__ void absorb_query_direct(const T* uk, const T* qp, int d, int rk, float qscale,
                                    float* s_part, float* s_qt) {
  const int nch = rk / VW;
  const int rb = nch >= kThreads / 8 ? max(1, kThreads / nch) : 8;
  for (int f = threadIdx.x; f < nch * rb; f += kThreads) {
    const int jc = f % nch, ib = f / nch;
    float acc[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) acc[e] = 0.f;
#pragma unroll 8
    for (int i = ib; i < d; i += rb) {
      float u[VW];
      load_vec<T, VW>(uk + (size_t)i * rk + jc * VW, u);
      const float qi = Elem<T>::get(qp, i);
#pragma unroll
      for (int e = 0; e < VW; ++e) acc[e] = fmaf(u[e], qi, acc[e]);
    }
#pragma unroll
    for (int e = 0; e < VW; ++e) s_part[ib * rk + jc * VW + e] = acc[e];
  }
  __syncthreads();
  for (int j = threadIdx.x; j < rk; j += kThreads) {
    float s = 0.f;
    for (int ib = 0; ib < rb; ++ib) s += s_part[ib * rk + j];
    s_qt[j] = s * qscale;
  }
}

// out[i] = sum_j U_v[i][j] zn[j] (+ mu_v[i]).  P consecutive threads share a
// row and split its column chunks; their partials combine by xor shuffles.
template <typename T, int VW, int kThreads>
__device__ void value_epilogue(const T* uv, const T* muv, int d, int rv, const float* s_zn,
                               bool bad, int out_dtype, void* out, size_t obase) {
  const int P = (kThreads / d) >= 8 ? 8 : (kThreads / d) >= 4 ? 4 : (kThreads / d) >= 2 ? 2 : 1;
  const int t = threadIdx.x, i = t / P, part = t % P;
  const int nch = rv / VW;
  float acc = 0.f;
  if (i < d) {
#pragma unroll 8
    for (int c = part; c < nch; c += P) {
      float u[VW];
      load_vec<T, VW>(uv + (size_t)i * rv + c * VW, u);
#pragma unroll
      for (int e = 0; e < VW; ++e) acc = fmaf(u[e], s_zn[c * VW + e], acc);
    }
  }
  for (int off = 1; off < P; off <<= 1) acc += xor_shfl(acc, off);
  if (i < d && part == 0) {
    if (muv) acc += Elem<T>::get(muv, i);
    if (bad) acc = __builtin_nanf("");
    if (out_dtype == LLA_F32)
      static_cast<float*>(out)[obase + i] = acc;
    else
      static_cast<bf16_t*>(out)[obase + i] = f32_to_bf16(acc);
  }
}

// Raw buffer resource (gfx9 family word 3) over one contiguous region.
typedef __amdgpu_buffer_rsrc_t BufRsrc;
__device__ __forceinline__ BufRsrc make_rsrc(const void* base, size_t bytes) {
  const int n = bytes >= 0xffffffffull ? -1 : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}
// 16-byte load at voffset (per lane) + soffset (uniform); offsets past the
// region's size read as zero.
// Latent pages are read exactly once per call: the loads carry the non-temporal
// cache policy (aux bit 1, "nt"), so they do not displace reusable lines in L2
// and the MALL (measured on the Ouro-1.4B-shaped call: 367 -> 325 us).
constexpr int kCpolNT = 2;
__device__ __forceinline__ uint4 buf_ld16(BufRsrc r, int voff, int soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kCpolNT));
}
// Rotary keys are shared by every head of a sequence (one rotary key per
// token): ordinary cache policy, so the heads after the first find them in
// L2 or the MALL (1.8% fewer bytes fetched per Ouro-1.4B-shaped call).
__device__ __forceinline__ uint4 buf_ld16_shared(BufRsrc r, int voff, int soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// x[lane] + x[lane ^ 32]
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <typename T>
__device__ __forceinline__ int vec_width(int r) {
  constexpr int E = 16 / sizeof(T);
  return (r % E == 0) ? E : (r % 4 == 0) ? 4 : (r % 2 == 0) ? 2 : 1;
}

// DEEP: at most two wavefronts per SIMD; the doubled register budget holds a
// second batch of loads in flight (software pipelining).  Otherwise four per
// SIMD, one batch at a time.  HALF: K groups of PPG / 2 pages, two feature rows
// per wave-wide load (short contexts).
template <typename TIn, int GV, int kWaves, bool DEEP, bool HALF>
__global__ __launch_bounds__(kWaves * kWave) __attribute__((amdgpu_waves_per_eu(DEEP ? 2 : 4)))
void decode_kernel(DecodeArgs a) {
  constexpr int kThreads = kWaves * kWave;
  constexpr int KB = 8;  // K rows per load batch (DEEP keeps two batches in flight)
  constexpr int VB = 8;  // V row groups per load batch
  constexpr int EPL = Elem<TIn>::kPer16B;  // tokens covered by one 16-byte load
  constexpr int LPR = kPage / EPL;         // lanes per 64-token feature row
  constexpr int PPG = kWave / LPR;         // pages per group (K phase) = rows per load (V phase)
  constexpr int KRL = HALF ? 2 : 1;        // feature rows per wave-wide K load
  constexpr int KPG = PPG / KRL;           // pages per K group
  constexpr int KRB = KB * KRL;            // feature rows per K batch

  // s_work holds the prologue's row-block partials, then (after the prologue's
  // last barrier) the per-wave probability buffers and latent partials.
  constexpr int kPWave = PPG * kPage;
  __shared__ float s_q[kMaxHead];
  // content rows padded to KRB, then the rotary rows padded to KRB
  __shared__ __attribute__((aligned(16))) float s_qt[kMaxRank + (HALF ? 16 : 0)];
  __shared__ __attribute__((aligned(16))) float s_work[kWaves * (kPWave + kMaxRank)];
  static_assert(kWaves * (kPWave + kMaxRank) >= kThreads * 8, "prologue partials do not fit");
  float* const s_part = s_work;
  float (*const s_p)[kPWave] = reinterpret_cast<float (*)[kPWave]>(s_work);
  float (*const s_z)[kMaxRank] = reinterpret_cast<float (*)[kMaxRank]>(s_work + kWaves * kPWave);
  __shared__ float s_zn[kMaxRank];
  __shared__ float s_m[kWaves], s_l[kWaves];
  __shared__ int s_last;

  // the wave index is uniform across a wavefront; saying so keeps the page and
  // row offsets of the buffer loads in scalar registers
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  // XCD head order only in the 4-page-group variant, which serves split
  // launches of few (b, h) units (in the 8-page variant it measured 0.8%
  // slower on the unsplit Ouro-1.4B step)
  int bx, h;
  xcd_head_order(bx, h, HALF && a.splits > 1 && !(a.dr > 0 && a.Hr == 1));
  const unsigned ubx = bx;  // a workgroup index: unsigned division, as on blockIdx
  const int bm = ubx / a.splits, split = ubx - bm * a.splits;
  int b, m, N;
  if (a.causal) {
    b = bm / a.M;
    m = bm - b * a.M;
    N = a.p0 + m + 1;
  } else {
    b = bm;
    m = 0;
    N = a.ctx_len ? a.ctx_len[b] : a.n_ctx;
  }
  const bool bad = (N < 1) || (N > a.n_ctx);
  const int pages = bad ? 0 : (N + kPage - 1) / kPage;
  const int per = (pages + a.splits - 1) / a.splits;
  const int pb = min(pages, split * per);
  const int pe = min(pages, pb + per);

  const size_t bh = (size_t)b * a.H + h;
  const size_t unit = bh * a.M + m;  // (b, h, m)
  const int rk = a.rk, rv = a.rv;
  // s_qt slot of the first rotary row; rotary rows padded to whole batches
  // (dr is a multiple of 8)
  const int rq0 = HALF ? (rk + KRB - 1) / KRB * KRB : (rk + 7) & ~7;
  const int drp = HALF ? (a.dr + KRB - 1) / KRB * KRB : a.dr;

  // ---- prologue: absorbed query q~ = U_k^T q, with scale * log2(e) folded in ----
  {
    const TIn* qp = static_cast<const TIn*>(a.q) + unit * a.d;
    for (int i = tid; i < a.d; i += kThreads) s_q[i] = Elem<TIn>::get(qp, i);
    __syncthreads();
    const TIn* uk = static_cast<const TIn*>(a.uk) + (size_t)h * a.d * rk;
    switch (vec_width<TIn>(rk)) {
      case 8: absorb_query<TIn, (EPL >= 8 ? 8 : 4), kThreads>(uk, a.d, rk, a.qscale, s_q, s_part, s_qt); break;
      case 4: absorb_query<TIn, 4, kThreads>(uk, a.d, rk, a.qscale, s_q, s_part, s_qt); break;
      case 2: absorb_query<TIn, 2, kThreads>(uk, a.d, rk, a.qscale, s_q, s_part, s_qt); break;
      default: absorb_query<TIn, 1, kThreads>(uk, a.d, rk, a.qscale, s_q, s_part, s_qt); break;
    }
    // the last content batch is padded to whole batches with zero weights; the
    // rotary branch: the (already rotated) query part joins q~ as extra rows,
    // from the 16-byte aligned slot past the padded content rows
    for (int j = rk + tid; j < rq0; j += kThreads) s_qt[j] = 0.f;
    if (a.dr) {
      const TIn* qr = static_cast<const TIn*>(a.qr) + unit * a.dr;
      for (int i = tid; i < a.dr; i += kThreads) s_qt[rq0 + i] = a.qscale * Elem<TIn>::get(qr, i);
      if constexpr (HALF)
        for (int i = a.dr + tid; i < drp; i += kThreads) s_qt[rq0 + i] = 0.f;
    }
    __syncthreads();
  }

  const int hi = lane / LPR, lo = lane - hi * LPR;
  const int kpg = HALF ? hi % KPG : hi;  // K phase: page of the group
  const int krw = HALF ? hi / KPG : 0;   // K phase (HALF): which row of each load's pair
  float zacc[GV];
#pragma unroll
  for (int k = 0; k < GV; ++k) zacc[k] = 0.f;
  float m_run = neg_inf(), l_lane = 0.f;

  // Buffer resources over this (b, h)'s latents: the row and page offsets are
  // wave-uniform (SGPR), the lane part is one VGPR.
  constexpr int ES = sizeof(TIn);
  const BufRsrc rk_src = make_rsrc(static_cast<const TIn*>(a.ck) + bh * (size_t)a.n_max * rk,
                                   (size_t)a.n_max * rk * ES);
  const BufRsrc rv_src = make_rsrc(static_cast<const TIn*>(a.cv) + bh * (size_t)a.n_max * rv,
                                   (size_t)a.n_max * rv * ES);
  const int kpage_bytes = kPage * rk * ES, vpage_bytes = kPage * rv * ES;
  // K phase: page kpg of the group, slice lo (HALF: and the odd row for krw = 1)
  const int vk_lane = kpg * kpage_bytes + krw * kPage * ES + lo * 16;
  // rotary keys of this (b, h): the same paging with dr feature rows
  const size_t bhr = (size_t)b * a.Hr + (a.Hr == 1 ? 0 : h);
  const BufRsrc rr_src = make_rsrc(a.dr ? static_cast<const TIn*>(a.rc) + bhr * (size_t)a.n_max * a.dr
                                        : static_cast<const TIn*>(a.ck),
                                   (size_t)a.n_max * a.dr * ES);
  const int rpage_bytes = kPage * a.dr * ES;
  const int vr_lane = kpg * rpage_bytes + krw * kPage * ES + lo * 16;
  // HALF: offsets past each region's size (rows beyond r_k or dr) read as zero
  // and touch no memory
  const int k_oob = a.n_max * rk * ES, r_oob = a.n_max * a.dr * ES;
  const int vv_lane = hi * kPage * ES + lo * 16;    // V phase: row hi of the row group, slice lo
  const int vg_full = rv / PPG, vg_part = rv % PPG;  // full row groups, rows of the partial one
  float* sp = s_p[wave];

  // ---- latent scan, PPG pages per wave per group ----
  // With PIPE (the DEEP variant's register budget) the next batch of rows is
  // always in flight while the current one is multiplied: K batches ping-pong
  // between two register sets, and V batches prefetch across row groups and
  // pages, so the FMAs of one batch overlap the memory latency of the next.
  constexpr bool PIPE = DEEP;
  const int nkb = (rk + KRB - 1) / KRB;                     // K batches (the last padded, zero weights)
  const int ntb = nkb + drp / KRB;                          // plus the rotary rows
  const int nvb = (vg_full + (vg_part ? 1 : 0) + VB - 1) / VB;  // V batches per page
  constexpr int NKC = (GV + VB - 1) / VB;

  // batch jb < nkb: content rows jb*KRB.. of c_k (rows past r_k re-read row
  // r_k - 1, weighted by zero); later batches: rotary rows.  Every batch issues
  // all its loads, so the compiler's waits count loads exactly.
  auto kload = [&](uint4 (&r)[KB], int g0p, int jb) {
    if constexpr (HALF) {
      // load u reads rows r0 = 2u (lanes krw = 0) and r0 + 1 (krw = 1) of the
      // batch's content or rotary rows, page g0p + kpg; the pair's offset is
      // uniform, and a lane whose row is past the range reads out of the region
      // (zero, no memory access)
      const bool rot = jb >= nkb;
      const BufRsrc src = rot ? rr_src : rk_src;
      const int lim = rot ? a.dr : rk, oob = rot ? r_oob : k_oob;
      const int lbase = rot ? vr_lane : vk_lane;
      const int pbase = g0p * (rot ? rpage_bytes : kpage_bytes);
      const int rb = (rot ? jb - nkb : jb) * KRB;
#pragma unroll
      for (int u = 0; u < KB; ++u) {
        const int r0 = rb + 2 * u;
        const int so = r0 < lim ? pbase + r0 * kPage * ES : 0;
        r[u] = buf_ld16(src, r0 + krw < lim ? lbase : oob, so);
      }
      return;
    }
    if (jb < nkb) {
#pragma unroll
      for (int u = 0; u < KB; ++u)
        r[u] = buf_ld16(rk_src, vk_lane, g0p * kpage_bytes + min(jb * KB + u, rk - 1) * kPage * ES);
    } else {
#pragma unroll
      for (int u = 0; u < KB; ++u)
        r[u] = buf_ld16_shared(rr_src, vr_lane, g0p * rpage_bytes + ((jb - nkb) * KB + u) * kPage * ES);
    }
  };
  auto kfma = [&](const uint4 (&r)[KB], int jb, float (&acc)[EPL]) {
    float qj[KB];
    const int q0 = jb < nkb ? jb * KRB : rq0 + (jb - nkb) * KRB;
    if constexpr (HALF) {
#pragma unroll
      for (int u = 0; u < KB; ++u) qj[u] = s_qt[q0 + 2 * u + krw];
    } else {
#pragma unroll
      for (int u = 0; u < KB; u += 4) {
        const float4 qa = *reinterpret_cast<const float4*>(&s_qt[q0 + u]);
        qj[u] = qa.x;
        qj[u + 1] = qa.y;
        qj[u + 2] = qa.z;
        qj[u + 3] = qa.w;
      }
    }
#pragma unroll
    for (int u = 0; u < KB; ++u) {
      float v[EPL];
      Elem<TIn>::unpack(r[u], v);
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = fmaf(qj[u], v[e], acc[e]);
    }
  };
  auto vload = [&](uint4 (&r)[VB], int pv, int kc) {
    const int pbase = pv * vpage_bytes;
#pragma unroll
    for (int u = 0; u < VB; ++u) {
      const int k = kc * VB + u;
      if (k < vg_full || (k == vg_full && hi < vg_part))
        r[u] = buf_ld16(rv_src, vv_lane, pbase + k * PPG * kPage * ES);
    }
  };

  for (int g0 = pb + wave * KPG; g0 < pe; g0 += kWaves * KPG) {
    const int np = min(KPG, pe - g0);
    float acc[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
    if (kpg < np) {
      if constexpr (PIPE) {
        uint4 ka[KB], kb2[KB];
        if (ntb > 0) kload(ka, g0, 0);
        for (int jb = 0; jb < ntb; jb += 2) {
          if (jb + 1 < ntb) kload(kb2, g0, jb + 1);
          kfma(ka, jb, acc);
          if (jb + 2 < ntb) kload(ka, g0, jb + 2);
          if (jb + 1 < ntb) kfma(kb2, jb + 1, acc);
        }
      } else {
        for (int jb = 0; jb < ntb; ++jb) {
          uint4 ka[KB];
          kload(ka, g0, jb);
          kfma(ka, jb, acc);
        }
      }
    }
    if constexpr (HALF) {  // each half of the wave holds half of every score's rows
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = sum_halves(acc[e]);
    }
    uint4 vcur[VB];
    if constexpr (PIPE) vload(vcur, g0, 0);  // first V batch in flight during the softmax

    // scores of invalid pages / tokens beyond N are -inf
    const int n0 = (g0 + kpg) * kPage + lo * EPL;
    float mb = neg_inf();
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      if (kpg >= np || n0 + e >= N) acc[e] = neg_inf();
      mb = fmaxf(mb, acc[e]);
    }
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) mb = fmaxf(mb, xor_shfl(mb, off));
    if (mb > m_run) {
      const float alpha = fast_exp2(m_run - mb);
      l_lane *= alpha;
#pragma unroll
      for (int k = 0; k < GV; ++k) zacc[k] *= alpha;
      m_run = mb;
    }
    float pr[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      pr[e] = fast_exp2(acc[e] - m_run);
      if (krw == 0) l_lane += pr[e];  // HALF: the upper half holds the same probabilities
    }
    if (krw == 0) {
#pragma unroll
      for (int e = 0; e < EPL; e += 4)
        *reinterpret_cast<float4*>(&sp[kpg * kPage + lo * EPL + e]) =
            make_float4(pr[e], pr[e + 1], pr[e + 2], pr[e + 3]);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // V phase: lane (hi = row in the row group, lo = token slice), page by page
    for (int pg = 0; pg < np; ++pg) {
      const int pv = g0 + pg;
      float p8[EPL];
#pragma unroll
      for (int e = 0; e < EPL; e += 4) {
        const float4 t = *reinterpret_cast<const float4*>(&sp[pg * kPage + lo * EPL + e]);
        p8[e] = t.x;
        p8[e + 1] = t.y;
        p8[e + 2] = t.z;
        p8[e + 3] = t.w;
      }
      const bool tail = (pv + 1) * kPage > N;
      if (tail) {  // tokens beyond N: weight 0 and value 0 (the slot may hold anything)
        const int nv0 = pv * kPage + lo * EPL;
#pragma unroll
        for (int e = 0; e < EPL; ++e)
          if (nv0 + e >= N) p8[e] = 0.f;
      }
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) {
        if (kc < nvb) {
          uint4 vnext[VB];
          if constexpr (PIPE) {
            if (kc + 1 < nvb)
              vload(vnext, pv, kc + 1);
            else if (pg + 1 < np)
              vload(vnext, pv + 1, 0);
          } else {
            vload(vcur, pv, kc);
          }
#pragma unroll
          for (int u = 0; u < VB; ++u) {
            const int k = kc * VB + u;
            if (k < GV && (k < vg_full || (k == vg_full && hi < vg_part))) {
              float v[EPL];
              Elem<TIn>::unpack(vcur[u], v);
              if (tail) {  // slots past N: value 0 (an attended NaN still propagates)
                const int nv0 = pv * kPage + lo * EPL;
#pragma unroll
                for (int e = 0; e < EPL; ++e)
                  if (nv0 + e >= N) v[e] = 0.f;
              }
              float t = 0.f;
#pragma unroll
              for (int e = 0; e < EPL; ++e) t = fmaf(p8[e], v[e], t);
              zacc[k] += t;
            }
          }
          if constexpr (PIPE) {
#pragma unroll
            for (int u = 0; u < VB; ++u) vcur[u] = vnext[u];
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // ---- wave reductions: l over all lanes, z over token slices ----
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) l_lane += xor_shfl(l_lane, off);
#pragma unroll
  for (int off = 1; off < LPR; off <<= 1)
#pragma unroll
    for (int k = 0; k < GV; ++k) zacc[k] += xor_shfl(zacc[k], off);
  if (lo == 0) {
#pragma unroll
    for (int k = 0; k < GV; ++k) {
      const int j = k * PPG + hi;
      if (j < rv) s_z[wave][j] = zacc[k];
    }
  }
  if (lane == 0) {
    s_m[wave] = m_run;
    s_l[wave] = l_lane;
  }
  __syncthreads();

  // ---- merge the waves of this workgroup (LDS) ----
  float wt[kWaves];
  float mg = neg_inf();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) mg = fmaxf(mg, s_m[w]);
  float lg = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    wt[w] = (s_m[w] == neg_inf()) ? 0.f : fast_exp2(s_m[w] - mg);
    lg = fmaf(wt[w], s_l[w], lg);
  }

  if (a.splits == 1) {
    for (int j = tid; j < rv; j += kThreads) {
      float z = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) z = fmaf(wt[w], s_z[w][j], z);
      s_zn[j] = z / lg;
    }
  } else {
    // ---- split-K: publish this workgroup's partial, last arrival merges ----
    const int stride = rv + 2;
    float* part = a.part + (unit * a.splits + split) * stride;
    for (int j = tid; j < rv; j += kThreads) {
      float z = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) z = fmaf(wt[w], s_z[w][j], z);
      part[2 + j] = z;
    }
    if (tid == 0) {
      part[0] = mg;
      part[1] = lg;
    }
    // Every wavefront's partial stores reach L2 before the barrier; thread
    // 0's counter update is then the workgroup's one agent-scope release (one
    // L2 write-back covering them all) and publishes the arrival, and the last
    // arrival's acquire (by thread 0, then the barrier) makes every split's
    // partial visible to the whole workgroup.
    wait_stores_in_l2();
    __syncthreads();
    if (tid == 0) {
      const uint32_t prev =
          __hip_atomic_fetch_add(a.cnt + unit, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == (uint32_t)(a.splits - 1));
    }
    __syncthreads();
    if (!s_last) return;
    const float* P = a.part + unit * a.splits * stride;
    float ma = neg_inf();
    for (int s = 0; s < a.splits; ++s) ma = fmaxf(ma, P[(size_t)s * stride]);
    float la = 0.f;
    for (int s = 0; s < a.splits; ++s) {
      const float ms = P[(size_t)s * stride];
      const float ws = (ms == neg_inf()) ? 0.f : fast_exp2(ms - ma);
      la = fmaf(ws, P[(size_t)s * stride + 1], la);
    }
    for (int j = tid; j < rv; j += kThreads) {
      float z = 0.f;
      for (int s = 0; s < a.splits; ++s) {
        const float ms = P[(size_t)s * stride];
        const float ws = (ms == neg_inf()) ? 0.f : fast_exp2(ms - ma);
        z = fmaf(ws, P[(size_t)s * stride + 2 + j], z);
      }
      s_zn[j] = z / la;
    }
    if (tid == 0) __hip_atomic_store(a.cnt + unit, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();

  // ---- value epilogue: out = U_v z + mu_v ----
  const TIn* uv = static_cast<const TIn*>(a.uv) + (size_t)h * a.d * rv;
  const TIn* muv = a.muv ? static_cast<const TIn*>(a.muv) + (size_t)h * a.d : nullptr;
  const size_t obase = unit * a.d;
  switch (vec_width<TIn>(rv)) {
    case 8: value_epilogue<TIn, (EPL >= 8 ? 8 : 4), kThreads>(uv, muv, a.d, rv, s_zn, bad, a.out_dtype, a.out, obase); break;
    case 4: value_epilogue<TIn, 4, kThreads>(uv, muv, a.d, rv, s_zn, bad, a.out_dtype, a.out, obase); break;
    case 2: value_epilogue<TIn, 2, kThreads>(uv, muv, a.d, rv, s_zn, bad, a.out_dtype, a.out, obase); break;
    default: value_epilogue<TIn, 1, kThreads>(uv, muv, a.d, rv, s_zn, bad, a.out_dtype, a.out, obase); break;
  }
}

// Row-split decode, bf16: the W = 4 or 8 wavefronts of a workgroup split the
// feature rows of each 8-page group instead of its pages, so a group's loads
// are spread over every wavefront whatever the page count.  A workgroup walks
// the groups of its (b, h) context, or of one slice of it (SPLIT), in turn;
// the launch heuristic uses it for short contexts, for slices of 8 to 64
// pages when few (b, h) units split their contexts, and for whole contexts of
// up to 128 pages in batches of one compute unit's worth of (b, h) or less.
//   * K phase -- wave w takes the 8-row blocks w, w + W, ... of the content
//     rows and then of the rotary rows; lane (pg, ts) owns tokens ts*8.. of
//     page pg, so one wave-wide load reads one feature row of all 8 pages.
//     The W partial scores of a token are summed through LDS (double
//     buffered over groups, one barrier per group), in the same order in
//     every wavefront, so all of them hold identical scores and softmax
//     statistics.
//   * V phase -- wave w takes the 8-row groups w, w + W, ... of the value
//     latents, each over all pages of the group (lane (rg, ts): row rg of the
//     group, token slice ts); its z rows are its own, so no merge follows.
// Eight wavefronts halve each one's chain of dependent row loads; they are
// used when every workgroup fits at one per compute unit.
// Slots that are not read (pages past the context, rows past r_k, r_v or dr)
// are requested out of the region: they read as zero and touch no memory.
template <int GV, bool SPLIT, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) __attribute__((amdgpu_waves_per_eu(2)))
void decode_short_kernel(DecodeArgs a) {
  typedef bf16_t TIn;
  constexpr int kWaves = WAVES, kThreads = kWaves * kWave;
  constexpr int KB = 8;                       // loads per K batch
  constexpr int EPL = 8;                      // tokens per 16-byte load
  constexpr int PPG = 8;                      // pages per group
  constexpr int VH = PPG / 2;                 // pages per V half-batch
  constexpr int GVW = (GV + kWaves - 1) / kWaves;  // value row groups per wavefront
  constexpr int ES = 2;
  __shared__ __attribute__((aligned(16))) float s_qt[kMaxRank];
  // partial scores [buffer][wave][page*64 + token]; the prologue's row-block
  // partials use the same memory before the first group
  __shared__ __attribute__((aligned(16))) float s_ps[2][kWaves][PPG * kPage];
  __shared__ __attribute__((aligned(16))) float s_p[kWaves][PPG * kPage];  // per-wave probabilities
  __shared__ float s_zn[kMaxRank];
  // U_v of this head when it fits (d_head * r_v * 2 bytes, r_v <= 64 at d_head 128): requested
  // before the query absorption and written to LDS after it (its loads return before the
  // absorption's own), so the epilogue pays no memory latency
  constexpr bool kUvPre = GV <= 8;
  constexpr int kUvBytes = kUvPre ? 16384 : 16;
  __shared__ __attribute__((aligned(16))) bf16_t s_uv[kUvBytes / 2];
  __shared__ int s_last;
  static_assert(2 * kWaves * PPG * kPage >= kThreads * 8, "prologue partials do not fit");
  float* const s_part = &s_ps[0][0][0];

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  // SPLIT: the workgroup takes one slice of its (b, h) context (split-K)
  int bx, h;
  xcd_head_order(bx, h, !(a.dr > 0 && a.Hr == 1));  // a shared rotary key keeps a sequence's heads together
  const unsigned ubx = bx;  // a workgroup index: unsigned division, as on blockIdx
  const int b = SPLIT ? ubx / a.splits : ubx;
  const int split = SPLIT ? ubx - b * a.splits : 0;
  const int N = a.ctx_len ? a.ctx_len[b] : a.n_ctx;
  const bool bad = (N < 1) || (N > a.n_ctx);
  const int pages = bad ? 0 : (N + kPage - 1) / kPage;
  // this slice's pages [pb, pe)
  const int per = SPLIT ? (pages + a.splits - 1) / a.splits : pages;
  const int pb = SPLIT ? min(pages, split * per) : 0, pe = SPLIT ? min(pages, pb + per) : pages;
  const size_t unit = (size_t)b * a.H + h;
  const int rk = a.rk, rv = a.rv, dr = a.dr;
  const int rq0 = (rk + 7) & ~7;  // s_qt slot of the first rotary row

  const int hi = lane >> 3, lo = lane & 7;  // K: page hi, slice lo; V: row hi of the group, slice lo
  const BufRsrc rk_src = make_rsrc(static_cast<const TIn*>(a.ck) + unit * (size_t)a.n_max * rk,
                                   (size_t)a.n_max * rk * ES);
  const BufRsrc rv_src = make_rsrc(static_cast<const TIn*>(a.cv) + unit * (size_t)a.n_max * rv,
                                   (size_t)a.n_max * rv * ES);
  const size_t bhr = (size_t)b * a.Hr + (a.Hr == 1 ? 0 : h);
  const BufRsrc rr_src = make_rsrc(dr ? static_cast<const TIn*>(a.rc) + bhr * (size_t)a.n_max * dr
                                      : static_cast<const TIn*>(a.ck),
                                   (size_t)a.n_max * dr * ES);
  const int kpage_bytes = kPage * rk * ES, vpage_bytes = kPage * rv * ES, rpage_bytes = kPage * dr * ES;
  const int k_oob = a.n_max * rk * ES, v_oob = a.n_max * rv * ES, r_oob = a.n_max * dr * ES;
  const int k_lane = hi * kpage_bytes + lo * 16, r_lane = hi * rpage_bytes + lo * 16;
  const int v_lane = hi * kPage * ES + lo * 16;
  const int nkb = (rk + 7) / 8, ntb = nkb + dr / 8;  // 8-row K blocks (content, then rotary)
  const int nmk = ntb > wave ? (ntb - 1 - wave) / kWaves + 1 : 0;  // this wave's K blocks
  const int nvg = (rv + 7) / 8;                                    // 8-row value groups
  const int nmv = nvg > wave ? (nvg - 1 - wave) / kWaves + 1 : 0;  // this wave's value groups

  // K block i of this wave over the group at page g0 (np pages): 8 rows, all
  // 8 loads issued by every lane
  auto kload = [&](uint4 (&r)[KB], int i, int g0, int np) {
    const int blk = wave + i * kWaves;
    const bool rot = blk >= nkb;
    const BufRsrc src = rot ? rr_src : rk_src;
    const int lim = rot ? dr : rk, oob = rot ? r_oob : k_oob;
    const int base = hi < np ? (rot ? r_lane : k_lane) : oob;
    const int pbase = g0 * (rot ? rpage_bytes : kpage_bytes);
    const int r0 = (rot ? blk - nkb : blk) * 8;
#pragma unroll
    for (int u = 0; u < KB; ++u) {
      const int row = r0 + u;
      const bool ok = row < lim;
      r[u] = buf_ld16(src, ok ? base : oob, ok ? pbase + row * kPage * ES : 0);
    }
  };
  auto kfma = [&](const uint4 (&r)[KB], int i, float (&acc)[EPL]) {
    const int blk = wave + i * kWaves;
    const int q0 = blk < nkb ? blk * 8 : rq0 + (blk - nkb) * 8;
    float qj[KB];
#pragma unroll
    for (int u = 0; u < KB; u += 4) {
      const float4 qa = *reinterpret_cast<const float4*>(&s_qt[q0 + u]);
      qj[u] = qa.x;
      qj[u + 1] = qa.y;
      qj[u + 2] = qa.z;
      qj[u + 3] = qa.w;
    }
#pragma unroll
    for (int u = 0; u < KB; ++u) {
      float v[EPL];
      Elem<TIn>::unpack(r[u], v);
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = fmaf(qj[u], v[e], acc[e]);
    }
  };
  // half pg0 / VH of value row group k of this wave over the group at page g0
  auto vload = [&](uint4 (&r)[VH], int k, int pg0, int g0, int np) {
    const int row0 = (wave + k * kWaves) * 8;
    const bool ok = row0 + hi < rv;
#pragma unroll
    for (int u = 0; u < VH; ++u) {
      const bool pok = pg0 + u < np;
      r[u] = buf_ld16(rv_src, ok && pok ? v_lane : v_oob,
                      pok ? (g0 + pg0 + u) * vpage_bytes + row0 * kPage * ES : 0);
    }
  };

  uint4 ka[KB], kb2[KB], va[VH], vb[VH];
  const TIn* uv_g = static_cast<const TIn*>(a.uv) + (size_t)h * a.d * rv;
  const bool uv_pre = kUvPre && a.d * rv * 2 <= kUvBytes;  // uniform
  const int n_uv16 = a.d * rv * 2 / 16;                     // d_head is a multiple of 32: whole 16-byte pieces
  constexpr int kUvPer = kUvBytes / 16 / kThreads > 0 ? kUvBytes / 16 / kThreads : 1;
  uint4 uvr[kUvPer];
  if (uv_pre) {
#pragma unroll
    for (int k = 0; k < kUvPer; ++k) {
      const int e = tid + k * kThreads;
      uvr[k] = e < n_uv16 ? reinterpret_cast<const uint4*>(uv_g)[e] : uint4{0, 0, 0, 0};
    }
  }

  // ---- prologue: q~ = U_k^T q (scale * log2 e folded in), then the rotary query ----
  {
    const TIn* qp = static_cast<const TIn*>(a.q) + unit * a.d;
    const TIn* uk = static_cast<const TIn*>(a.uk) + (size_t)h * a.d * rk;
    switch (vec_width<TIn>(rk)) {
      case 8: absorb_query_direct<TIn, 8, kThreads>(uk, qp, a.d, rk, a.qscale, s_part, s_qt); break;
      case 4: absorb_query_direct<TIn, 4, kThreads>(uk, qp, a.d, rk, a.qscale, s_part, s_qt); break;
      case 2: absorb_query_direct<TIn, 2, kThreads>(uk, qp, a.d, rk, a.qscale, s_part, s_qt); break;
      default: absorb_query_direct<TIn, 1, kThreads>(uk, qp, a.d, rk, a.qscale, s_part, s_qt); break;
    }
    for (int j = rk + tid; j < rq0; j += kThreads) s_qt[j] = 0.f;
    if (dr) {
      const TIn* qr = static_cast<const TIn*>(a.qr) + unit * dr;
      for (int i = tid; i < dr; i += kThreads) s_qt[rq0 + i] = a.qscale * Elem<TIn>::get(qr, i);
    }
    __syncthreads();
  }
  if (uv_pre) {  // read by the epilogue, after the final barrier
#pragma unroll
    for (int k = 0; k < kUvPer; ++k) {
      const int e = tid + k * kThreads;
      if (e < n_uv16) reinterpret_cast<uint4*>(s_uv)[e] = uvr[k];
    }
  }

  float zacc[GVW];
#pragma unroll
  for (int k = 0; k < GVW; ++k) zacc[k] = 0.f;
  float m_run = neg_inf(), l_lane = 0.f;

  int buf = 0;
  for (int g0 = pb; g0 < pe; g0 += PPG, buf ^= 1) {
    const int np = min(PPG, pe - g0);

    // ---- K phase: this wave's row blocks over all pages of the group ----
    float acc[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
    if (nmk > 0) kload(ka, 0, g0, np);
    for (int i = 0; i < nmk; i += 2) {
      if (i + 1 < nmk) kload(kb2, i + 1, g0, np);
      kfma(ka, i, acc);
      if (i + 2 < nmk) kload(ka, i + 2, g0, np);
      if (i + 1 < nmk) kfma(kb2, i + 1, acc);
    }
    float* ps = &s_ps[buf][0][0];
#pragma unroll
    for (int e = 0; e < EPL; e += 4)
      *reinterpret_cast<float4*>(&ps[wave * PPG * kPage + hi * kPage + lo * EPL + e]) =
          make_float4(acc[e], acc[e + 1], acc[e + 2], acc[e + 3]);
    __syncthreads();
    // the wavefronts' partials, summed in wave order (identical in every wavefront)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
#pragma unroll
      for (int e = 0; e < EPL; e += 4) {
        const float4 t = *reinterpret_cast<const float4*>(&ps[w * PPG * kPage + hi * kPage + lo * EPL + e]);
        acc[e] += t.x;
        acc[e + 1] += t.y;
        acc[e + 2] += t.z;
        acc[e + 3] += t.w;
      }
    }

    // ---- softmax over the group (pages past the context and tokens past N: -inf) ----
    const int n0 = (g0 + hi) * kPage + lo * EPL;
    float mb = neg_inf();
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      if (hi >= np || n0 + e >= N) acc[e] = neg_inf();
      mb = fmaxf(mb, acc[e]);
    }
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) mb = fmaxf(mb, xor_shfl(mb, off));
    if (mb > m_run) {
      const float alpha = fast_exp2(m_run - mb);
      l_lane *= alpha;
#pragma unroll
      for (int k = 0; k < GVW; ++k) zacc[k] *= alpha;
      m_run = mb;
    }
    float* sp = s_p[wave];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      acc[e] = fast_exp2(acc[e] - m_run);
      l_lane += acc[e];
    }
#pragma unroll
    for (int e = 0; e < EPL; e += 4)
      *reinterpret_cast<float4*>(&sp[hi * kPage + lo * EPL + e]) =
          make_float4(acc[e], acc[e + 1], acc[e + 2], acc[e + 3]);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---- V phase: this wave's value row groups over all pages of the group ----
    // The probabilities of lane (rg, ts) are those of token slice ts of every
    // page: 64 registers, read once per group.  Each row group is loaded in two
    // halves of 4 pages, one half always in flight.
    float p8[PPG][EPL];
#pragma unroll
    for (int pg = 0; pg < PPG; ++pg) {
#pragma unroll
      for (int e = 0; e < EPL; e += 4) {
        const float4 t = *reinterpret_cast<const float4*>(&sp[pg * kPage + lo * EPL + e]);
        p8[pg][e] = t.x;
        p8[pg][e + 1] = t.y;
        p8[pg][e + 2] = t.z;
        p8[pg][e + 3] = t.w;
      }
    }
    // value slots past N may hold anything: their weight is 0 and their value
    // is zeroed (an attended NaN still propagates)
    const int tail_pg = (N - 1) / kPage - g0;  // page of the group holding position N - 1
    auto vfma = [&](const uint4 (&r)[VH], auto pg0c, float& t) {
      constexpr int pg0 = decltype(pg0c)::value;
#pragma unroll
      for (int u = 0; u < VH; ++u) {
        float v[EPL];
        Elem<TIn>::unpack(r[u], v);
        if (pg0 + u == tail_pg) {
          const int nv0 = (g0 + pg0 + u) * kPage + lo * EPL;
#pragma unroll
          for (int e = 0; e < EPL; ++e)
            if (nv0 + e >= N) v[e] = 0.f;
        }
#pragma unroll
        for (int e = 0; e < EPL; ++e) t = fmaf(p8[pg0 + u][e], v[e], t);
      }
    };
    if (nmv > 0) vload(va, 0, 0, g0, np);
    for (int k = 0; k < nmv; ++k) {
      float t = 0.f;
      vload(vb, k, VH, g0, np);
      vfma(va, std::integral_constant<int, 0>{}, t);
      if (k + 1 < nmv) vload(va, k + 1, 0, g0, np);
      vfma(vb, std::integral_constant<int, VH>{}, t);
#pragma unroll
      for (int kk = 0; kk < GVW; ++kk)
        if (kk == k) zacc[kk] += t;
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // ---- this wave's z rows: reduce over the token slices, normalise ----
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) l_lane += xor_shfl(l_lane, off);
#pragma unroll
  for (int off = 1; off < 8; off <<= 1)
#pragma unroll
    for (int k = 0; k < GVW; ++k) zacc[k] += xor_shfl(zacc[k], off);
  if constexpr (!SPLIT) {
    if (lo == 0) {
#pragma unroll
      for (int k = 0; k < GVW; ++k) {
        const int j = (wave + k * kWaves) * 8 + hi;
        if (k < nmv && j < rv) s_zn[j] = zacc[k] / l_lane;
      }
    }
  } else {
    // ---- split-K: publish (m, l, z) of this split's pages; the last arrival merges ----
    // (every wavefront holds the same m and l; each holds its own z rows)
    const int stride = rv + 2;
    float* part = a.part + (unit * a.splits + split) * stride;
    if (lo == 0) {
#pragma unroll
      for (int k = 0; k < GVW; ++k) {
        const int j = (wave + k * kWaves) * 8 + hi;
        if (k < nmv && j < rv) part[2 + j] = zacc[k];
      }
    }
    if (tid == 0) {
      part[0] = m_run;
      part[1] = l_lane;
    }
    // every wavefront's stores reach L2 before the barrier; thread 0's counter
    // update is the workgroup's one agent-scope release and the last arrival's
    // acquire makes every split's partial visible
    wait_stores_in_l2();
    __syncthreads();
    if (tid == 0) {
      const uint32_t prev =
          __hip_atomic_fetch_add(a.cnt + unit, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == (uint32_t)(a.splits - 1));
    }
    __syncthreads();
    if (!s_last) return;
    const float* P = a.part + unit * a.splits * stride;
    float ma = neg_inf();
    for (int s = 0; s < a.splits; ++s) ma = fmaxf(ma, P[(size_t)s * stride]);
    float la = 0.f;
    for (int s = 0; s < a.splits; ++s) {
      const float ms = P[(size_t)s * stride];
      const float ws = (ms == neg_inf()) ? 0.f : fast_exp2(ms - ma);
      la = fmaf(ws, P[(size_t)s * stride + 1], la);
    }
    for (int j = tid; j < rv; j += kThreads) {
      float z = 0.f;
      for (int s = 0; s < a.splits; ++s) {
        const float ms = P[(size_t)s * stride];
        const float ws = (ms == neg_inf()) ? 0.f : fast_exp2(ms - ma);
        z = fmaf(ws, P[(size_t)s * stride + 2 + j], z);
      }
      s_zn[j] = z / la;
    }
    if (tid == 0) __hip_atomic_store(a.cnt + unit, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();

  // ---- value epilogue: out = U_v z + mu_v ----
  const TIn* uv = uv_pre ? s_uv : uv_g;
  const TIn* muv = a.muv ? static_cast<const TIn*>(a.muv) + (size_t)h * a.d : nullptr;
  const size_t obase = unit * a.d;
  switch (vec_width<TIn>(rv)) {
    case 8: value_epilogue<TIn, 8, kThreads>(uv, muv, a.d, rv, s_zn, bad, a.out_dtype, a.out, obase); break;
    case 4: value_epilogue<TIn, 4, kThreads>(uv, muv, a.d, rv, s_zn, bad, a.out_dtype, a.out, obase); break;
    case 2: value_epilogue<TIn, 2, kThreads>(uv, muv, a.d, rv, s_zn, bad, a.out_dtype, a.out, obase); break;
    default: value_epilogue<TIn, 1, kThreads>(uv, muv, a.d, rv, s_zn, bad, a.out_dtype, a.out, obase); break;
  }
}

template <typename TIn, int GV>
hipError_t launch_t(const DecodeArgs& a, hipStream_t stream) {
  dim3 grid(a.B * a.M * a.splits, a.H);
  if (a.shortk) {  // row-split kernel (rows of each 8-page group split over the wavefronts): bf16, decode
    if constexpr (sizeof(TIn) == 2) {
      if (a.causal || a.M != 1) return hipErrorInvalidValue;
      if (a.waves != 4 && a.waves != 8) return hipErrorInvalidValue;
      if (a.waves == 8) {
        if (a.splits > 1)
          hipLaunchKernelGGL((decode_short_kernel<GV, true, 8>), grid, dim3(8 * kWave), 0, stream, a);
        else
          hipLaunchKernelGGL((decode_short_kernel<GV, false, 8>), grid, dim3(8 * kWave), 0, stream, a);
      } else if (a.splits > 1) {
        hipLaunchKernelGGL((decode_short_kernel<GV, true, 4>), grid, dim3(4 * kWave), 0, stream, a);
      } else {
        hipLaunchKernelGGL((decode_short_kernel<GV, false, 4>), grid, dim3(4 * kWave), 0, stream, a);
      }
      return hipGetLastError();
    } else {
      return hipErrorInvalidValue;
    }
  }
  if (a.half) {  // 4-page K groups: bf16, pipelined, 4 or 8 wavefronts
    if constexpr (sizeof(TIn) == 2) {
      if (!a.deep || (a.waves != 4 && a.waves != 8)) return hipErrorInvalidValue;
      if (a.waves == 8)
        hipLaunchKernelGGL((decode_kernel<TIn, GV, 8, true, true>), grid, dim3(8 * kWave), 0, stream, a);
      else
        hipLaunchKernelGGL((decode_kernel<TIn, GV, 4, true, true>), grid, dim3(4 * kWave), 0, stream, a);
      return hipGetLastError();
    } else {
      return hipErrorInvalidValue;
    }
  }
  if (a.waves == 8) {
    if (a.deep)
      hipLaunchKernelGGL((decode_kernel<TIn, GV, 8, true, false>), grid, dim3(8 * kWave), 0, stream, a);
    else
      hipLaunchKernelGGL((decode_kernel<TIn, GV, 8, false, false>), grid, dim3(8 * kWave), 0, stream, a);
  } else {
    if (a.deep)
      hipLaunchKernelGGL((decode_kernel<TIn, GV, 4, true, false>), grid, dim3(4 * kWave), 0, stream, a);
    else
      hipLaunchKernelGGL((decode_kernel<TIn, GV, 4, false, false>), grid, dim3(4 * kWave), 0, stream, a);
  }
  return hipGetLastError();
}

template <typename TIn>
hipError_t dispatch(const DecodeArgs& a, hipStream_t stream) {
  constexpr int RPL = kWave / (kPage / Elem<TIn>::kPer16B);  // V rows per wave-wide load
  const int gv = (a.rv + RPL - 1) / RPL;
  if (gv <= 4) return launch_t<TIn, 4>(a, stream);
  if (gv <= 8) return launch_t<TIn, 8>(a, stream);
  if (gv <= 16) return launch_t<TIn, 16>(a, stream);
  if (gv <= 24) return launch_t<TIn, 24>(a, stream);
  if (gv <= 32) return launch_t<TIn, 32>(a, stream);
  if (gv <= 40) return launch_t<TIn, 40>(a, stream);
  if (gv <= 48) return launch_t<TIn, 48>(a, stream);
  if (gv <= 56) return launch_t<TIn, 56>(a, stream);
  if (gv <= 64) return launch_t<TIn, 64>(a, stream);
  if constexpr (RPL == 4) {
    if (gv <= 96) return launch_t<TIn, 96>(a, stream);
    if (gv <= 128) return launch_t<TIn, 128>(a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  if (a.dtype == LLA_BF16) return dispatch<bf16_t>(a, stream);
  return dispatch<float>(a, stream);
}

}  // namespace lla
