// Loop-l decode with full RoPE over the paged latent cache: the
// reconstruct-then-attend path (Sec. 3 "RoPE and reconstruction").  The latent
// is fit to the pre-RoPE content projection, so every cached key is rebuilt
// with Eq. 3, K_l[n] = U_k c_k[n] + mu_k, and turned by its position's rotary
// phase; values carry no phase.  The rotation differs from key to key, so the
// key up-projection cannot move to the query side (App. J); the value side
// still can: z = sum_n p_n c_v[n], out = U_v z + mu_v.
//
// Score of key n with the query rotated at p_q (half-split pairs (i, i + 64)
// as complex numbers):  <RoPE(q, p_q), RoPE(k, n)> = <RoPE(q, p_q - n), k>.
// With n = n0 + t (n0 a 32-token tile base) the query weight of token t is
// RoPE(QP, -t), QP = RoPE(q, p_q - n0): QP is formed once per tile (angle in
// double precision), and cos / sin of t * theta_f, the same for every tile,
// are tabulated in LDS once per workgroup.
//
// bf16 kernel (d_head = 128): a workgroup of 8 wavefronts (two per SIMD) takes
// one (b, h) and a range of 64-token pages.  Wavefront w rebuilds rows
// 32m .. 32m + 31 (m = w % 4) of K^T for 32-token tile w / 4 of every page on
// v_mfma_f32_32x32x16_bf16:
//   A = U_k rows 32m + i (staged in LDS once per workgroup),
//   B = the key page, staged in LDS with XOR-swizzled 16-byte chunks and read
//       with ds_read_b64_tr_b16 (lane l gets one token's 4 features),
// so lane (col + 32 g), register r holds K[32m + 8(r/4) + 4g + r%4][token col].
// The lane multiplies its 16 reconstructed features by the rotated query
// weights, the two lane halves and the four M-tiles add their parts (LDS, one
// barrier per page), and every wavefront runs the same online softmax.
// Values: wavefront w owns latent rows [8 VR w, 8 VR (w + 1)) and streams them
// with 16-byte loads of 8 tokens, as in the absorbed decode.  Key pages are
// loaded into registers two pages ahead and written to a two-slot LDS ring;
// value pages are loaded two pages ahead (two register sets alternate).
//
// A plain kernel (one thread per token and feature, reconstruction in fp32)
// serves fp32 inputs and every shape the MFMA kernel does not take.

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
#define LLA_LDS __attribute__((address_space(3)))

constexpr int kFrWaves = 8;  // two per SIMD: wavefront w takes M-tile w % 4 of token tile w / 4
constexpr int kFrThreads = kFrWaves * kWave;
constexpr int kFrD = 128;  // d_head of the MFMA kernel
constexpr double kTwoPi = 6.283185307179586476925286766559;

typedef __amdgpu_buffer_rsrc_t BufRsrc;
__device__ __forceinline__ BufRsrc make_rsrc(const void* base, size_t bytes) {
  const int n = bytes >= 0xffffffffull ? -1 : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}
// Latent pages are read exactly once per call: non-temporal cache policy
// (aux bit 1, "nt"), so they do not displace reusable lines in L2 and the MALL.
constexpr int kCpolNT = 2;
__device__ __forceinline__ uint4 buf_ld16(BufRsrc r, int voff, int soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kCpolNT));
}
__device__ __forceinline__ uint2 lds_tr16(const bf16_t* p) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((LLA_LDS i16x4*)(p)));
}
__device__ __forceinline__ f32x16 mfma32(uint4 a, uint4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                 c, 0, 0, 0);
}

// (cos, sin) of p * theta with the angle formed and reduced in double.
__device__ __forceinline__ void rot_cs(double p, double theta, float& c, float& s) {
  const double ang = p * theta;
  const double r = ang - rint(ang * (1.0 / kTwoPi)) * kTwoPi;
  sincosf((float)r, &s, &c);
}

// Lane exchanges without LDS: DPP within 8-lane groups, permlane32 swap
// across the two wave halves.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
// over lanes 8k .. 8k + 7: quad xor 1, quad xor 2, then mirror within 8 lanes
__device__ __forceinline__ float max8(float x) {
  x = fmaxf(x, dpp<0xB1>(x));
  x = fmaxf(x, dpp<0x4E>(x));
  return fmaxf(x, dpp<0x141>(x));
}
__device__ __forceinline__ float sum8(float x) {
  x += dpp<0xB1>(x);
  x += dpp<0x4E>(x);
  return x + dpp<0x141>(x);
}
// x[lane] + x[lane ^ 32]
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// out[i] = sum_j U_v[i][j] zn[j] + mu_v[i] (zn already normalised), NT
// threads: P consecutive threads share row i and take every P-th column; their
// partial sums combine by xor shuffles in a fixed order.
template <typename T, int NT>
__device__ void fr_epilogue(const FullRopeArgs& a, int h, size_t unit, const float* s_zn, bool bad) {
  const int d = a.d, rv = a.rv;
  const int P = NT / d >= 8 ? 8 : NT / d >= 4 ? 4 : NT / d >= 2 ? 2 : 1;
  const int i = threadIdx.x / P, part = threadIdx.x % P;
  const T* uv = static_cast<const T*>(a.uv) + (size_t)h * d * rv;
  float acc = 0.f;
  if (i < d) {
    const T* row = uv + (size_t)i * rv;
    for (int j = part; j < rv; j += P) acc = fmaf(Elem<T>::get(row, j), s_zn[j], acc);
  }
  for (int off = 1; off < P; off <<= 1) acc += __shfl_xor(acc, off, kWave);
  if (i < d && part == 0) {
    if (a.muv) acc += Elem<T>::get(static_cast<const T*>(a.muv), (size_t)h * d + i);
    if (bad) acc = __builtin_nanf("");
    if (a.out_dtype == LLA_F32)
      static_cast<float*>(a.out)[unit * d + i] = acc;
    else
      static_cast<bf16_t*>(a.out)[unit * d + i] = f32_to_bf16(acc);
  }
}

// ---------------------------------------------------------------------------
// MFMA kernel: bf16, d_head = 128, r_k <= 16 KS, r_v <= 64 VR.
// ---------------------------------------------------------------------------
template <int KS, int VR, bool MU>
__global__ __launch_bounds__(kFrThreads) __attribute__((amdgpu_waves_per_eu(2)))
void fullrope_mfma_kernel(FullRopeArgs a) {
  constexpr int RKP = KS * 16;            // padded key rank (K of the product)
  constexpr int KI = RKP / 8;             // 8-row load instructions per key page
  constexpr int KD = (KI + kFrWaves - 1) / kFrWaves;  // ... per wavefront
  constexpr int kSlot = RKP * kPage;      // bf16 elements of one staged page
  constexpr int US = RKP + 8;             // U_k row stride (bf16): 16-byte reads of 16 rows hit distinct banks
  __shared__ __attribute__((aligned(16))) bf16_t s_k[2 * kSlot];
  __shared__ __attribute__((aligned(16))) bf16_t s_u[kFrD * US];
  // cos / sin of t * theta_f for token offsets t < 32 and the 64 frequencies,
  // [half][t][f - 32 half], each row rotated by 4 (t / 2) floats so that lanes
  // reading different t hit different banks
  __shared__ __attribute__((aligned(16))) float s_cos[2][32][32];
  __shared__ __attribute__((aligned(16))) float s_sin[2][32][32];
  __shared__ __attribute__((aligned(16))) float s_qp[kFrWaves][2][32];  // [wave][re/im][freq] of its tile
  __shared__ __attribute__((aligned(16))) float s_sc[2][4][kPage];      // partial scores per M-tile
  __shared__ float s_z[kMaxRank];
  __shared__ float s_ml[2];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane & 31, g = lane >> 5;
  const int mt = wave & 3, nt = wave >> 2;  // M-tile (32 features of K) and 32-token tile of the page
  const int hi = lane >> 3, lo = lane & 7;  // value phase: row in the 8-row group, token slice
  const int b = blockIdx.x / a.splits, split = blockIdx.x - b * a.splits, h = blockIdx.y;
  const int N = a.ctx_len ? a.ctx_len[b] : a.n_ctx;
  const bool bad = (N < 1) || (N > a.n_ctx);
  const int pages = bad ? 0 : (N + kPage - 1) / kPage;
  const int per = (pages + a.splits - 1) / a.splits;
  const int pb = min(pages, split * per), pe = min(pages, pb + per);
  const int pq = a.q_pos ? a.q_pos[b] : N - 1;
  const size_t bh = (size_t)b * a.H + h;
  const int rk = a.rk, rv = a.rv;

  // Lane (col, g), register r of M-tile mt: feature i = 32 mt + fr(r) with
  // fr(r) = 8 (r/4) + 4 g + r%4, frequency f = i mod 64 = 32 (mt & 1) + fr(r).
  const bool first_half = mt < 2;
  const int hf = mt & 1;
  // query rotation: lane col forms QP for frequency 32 (mt & 1) + col of this
  // wavefront's token tile of every page
  const int fq = 32 * (mt & 1) + col;
  const double theta_q = pow(a.base, -2.0 * fq / kFrD);
  float q1, q2;
  {
    const bf16_t* qp = static_cast<const bf16_t*>(a.q) + bh * kFrD;
    q1 = bf16_to_f32(qp[fq]) * a.qscale;
    q2 = bf16_to_f32(qp[fq + 64]) * a.qscale;
  }
  float mu[16];
  if constexpr (MU) {
    const bf16_t* mk = static_cast<const bf16_t*>(a.muk) + (size_t)h * kFrD + 32 * mt;
#pragma unroll
    for (int r = 0; r < 16; ++r) mu[r] = bf16_to_f32(mk[8 * (r / 4) + 4 * g + r % 4]);
  }

  // ---- buffers over this (b, h)'s latents ----
  const BufRsrc ksrc = make_rsrc(static_cast<const bf16_t*>(a.ck) + bh * (size_t)a.n_max * rk,
                                 (size_t)a.n_max * rk * 2);
  const BufRsrc vsrc = make_rsrc(static_cast<const bf16_t*>(a.cv) + bh * (size_t)a.n_max * rv,
                                 (size_t)a.n_max * rv * 2);
  const int kpage = kPage * rk * 2, vpage = kPage * rv * 2;  // bytes per page
  // key loads: instruction k = wave + 8 u covers page rows 8k .. 8k+7; lane ->
  // row 8k + lane/8, 16-byte chunk lane%8 (one contiguous KB per instruction)
  const int krow = lane >> 3;
  const int kswz = ((lane >> 4) & 1) << 2;                            // chunk XOR of row 8k + krow
  const int kdst = krow * kPage + (((lane & 7) ^ kswz) << 3);          // LDS element offset in the row block
  // transposed reads: lane (x16 = lane % 16, G = lane / 16) of tile nt reads
  // rows 16 s + 8 g + 4 e2 + x16/4, tokens 32 nt + 16 (G % 2) + 4 (x16 % 4) .. +3
  const int x16 = lane & 15, th = (lane >> 4) & 1, sw1 = (x16 >> 3) & 1;
  const int cl = 2 * th + ((x16 & 3) >> 1);
  const int troff = (8 * g + (x16 >> 2)) * kPage + ((4 * (nt ^ sw1) + cl) << 3) + 4 * (x16 & 1);
  // value rows of this wavefront: 8 VR wave + 8 k + hi, tokens 8 lo .. 8 lo + 7
  const int vrow0 = 8 * VR * wave;

  // Two register sets of key and value loads alternate between even and odd
  // pages, so every load is issued two pages before it is used.
  uint4 kA[KD], kB[KD], vA[VR], vB[VR];
  // A lane whose row is past r_k reads row r_k - 1 instead (every address
  // stays inside the page's r_k rows); rows past r_k are stored as zeros.  The
  // loaded registers are not touched until they are stored, so no wait is
  // needed before the next page's loads are issued.
  // Every lane issues every load (instructions wholly past r_k re-read the
  // last rows), so the compiler's waits count loads exactly.
  // A prefetch of a page past the range (p >= pe, uniform) takes a vector
  // offset at the end of the (b, h) buffer: the raw buffer load is out of
  // range, returns zeros and reads no memory, and still counts as a load for
  // the wait counters.  Those registers are never consumed.
  const int k_oob = a.n_max * rk * 2, v_oob = a.n_max * rv * 2;
  auto kload = [&](uint4 (&kr)[KD], int p) {
    const bool past = p >= pe;
#pragma unroll
    for (int u = 0; u < KD; ++u) {
      const int k8 = min(8 * (wave + kFrWaves * u), (rk - 1) & ~7);  // first row of the instruction
      const int voff = (min(k8 + krow, rk - 1) - k8) * (kPage * 2) + (lane & 7) * 16;
      kr[u] = buf_ld16(ksrc, past ? k_oob : voff, past ? 0 : p * kpage + k8 * kPage * 2);
    }
  };
  auto kstore = [&](const uint4 (&kr)[KD], int slot) {
#pragma unroll
    for (int u = 0; u < KD; ++u) {
      const int k = wave + kFrWaves * u;
      if (k < KI) {  // uniform
        const bool live = 8 * k + krow < rk;
        *reinterpret_cast<uint4*>(&s_k[slot * kSlot + 8 * k * kPage + kdst]) = live ? kr[u] : uint4{0, 0, 0, 0};
      }
    }
  };
  // A lane whose row is past r_v reads row r_v - 1 (never used); every lane
  // issues every load, as for the keys.
  auto vload = [&](uint4 (&vr)[VR], int p) {
    const bool past = p >= pe;
#pragma unroll
    for (int k = 0; k < VR; ++k) {
      const int j0 = min(vrow0 + 8 * k, rv - 1);
      const int voff = (min(vrow0 + 8 * k + hi, rv - 1) - j0) * (kPage * 2) + lo * 16;
      vr[k] = buf_ld16(vsrc, past ? v_oob : voff, past ? 0 : p * vpage + j0 * kPage * 2);
    }
  };

  float zacc[VR];
#pragma unroll
  for (int k = 0; k < VR; ++k) zacc[k] = 0.f;
  float m_run = neg_inf(), l_lane = 0.f;
  // softmax weights of the last scored page and its rescale factor; its value
  // products run at the start of the next page
  float pr[8], alpha = 1.f;

  // z[row] = alpha z[row] + sum over the lane's 8 tokens of pr * value; on the
  // context's last page, value slots past N (which may hold anything) are zeroed
  auto vconsume = [&](const uint4 (&vr)[VR], int p) {
#pragma unroll
    for (int k = 0; k < VR; ++k) zacc[k] *= alpha;
    const int nv = N - (p * kPage + 8 * lo);  // valid tokens of this lane's slice
    if ((p + 1) * kPage > N) {  // uniform
      uint32_t keep[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) keep[i] = nv > 2 * i + 1 ? 0xffffffffu : nv > 2 * i ? 0x0000ffffu : 0u;
#pragma unroll
      for (int k = 0; k < VR; ++k) {
        if (vrow0 + 8 * k < rv) {  // uniform
          const uint4 w = uint4{vr[k].x & keep[0], vr[k].y & keep[1], vr[k].z & keep[2], vr[k].w & keep[3]};
          float v[8];
          Elem<bf16_t>::unpack(w, v);
          float t = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) t = fmaf(pr[e], v[e], t);
          zacc[k] += t;
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < VR; ++k) {
        if (vrow0 + 8 * k < rv) {  // uniform
          float v[8];
          Elem<bf16_t>::unpack(vr[k], v);
          float t = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) t = fmaf(pr[e], v[e], t);
          zacc[k] += t;
        }
      }
    }
  };

  // Page p = pb + i.  Set (i + 1) % 2 of the key and value registers holds
  // page p + 1's keys and page p - 1's values on entry: the keys go to LDS and
  // page p + 3's are requested, the values are multiplied and page p + 1's
  // requested -- all before this page's products, so two pages of keys and of
  // values stay in flight while the wavefront computes.  Past the last page
  // the loads are issued out of range (zeros, no memory read): every load is
  // issued, so the waits count exactly.
  auto body = [&](int i, uint4 (&kr)[KD], uint4 (&vr)[VR]) {
    const int p = pb + i, slot = i & 1;
    kstore(kr, slot ^ 1);
    kload(kr, p + 3);
    if (i > 0) vconsume(vr, p - 1);
    vload(vr, p + 1);
    // ---- rotated query of this wavefront's token tile ----
    {
      float c, sn;
      rot_cs((double)pq - (double)(p * kPage + 32 * nt), theta_q, c, sn);
      s_qp[wave][0][col] = q1 * c - q2 * sn;  // both lane halves write the same value
      s_qp[wave][1][col] = q2 * c + q1 * sn;
    }
    // ---- K^T rows 32 mt .. +31 of token tile nt ----
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = MU ? mu[r] : 0.f;
    const bf16_t* kb = &s_k[slot * kSlot];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const uint4 ua = *reinterpret_cast<const uint4*>(&s_u[(32 * mt + col) * US + 16 * s + 8 * g]);
      const uint2 r0 = lds_tr16(kb + troff + 16 * s * kPage);
      const uint2 r1 = lds_tr16(kb + troff + (16 * s + 4) * kPage);
      acc = mfma32(ua, uint4{r0.x, r0.y, r1.x, r1.y}, acc);
    }
    wave_sync();
    // ---- rotated dot products: this lane's 16 features of token col ----
    float cs_c[16], cs_s[16];
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) {
      const int f0 = (8 * a4 + 4 * g + 4 * (col >> 1)) & 31;
      const float4 c4 = *reinterpret_cast<const float4*>(&s_cos[hf][col][f0]);
      const float4 s4 = *reinterpret_cast<const float4*>(&s_sin[hf][col][f0]);
      cs_c[4 * a4] = c4.x; cs_c[4 * a4 + 1] = c4.y; cs_c[4 * a4 + 2] = c4.z; cs_c[4 * a4 + 3] = c4.w;
      cs_s[4 * a4] = s4.x; cs_s[4 * a4 + 1] = s4.y; cs_s[4 * a4 + 2] = s4.z; cs_s[4 * a4 + 3] = s4.w;
    }
    float sum = 0.f;
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) {
      const float4 p1 = *reinterpret_cast<const float4*>(&s_qp[wave][0][8 * a4 + 4 * g]);
      const float4 p2 = *reinterpret_cast<const float4*>(&s_qp[wave][1][8 * a4 + 4 * g]);
      const float x1[4] = {p1.x, p1.y, p1.z, p1.w}, x2[4] = {p2.x, p2.y, p2.z, p2.w};
#pragma unroll
      for (int b4 = 0; b4 < 4; ++b4) {
        const int r = 4 * a4 + b4;
        const float w = first_half ? fmaf(x1[b4], cs_c[r], x2[b4] * cs_s[r])
                                   : fmaf(x2[b4], cs_c[r], -(x1[b4] * cs_s[r]));
        sum = fmaf(w, acc[r], sum);
      }
    }
    sum = sum_halves(sum);  // M-tile mt's part of the score of token 32 nt + col
    if (g == 0) s_sc[slot][mt][32 * nt + col] = sum;
    __syncthreads();

    // ---- softmax over the page: lane (hi, lo) holds tokens 8 lo .. 8 lo + 7 ----
    float sc[8];
#pragma unroll
    for (int e = 0; e < 8; e += 4) {
      float4 t = *reinterpret_cast<const float4*>(&s_sc[slot][0][8 * lo + e]);
#pragma unroll
      for (int w = 1; w < 4; ++w) {
        const float4 u = *reinterpret_cast<const float4*>(&s_sc[slot][w][8 * lo + e]);
        t.x += u.x;
        t.y += u.y;
        t.z += u.z;
        t.w += u.w;
      }
      sc[e] = t.x;
      sc[e + 1] = t.y;
      sc[e + 2] = t.z;
      sc[e + 3] = t.w;
    }
    const int n0 = p * kPage + 8 * lo;
    float mx = neg_inf();
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (n0 + e >= N) sc[e] = neg_inf();
      mx = fmaxf(mx, sc[e]);
    }
    mx = max8(mx);
    alpha = 1.f;
    if (mx > m_run) {
      alpha = __builtin_amdgcn_exp2f(m_run - mx);
      l_lane *= alpha;
      m_run = mx;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pr[e] = __builtin_amdgcn_exp2f(sc[e] - m_run);  // exp2(-inf) = 0 past N
      l_lane += pr[e];
    }
  };

  // Prologue: page pb's keys into slot 0; keys of pb + 1 in set B, pb + 2 in
  // set A; values of pb in set A (set B is loaded by the first page).
  // The first pages are requested before U_k and the rotation table are
  // staged, so their latency overlaps the staging.
  if (pb < pe) {
    kload(kA, pb);
    kload(kB, pb + 1);
    vload(vA, pb);
  }
  // ---- U_k of head h into LDS (rows = features of K, columns past r_k zero) ----
  {
    const bf16_t* uk = static_cast<const bf16_t*>(a.uk) + (size_t)h * kFrD * rk;
    constexpr int C8 = US / 8;  // 16-byte chunks per LDS row
    for (int e = tid; e < kFrD * C8; e += kFrThreads) {
      const int i = e / C8, j0 = 8 * (e - i * C8);
      uint4 v;
      if ((rk & 7) == 0) {
        v = j0 < rk ? *reinterpret_cast<const uint4*>(uk + (size_t)i * rk + j0) : uint4{0, 0, 0, 0};
      } else {
        uint32_t w[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const uint32_t x0 = j0 + 2 * x < rk ? uk[(size_t)i * rk + j0 + 2 * x] : 0u;
          const uint32_t x1 = j0 + 2 * x + 1 < rk ? uk[(size_t)i * rk + j0 + 2 * x + 1] : 0u;
          w[x] = x0 | (x1 << 16);
        }
        v = uint4{w[0], w[1], w[2], w[3]};
      }
      *reinterpret_cast<uint4*>(&s_u[i * US + j0]) = v;
    }
    // the thread's frequencies are fr = tid % 32 and 32 + fr for every e
    static_assert(kFrThreads % 32 == 0, "");
    const double th0 = pow(a.base, -2.0 * (tid & 31) / kFrD), th1 = pow(a.base, -2.0 * (32 + (tid & 31)) / kFrD);
    for (int e = tid; e < 2 * 32 * 32; e += kFrThreads) {
      const int hf = e >> 10, t = (e >> 5) & 31, fr = e & 31;
      float c, sn;
      rot_cs((double)t, hf ? th1 : th0, c, sn);
      s_cos[hf][t][(fr + 4 * (t >> 1)) & 31] = c;
      s_sin[hf][t][(fr + 4 * (t >> 1)) & 31] = sn;
    }
  }
  if (pb < pe) {
    kstore(kA, 0);
    kload(kA, pb + 2);
  }
  __syncthreads();
  const int npg = pe - pb;
  int i = 0;
  for (; i + 1 < npg; i += 2) {
    body(i, kB, vB);
    body(i + 1, kA, vA);
  }
  if (i < npg) {
    body(i, kB, vB);
    vconsume(vA, pe - 1);  // npg odd: the last page's values are in set A
  } else if (npg > 0) {
    vconsume(vB, pe - 1);  // npg even: in set B
  }

  // ---- reductions: z over token slices, l over token slices ----
  l_lane = sum8(l_lane);
#pragma unroll
  for (int k = 0; k < VR; ++k) zacc[k] = sum8(zacc[k]);
  if (lo == 0) {
#pragma unroll
    for (int k = 0; k < VR; ++k) {
      const int j = vrow0 + 8 * k + hi;
      if (j < rv) s_z[j] = zacc[k];
    }
  }
  if (tid == 0) {
    s_ml[0] = m_run;
    s_ml[1] = l_lane;
  }
  __syncthreads();

  const size_t unit = bh;
  if (a.splits == 1) {
    const float inv = 1.0f / s_ml[1];
    for (int j = tid; j < rv; j += kFrThreads) s_z[j] *= inv;
  } else {
    const int stride = rv + 2;
    float* part = a.part + (unit * a.splits + split) * stride;
    for (int j = tid; j < rv; j += kFrThreads) part[2 + j] = s_z[j];
    if (tid == 0) {
      part[0] = s_ml[0];
      part[1] = s_ml[1];
    }
    // every wavefront's partial stores reach L2 before the barrier; thread
    // 0's counter update is the workgroup's one agent-scope release (one L2
    // write-back), and the last arrival's acquire makes every split's partial
    // visible
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
      la = fmaf(ms == neg_inf() ? 0.f : __builtin_amdgcn_exp2f(ms - ma), P[(size_t)s * stride + 1], la);
    }
    __syncthreads();
    for (int j = tid; j < rv; j += kFrThreads) {
      float z = 0.f;
      for (int s = 0; s < a.splits; ++s) {
        const float ms = P[(size_t)s * stride];
        z = fmaf(ms == neg_inf() ? 0.f : __builtin_amdgcn_exp2f(ms - ma), P[(size_t)s * stride + 2 + j], z);
      }
      s_z[j] = z / la;
    }
    if (tid == 0) __hip_atomic_store(a.cnt + unit, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  fr_epilogue<bf16_t, kFrThreads>(a, h, unit, s_z, bad);
}

// ---------------------------------------------------------------------------
// Plain kernel: one workgroup per (b, h), 32-token chunks.  K is rebuilt into
// LDS in fp32 (one thread per (token, feature)), each of 32 threads rotates
// the query to its key's position and takes the dot product, then the chunk
// joins the online softmax and the latent-space value sum.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void fullrope_plain_kernel(FullRopeArgs a) {
  constexpr int kChunk = 32;
  __shared__ float s_q[kMaxHead];
  __shared__ double s_theta[kMaxHead / 2];
  __shared__ float s_key[kChunk * kMaxHead];
  __shared__ float s_sc[kChunk];
  __shared__ float s_z[kMaxRank];
  const int tid = threadIdx.x, b = blockIdx.x, h = blockIdx.y;
  const int d = a.d, half = d / 2, rk = a.rk, rv = a.rv;
  const int N = a.ctx_len ? a.ctx_len[b] : a.n_ctx;
  const bool bad = (N < 1) || (N > a.n_ctx);
  const int n_end = bad ? 0 : N;
  const int pq = a.q_pos ? a.q_pos[b] : N - 1;
  const size_t bh = (size_t)b * a.H + h;
  const T* q = static_cast<const T*>(a.q) + bh * d;
  for (int i = tid; i < d; i += 256) s_q[i] = Elem<T>::get(q, i) * a.qscale;
  for (int f = tid; f < half; f += 256) s_theta[f] = pow(a.base, -2.0 * f / d);
  const T* ck = static_cast<const T*>(a.ck) + bh * (size_t)a.n_max * rk;
  const T* cv = static_cast<const T*>(a.cv) + bh * (size_t)a.n_max * rv;
  const T* uk = static_cast<const T*>(a.uk) + (size_t)h * d * rk;
  const T* mk = a.muk ? static_cast<const T*>(a.muk) + (size_t)h * d : nullptr;
  // paged feature-major element (n, j) of a rank-r cache
  auto at = [](int n, int j, int r) { return (size_t)(n / kPage) * kPage * r + (size_t)j * kPage + n % kPage; };
  float z[2] = {0.f, 0.f};
  float m_run = neg_inf(), l_run = 0.f;
  __syncthreads();
  for (int n0 = 0; n0 < n_end; n0 += kChunk) {
    for (int e = tid; e < kChunk * d; e += 256) {
      const int t = e % kChunk, i = e / kChunk, n = n0 + t;
      float k = 0.f;
      if (n < N) {
        for (int j = 0; j < rk; ++j) k = fmaf(Elem<T>::get(uk, (size_t)i * rk + j), Elem<T>::get(ck, at(n, j, rk)), k);
        if (mk) k += Elem<T>::get(mk, i);
      }
      s_key[t * d + i] = k;
    }
    __syncthreads();
    if (tid < kChunk) {
      const int n = n0 + tid;
      float s = neg_inf();
      if (n < N) {
        s = 0.f;
        for (int f = 0; f < half; ++f) {
          float c, sn;
          rot_cs((double)pq - (double)n, s_theta[f], c, sn);
          const float w1 = s_q[f] * c - s_q[f + half] * sn, w2 = s_q[f + half] * c + s_q[f] * sn;
          s = fmaf(w1, s_key[tid * d + f], fmaf(w2, s_key[tid * d + f + half], s));
        }
      }
      s_sc[tid] = s;
    }
    __syncthreads();
    float cm = neg_inf();
    for (int t = 0; t < kChunk; ++t) cm = fmaxf(cm, s_sc[t]);
    const float mn = fmaxf(m_run, cm);
    const float alpha = m_run == neg_inf() ? 0.f : exp2f(m_run - mn);
    float ls = 0.f;
    for (int t = 0; t < kChunk; ++t) ls += s_sc[t] == neg_inf() ? 0.f : exp2f(s_sc[t] - mn);
    l_run = l_run * alpha + ls;
    for (int u = 0; u < 2; ++u) {
      const int j = tid + 256 * u;
      if (j < rv) {
        float acc = z[u] * alpha;
        for (int t = 0; t < kChunk && n0 + t < N; ++t)
          acc = fmaf(exp2f(s_sc[t] - mn), Elem<T>::get(cv, at(n0 + t, j, rv)), acc);
        z[u] = acc;
      }
    }
    m_run = mn;
    __syncthreads();
  }
  for (int u = 0; u < 2; ++u) {
    const int j = tid + 256 * u;
    if (j < rv) s_z[j] = z[u] / l_run;
  }
  __syncthreads();
  fr_epilogue<T, 256>(a, h, bh, s_z, bad);
}

template <int KS, int VR>
hipError_t launch_mfma(const FullRopeArgs& a, hipStream_t stream) {
  const dim3 grid(a.B * a.splits, a.H);
  if (a.muk)
    hipLaunchKernelGGL((fullrope_mfma_kernel<KS, VR, true>), grid, dim3(kFrThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((fullrope_mfma_kernel<KS, VR, false>), grid, dim3(kFrThreads), 0, stream, a);
  return hipGetLastError();
}

// Template buckets: K-steps of 16 key features, 8-row value groups per wavefront.
int ks_bucket(int r_k) {
  const int ks = (r_k + 15) / 16;
  return ks <= 2 ? 2 : ks <= 4 ? 4 : ks <= 6 ? 6 : ks <= 8 ? 8 : ks <= 10 ? 10 : ks <= 12 ? 12 : 16;
}
int vr_bucket(int r_v) {
  const int vr = (r_v + 8 * kFrWaves - 1) / (8 * kFrWaves);  // 8-row value groups per wavefront
  return vr <= 1 ? 1 : vr <= 2 ? 2 : vr <= 3 ? 3 : vr <= 4 ? 4 : vr <= 5 ? 5 : vr <= 6 ? 6 : 8;
}

template <int KS>
hipError_t launch_vr(const FullRopeArgs& a, hipStream_t stream) {
  switch (vr_bucket(a.rv)) {
    case 1: return launch_mfma<KS, 1>(a, stream);
    case 2: return launch_mfma<KS, 2>(a, stream);
    case 3: return launch_mfma<KS, 3>(a, stream);
    case 4: return launch_mfma<KS, 4>(a, stream);
    case 5: return launch_mfma<KS, 5>(a, stream);
    case 6: return launch_mfma<KS, 6>(a, stream);
    default: return launch_mfma<KS, 8>(a, stream);
  }
}

}  // namespace

bool fullrope_mfma_ok(int dtype, int d_head, int r_k, int r_v) {
  return dtype == LLA_BF16 && d_head == kFrD && r_k <= kFullRopeMaxRankK && r_v <= kMaxRank;
}

int fullrope_occupancy(int r_k, int r_v) {
  (void)r_k;
  (void)r_v;
  return 1;  // one 8-wavefront workgroup per compute unit
}

hipError_t launch_decode_fullrope(const FullRopeArgs& a, hipStream_t stream) {
  if (!fullrope_mfma_ok(a.dtype, a.d, a.rk, a.rv)) {
    const dim3 grid(a.B, a.H);
    if (a.dtype == LLA_BF16)
      hipLaunchKernelGGL(fullrope_plain_kernel<bf16_t>, grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL(fullrope_plain_kernel<float>, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
  }
  switch (ks_bucket(a.rk)) {
    case 2: return launch_vr<2>(a, stream);
    case 4: return launch_vr<4>(a, stream);
    case 6: return launch_vr<6>(a, stream);
    case 8: return launch_vr<8>(a, stream);
    case 10: return launch_vr<10>(a, stream);
    case 12: return launch_vr<12>(a, stream);
    default: return launch_vr<16>(a, stream);
  }
}

}  // namespace lla
