// Loop-l decode attention over the paged latent cache, absorbed form
// (App. J "Absorbed attention"): scores q~ . c_k[n] with q~ = U_k^T q, online
// softmax, z = sum_n a_n c_v[n], out = U_v z + mu_v.  K and V are never
// materialised.
//
// The pass is HBM-bound (about 1 flop per latent byte).  Each wavefront
// streams whole 64-token pages: one 16-byte load per lane covers EPL
// consecutive tokens of one latent feature (the page is feature-major), so a
// wave-wide load reads RPI full 128/256-byte feature rows.  Lane (rg, ts) owns
// feature rows j = k*RPI + rg and token slice ts of every page:
//   * scores: each lane accumulates q~_j * c_k[j][tokens of ts] over its rows,
//     then a 3-step (bf16) xor butterfly over rg completes the dot products;
//   * softmax: per-page max over the wave, running max m, running sum l, with
//     the z accumulators rescaled only when m grows;
//   * values: zacc[k] += sum over the lane's tokens of p_n c_v[j][n]; the
//     reduction over token slices is deferred to the end of the scan.
// The waves of a workgroup interleave pages and merge their (m, l, z) in LDS.
// When the context is split over several workgroups (split-K), each writes its
// merged partial to the workspace and the last to arrive (an agent-scope
// atomic counter) merges all partials and runs the value epilogue
// out = U_v (z / l) + mu_v; the counter is left at zero.
//
// The same kernel serves the fp32 causal prefill: M queries per (b, h), query m
// attending positions [0, p0 + m], one workgroup per query.

#include "lla_device.h"
#include "lla_internal.h"
#include "../../include/lla.h"

namespace lla {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;

template <typename TIn, int GK, int GV>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeArgs a) {
  constexpr int EPL = Elem<TIn>::kPer16B;  // tokens covered by one 16-byte load
  constexpr int LPR = kPage / EPL;         // lanes per 64-token feature row
  constexpr int RPI = kWave / LPR;         // feature rows per wave-wide load

  __shared__ float s_q[kMaxHead];
  __shared__ float s_qt[kMaxRank];
  __shared__ float s_z[kWaves][kMaxRank];
  __shared__ float s_zn[kMaxRank];
  __shared__ float s_m[kWaves], s_l[kWaves];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int bm = blockIdx.x / a.splits, split = blockIdx.x - bm * a.splits, h = blockIdx.y;
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

  // ---- prologue: absorbed query q~ = U_k^T q, scale * log2(e) folded in ----
  const TIn* qp = static_cast<const TIn*>(a.q) + unit * a.d;
  for (int i = tid; i < a.d; i += kThreads) s_q[i] = Elem<TIn>::get(qp, i);
  __syncthreads();
  const TIn* uk = static_cast<const TIn*>(a.uk) + (size_t)h * a.d * a.rk;
  for (int j = tid; j < a.rk; j += kThreads) {
    float acc = 0.f;
    for (int i = 0; i < a.d; ++i) acc = fmaf(Elem<TIn>::get(uk, (size_t)i * a.rk + j), s_q[i], acc);
    s_qt[j] = acc * a.qscale;
  }
  __syncthreads();

  const int rg = lane / LPR, ts = lane - rg * LPR;
  const int rk = a.rk, rv = a.rv;
  float qreg[GK];
#pragma unroll
  for (int k = 0; k < GK; ++k) {
    const int j = k * RPI + rg;
    qreg[k] = (j < rk) ? s_qt[j] : 0.f;
  }
  float zacc[GV];
#pragma unroll
  for (int k = 0; k < GV; ++k) zacc[k] = 0.f;
  float m_run = neg_inf(), l_run = 0.f;

  const TIn* ckb = static_cast<const TIn*>(a.ck) + bh * (size_t)a.n_max * rk + ts * EPL;
  const TIn* cvb = static_cast<const TIn*>(a.cv) + bh * (size_t)a.n_max * rv + ts * EPL;

  // ---- latent scan ----
  for (int p = pb + wave; p < pe; p += kWaves) {
    const TIn* kp = ckb + (size_t)p * kPage * rk;
    float acc[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
#pragma unroll
    for (int k = 0; k < GK; ++k) {
      const int j = k * RPI + rg;
      if (j < rk) {
        float v[EPL];
        Elem<TIn>::unpack(ld16(kp + (size_t)j * kPage), v);
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] = fmaf(qreg[k], v[e], acc[e]);
      }
    }
#pragma unroll
    for (int off = LPR; off < kWave; off <<= 1)
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] += xor_shfl(acc[e], off);

    const int n0 = p * kPage + ts * EPL;
    const bool tail = (p + 1) * kPage > N;
    float mb = neg_inf();
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      if (tail && n0 + e >= N) acc[e] = neg_inf();
      mb = fmaxf(mb, acc[e]);
    }
#pragma unroll
    for (int off = 1; off < LPR; off <<= 1) mb = fmaxf(mb, xor_shfl(mb, off));
    if (mb > m_run) {
      const float alpha = exp2f(m_run - mb);
      l_run *= alpha;
#pragma unroll
      for (int k = 0; k < GV; ++k) zacc[k] *= alpha;
      m_run = mb;
    }
    float pr[EPL];
    float ls = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      pr[e] = exp2f(acc[e] - m_run);
      ls += pr[e];
    }
    l_run += ls;

    const TIn* vp = cvb + (size_t)p * kPage * rv;
#pragma unroll
    for (int k = 0; k < GV; ++k) {
      const int j = k * RPI + rg;
      if (j < rv) {
        float v[EPL];
        Elem<TIn>::unpack(ld16(vp + (size_t)j * kPage), v);
        if (tail) {
#pragma unroll
          for (int e = 0; e < EPL; ++e)
            if (n0 + e >= N) v[e] = 0.f;
        }
        float t = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) t = fmaf(pr[e], v[e], t);
        zacc[k] += t;
      }
    }
  }

  // ---- wave reduction over token slices ----
#pragma unroll
  for (int off = 1; off < LPR; off <<= 1) {
    l_run += xor_shfl(l_run, off);
#pragma unroll
    for (int k = 0; k < GV; ++k) zacc[k] += xor_shfl(zacc[k], off);
  }
  if (ts == 0) {
#pragma unroll
    for (int k = 0; k < GV; ++k) {
      const int j = k * RPI + rg;
      if (j < rv) s_z[wave][j] = zacc[k];
    }
  }
  if (lane == 0) {
    s_m[wave] = m_run;
    s_l[wave] = l_run;
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
    wt[w] = (s_m[w] == neg_inf()) ? 0.f : exp2f(s_m[w] - mg);
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
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      const uint32_t prev =
          __hip_atomic_fetch_add(a.cnt + unit, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == (uint32_t)(a.splits - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    const float* P = a.part + unit * a.splits * stride;
    float ma = neg_inf();
    for (int s = 0; s < a.splits; ++s) ma = fmaxf(ma, P[(size_t)s * stride]);
    float la = 0.f;
    for (int s = 0; s < a.splits; ++s) {
      const float ms = P[(size_t)s * stride];
      const float ws = (ms == neg_inf()) ? 0.f : exp2f(ms - ma);
      la = fmaf(ws, P[(size_t)s * stride + 1], la);
    }
    for (int j = tid; j < rv; j += kThreads) {
      float z = 0.f;
      for (int s = 0; s < a.splits; ++s) {
        const float ms = P[(size_t)s * stride];
        const float ws = (ms == neg_inf()) ? 0.f : exp2f(ms - ma);
        z = fmaf(ws, P[(size_t)s * stride + 2 + j], z);
      }
      s_zn[j] = z / la;
    }
    if (tid == 0) __hip_atomic_store(a.cnt + unit, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();

  // ---- value epilogue: out = U_v z + mu_v (16 lanes per output row) ----
  const TIn* uv = static_cast<const TIn*>(a.uv) + (size_t)h * a.d * rv;
  const TIn* muv = a.muv ? static_cast<const TIn*>(a.muv) + (size_t)h * a.d : nullptr;
  const int sub = lane >> 4, sl = lane & 15;
  for (int i0 = wave * 4; i0 < a.d; i0 += kWaves * 4) {
    const int i = i0 + sub;
    float t = 0.f;
    if (i < a.d)
      for (int j = sl; j < rv; j += 16) t = fmaf(Elem<TIn>::get(uv, (size_t)i * rv + j), s_zn[j], t);
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) t += xor_shfl(t, off);
    if (sl == 0 && i < a.d) {
      if (muv) t += Elem<TIn>::get(muv, i);
      if (bad) t = __builtin_nanf("");
      if (a.out_dtype == LLA_F32)
        static_cast<float*>(a.out)[unit * a.d + i] = t;
      else
        static_cast<bf16_t*>(a.out)[unit * a.d + i] = f32_to_bf16(t);
    }
  }
}

template <typename TIn, int GK, int GV>
hipError_t launch_t(const DecodeArgs& a, hipStream_t stream) {
  dim3 grid(a.B * a.M * a.splits, a.H);
  hipLaunchKernelGGL((decode_kernel<TIn, GK, GV>), grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

int bucket(int g) { return g <= 8 ? 8 : g <= 16 ? 16 : g <= 32 ? 32 : g <= 64 ? 64 : 128; }

template <typename TIn>
hipError_t dispatch(const DecodeArgs& a, hipStream_t stream) {
  constexpr int RPI = kWave / (kPage / Elem<TIn>::kPer16B);
  const int gk = bucket((a.rk + RPI - 1) / RPI);
  const int gv = bucket((a.rv + RPI - 1) / RPI);
#define LLA_CASE(K, V) \
  if (gk == K && gv == V) return launch_t<TIn, K, V>(a, stream);
  LLA_CASE(8, 8) LLA_CASE(8, 16) LLA_CASE(8, 32) LLA_CASE(8, 64)
  LLA_CASE(16, 8) LLA_CASE(16, 16) LLA_CASE(16, 32) LLA_CASE(16, 64)
  LLA_CASE(32, 8) LLA_CASE(32, 16) LLA_CASE(32, 32) LLA_CASE(32, 64)
  LLA_CASE(64, 8) LLA_CASE(64, 16) LLA_CASE(64, 32) LLA_CASE(64, 64)
  if constexpr (RPI == 4) {
    LLA_CASE(8, 128) LLA_CASE(16, 128) LLA_CASE(32, 128) LLA_CASE(64, 128)
    LLA_CASE(128, 8) LLA_CASE(128, 16) LLA_CASE(128, 32) LLA_CASE(128, 64) LLA_CASE(128, 128)
  }
#undef LLA_CASE
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  if (a.dtype == LLA_BF16) return dispatch<bf16_t>(a, stream);
  return dispatch<float>(a, stream);
}

}  // namespace lla
