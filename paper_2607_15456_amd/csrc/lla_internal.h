// Internal launch interface between the C ABI (lla_api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lla {

// Decode (and the fp32 causal multi-query path used by prefill).
struct DecodeArgs {
  int dtype;      // LLA_F32 / LLA_BF16: element type of every input
  int out_dtype;  // element type of out
  int B, H, d, rk, rv, n_max, n_ctx;
  int M;       // queries per (b, h): 1 for decode
  int p0;      // causal mode: position of query 0
  int causal;  // 0: decode (N_b from ctx_len / n_ctx); 1: query m attends [0, p0+m]
  int splits;  // workgroups per (b, h, m) along the context
  int waves;   // wavefronts per workgroup (4 or 8)
  int deep;    // 1: at most 2 wavefronts per SIMD, 16-row load batches
  int half;    // 1 (bf16, 4 waves, deep): K groups of 4 pages, two feature rows per load
  int shortk;  // 1 (bf16 decode, not split): wavefronts split the rows of each 8-page group
  const int32_t* ctx_len;
  const void* q;
  const void* ck;
  const void* cv;
  const void* uk;
  const void* uv;
  const void* muv;
  float qscale;  // softmax scale * log2(e)
  void* out;
  float* part;    // [units][splits][rv + 2] split partials (m, l, z)
  uint32_t* cnt;  // [units] arrival counters
  // decoupled rotary branch (dr = 0: none): score += q_r . k_r[n]
  int dr, Hr;      // rotary width; rotary keys per token (1: shared by the heads, or H)
  const void* qr;  // [B][H][M][dr] rotated query parts
  const void* rc;  // [B][Hr][n_max/64][dr][64] rotated keys, paged like the latents
};

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);

struct EncodeArgs {
  int dtype;
  int B, M, H, K;  // K = T * d_head
  int r[2];
  const void* x[2];
  const void* mu[2];
  const void* wdt[2];
  void* c[2];
  int n_max, pos0;
  int sink, window;  // eviction budget: position p goes to slot ring_slot(p) (window 0: slot p)
  int k_token_major;  // 1: the K latents are written token-major (the LLA-2D key cache)
  // Few-token writes with a long K: the K range is split over ksplit
  // workgroups per output tile (ksplit 1: no split, no workspace); part holds
  // the fp32 partial tiles a second launch adds.
  int ksplit;
  float* part;
};

// Split count and workspace size of a few-token write (0 bytes: not split).
int encode_ksplit(int TT, int K);
size_t encode_ws_bytes(int B, int M, int H, int K, int r_k, int r_v);

hipError_t launch_encode(const EncodeArgs& a, hipStream_t stream);

// LLA-2D decode: one latent per token for all heads.
struct Decode2dArgs {
  int out_dtype;
  int B, H, d, rk, rv, n_max, n_ctx, splits;
  const int32_t* ctx_len;
  const void* q;   // [B][H][d]
  const void* ck;  // [B][n_max][rk] token-major
  const void* cv;  // [B][n_max/64][rv][64] paged feature-major
  const void* uk;  // [H][d][rk]
  const void* uv;  // [H][d][rv]
  const void* muv; // [H][d] or null
  float qscale;    // scale * log2(e)
  void* out;       // [B][H][d]
  uint16_t* qt;    // workspace: [B][2][H][rk] absorbed queries (scaled), hi and lo bf16 planes
  float* part;     // workspace: [B][splits][H][rv + 2] partials (m, l, z)
};

hipError_t launch_decode_2d(const Decode2dArgs& a, hipStream_t stream);
int decode_2d_splits(int B, int n_ctx);  // split count the launch uses (also sizes the workspace)

struct PrefillArgs {
  int out_dtype;
  int B, H, M, d, rk, rv, n_max, p0;
  const void* q;
  const void* ck;
  const void* cv;
  const void* uk;
  const void* uv;
  const void* muv;
  float qscale;
  void* out;
  int dr, Hr;  // decoupled rotary branch, as in DecodeArgs (dr = 0: none)
  const void* qr;
  const void* rc;
};

// bf16 MFMA causal prefill.
hipError_t launch_prefill_bf16(const PrefillArgs& a, hipStream_t stream);

// LLA-2D causal prefill: each head's K and V rebuilt into the workspace, then
// attention over them (d_head = 128, bf16).
struct Prefill2dArgs {
  int out_dtype;
  int B, H, M, rk, rv, n_max, p0;
  int nk;           // rebuilt keys per sequence: p0 + M rounded up to a page
  const void* q;    // [B][H][M][128]
  const void* ck;   // [B][n_max][rk] token-major (per head: [B][H][n_max/64][rk][64])
  const void* cv;   // [B][n_max/64][rv][64] paged feature-major (per head: [B][H][...])
  const void* uk;   // [H][128][rk]
  const void* uv;   // [H][128][rv]
  const void* muv;  // [H][128] or null
  float qscale;     // softmax scale * log2(e)
  void* out;        // [B][H][M][128]
  void* kh;         // workspace: [B][H][nk][128] rebuilt keys
  void* vt;         // workspace: [B][H][nk/64][128][64] rebuilt values, feature-major pages
};
size_t prefill_2d_ws_bytes(int B, int H, int n_keys);  // both rebuilt tensors
hipError_t launch_prefill_2d(const Prefill2dArgs& a, hipStream_t stream);
// The same attention over per-head latents (ck, cv paged feature-major per
// (b, h), ranks multiples of 8 up to 512): each head's K and V rebuilt from
// its own latents, then flash2d_kernel.
hipError_t launch_prefill_rebuild(const Prefill2dArgs& a, hipStream_t stream);

// Rotary embedding (half-split) of rows of dr elements.
struct RopeArgs {
  int dtype;
  int B, G, M, dr;     // rows (b, g, m); write: x is [B][M][G][dr], rotate: [B][G][M][dr]
  const void* x;
  const int32_t* pos;  // rotate: per-batch base position (or null: pos0)
  int pos0;
  double base;
  void* y;             // rotate: dense output like x; write: paged cache [B][G][n_max/64][dr][64]
  int n_max;
  int sink, window;    // write: eviction budget as in EncodeArgs
};

hipError_t launch_rope_write(const RopeArgs& a, hipStream_t stream);
hipError_t launch_rope_rotate(const RopeArgs& a, hipStream_t stream);

// Full-RoPE reconstruct-then-attend decode (keys rebuilt and rotated per position).
constexpr int kFullRopeMaxRankK = 256;  // largest r_k of the MFMA kernel
struct FullRopeArgs {
  int dtype, out_dtype;
  int B, H, d, rk, rv, n_max, n_ctx;
  int splits;               // workgroups per (b, h) along the context
  const int32_t* ctx_len;   // [B] or null (n_ctx)
  const int32_t* q_pos;     // [B] query positions or null (N_b - 1)
  const void* q;            // [B][H][d] unrotated queries
  const void* ck;           // paged latents, like the absorbed decode
  const void* cv;
  const void* uk;           // [H][d][rk]
  const void* uv;           // [H][d][rv]
  const void* muk;          // [H][d] or null
  const void* muv;          // [H][d] or null
  double base;              // RoPE base
  float qscale;             // softmax scale * log2(e)
  void* out;                // [B][H][d]
  float* part;              // [B*H][splits][rv + 2] split partials (m, l, z)
  uint32_t* cnt;            // [B*H] arrival counters
};

hipError_t launch_decode_fullrope(const FullRopeArgs& a, hipStream_t stream);
bool fullrope_mfma_ok(int dtype, int d_head, int r_k, int r_v);  // the MFMA kernel takes this shape
int fullrope_occupancy(int r_k, int r_v);  // resident workgroups per compute unit of the MFMA kernel

int device_cu_count();  // compute units of the current device (cached)

}  // namespace lla
