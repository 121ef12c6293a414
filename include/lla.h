/*
 * lla.h -- C ABI of the Looped Latent Attention (LLA) latent-cache library for
 * AMD Instinct MI355X (gfx950).
 *
 * LLA (arxiv 2607.15456) stores the KV cache of a weight-tied looped
 * transformer (T recurrence steps over one stack of D layers, H heads of width
 * d_head) as one low-rank latent per (layer, head, token) and axis that
 * jointly covers all T loops:
 *
 *   x   = [x_1; ...; x_T]            loop-stacked teacher K or V   (Sec. 3, Eq. 1)
 *   c   = (x - mu) W_down            latent of rank r              (Sec. 3, Eq. 2)
 *   x_t = c W_up,t^T + mu_t          loop-t reconstruction         (Sec. 3, Eq. 3)
 *   rho = 2 T d_head / (r_k + r_v)   exact compression ratio       (Sec. 3, Eq. 4)
 *
 * The attention entry points never materialise K or V.  They use the absorbed
 * form of App. J ("Absorbed attention"): scores q^T (W^K_up c) are computed as
 * (W^K_up^T q)^T c, and the value path sum_n a_n W^V_up c_n as
 * W^V_up (sum_n a_n c_n).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Loop indices are 0-based; the caller passes the loop-l parameters.
 * - All tensor arguments are DEVICE pointers owned by the caller, row-major,
 *   dense, and 16-byte aligned.  The library keeps no pointer after a call
 *   returns, allocates no memory and never synchronises: it only enqueues
 *   kernels on `stream` (a hipStream_t; NULL means the default stream).
 *   Outputs are valid once the stream has reached that point.
 * - Every entry point validates all scalar arguments and pointers on the host
 *   before launching anything.  On any error nothing is launched and no
 *   output is touched.  NaN/Inf in the data are not checked: a non-finite
 *   value in data an output depends on makes that output non-finite, and
 *   cache slots a call does not attend are never read into a result.  The
 *   prefills add one exception, stated with lla_prefill_attn.
 * - dtype arguments take lla_dtype values.  "dtype" is the element type of
 *   every input tensor of the call (queries, latents, projections, means);
 *   accumulation is always fp32.
 * - The attention calls address one latent region with 32-bit byte offsets:
 *   n_max * r * (element bytes) must be below 2^31 for every cache they read
 *   (r = r_k, r_v or d_rope; one region is one (b, h) of a per-head cache,
 *   one sequence of an LLA-2D cache), else LLA_ERR_UNSUPPORTED.
 * - Calls are stateless and reentrant.  Calls that share a workspace or write
 *   the same cache region must be ordered by the caller (same stream).
 *
 * Latent cache layout (one buffer per layer and axis)
 * ---------------------------------------------------
 * A cache of capacity n_max tokens and rank r for B sequences and H heads
 * holds B*H*n_max*r elements.  Tokens are grouped in pages of
 * LLA_PAGE_TOKENS = 64 consecutive positions; inside a page the latent is
 * stored feature-major, so that one feature of 64 consecutive tokens is
 * contiguous:
 *
 *   element (b, h, token n, feature j) lives at index
 *     ((b*H + h) * n_max + (n/64)*64) * r  +  j*64  +  (n % 64)
 *
 * i.e. logical c[b][h][n][j] is stored as c[b][h][n/64][j][n%64].  n_max must
 * be a multiple of 64.  The stored scalar count is exactly (r_k + r_v) per
 * (head, token) per layer, so Eq. 4 holds for the resident cache.
 */
#ifndef LLA_H_
#define LLA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LLA_ABI_VERSION 10
#define LLA_PAGE_TOKENS 64
#define LLA_MAX_RANK 512
#define LLA_MAX_ROPE 256
#define LLA_MAX_RANK_2D 1024
#define LLA_MAX_SPLITS 64
#define LLA_NOALLOC_SCRATCH_BYTES (4u << 20) /* static scratch per device of lla_decode_attn_noalloc */

typedef enum lla_status {
  LLA_OK = 0,
  LLA_ERR_INVALID_ARG = 1, /* a size, pointer, alignment or value is invalid */
  LLA_ERR_UNSUPPORTED = 2, /* valid in the paper's terms, not supported here */
  LLA_ERR_WORKSPACE = 3,   /* the decode workspace is missing or too small  */
  LLA_ERR_HIP = 4,         /* the HIP runtime reported an error on launch    */
  LLA_ERR_SCRATCH = 5      /* lla_decode_attn_noalloc: more than its static scratch */
} lla_status;

typedef enum lla_dtype {
  LLA_F32 = 0,  /* IEEE binary32 */
  LLA_BF16 = 1  /* bfloat16 (round-to-nearest-even wherever the library rounds) */
} lla_dtype;

/* Static, NUL-terminated description of a status code (never NULL). */
const char* lla_status_string(int status);

/* LLA_ABI_VERSION of the built library. */
int lla_abi_version(void);

/*
 * Exact compression ratio, Sec. 3 Eq. 4: rho = 2*T*d_head / (r_k + r_v),
 * returned as the reduced fraction num/den.  Host only.
 * Errors: LLA_ERR_INVALID_ARG if any size is <= 0 or an output pointer is NULL.
 */
lla_status lla_rho(int64_t T, int64_t d_head, int64_t r_k, int64_t r_v,
                   int64_t* num, int64_t* den);

/*
 * Bytes of a `layers`-layer KV cache holding `tokens` tokens (Sec. 3, the
 * "Teacher cache" and "Cross-loop codec" paragraphs; tab:memory):
 *   latent == 0 (teacher): layers * 2*T*heads*d_head * elem_bytes * tokens
 *   latent != 0 (LLA):     layers * (r_k + r_v)*heads * elem_bytes * tokens
 * Host only.  Errors: LLA_ERR_INVALID_ARG for non-positive sizes (tokens may
 * be 0), a NULL output, or a result that overflows int64.
 */
lla_status lla_cache_bytes(int64_t layers, int64_t heads, int64_t T, int64_t d_head,
                           int64_t r_k, int64_t r_v, int64_t tokens, int64_t elem_bytes,
                           int latent, int64_t* bytes);

/*
 * Encode / cache write, Sec. 3 Eq. 2 (with Eq. 1's loop-major stacking):
 *   c[b][h][pos0+m][:] = (x[b][m][h][:] - mu[h][:]) W_down[h]
 * for both axes (K with rank r_k, V with rank r_v), every sequence b < B,
 * new token m < M and head h < H.
 *
 *   x_k, x_v   [B][M][H][T*d_head]  loop-stacked K/V of the new tokens
 *                                    (element i = l*d_head + e is loop l,
 *                                    channel e)
 *   mu_k, mu_v [H][T*d_head] or NULL (NULL means a zero mean)
 *   wdt_k      [H][r_k][T*d_head]   W_down^T for K, one per head
 *   wdt_v      [H][r_v][T*d_head]   W_down^T for V
 *   c_k, c_v   latent caches in the paged layout above, capacity n_max
 *
 * All inputs and both caches have element type `dtype`.  Results are rounded
 * once, from the fp32 accumulator, to the cache type (RNE for bf16).  Cache
 * slots outside [pos0, pos0+M) are not touched.
 * Requires B, M, H, T >= 1; d_head a multiple of 32 in [32, 256];
 * 1 <= r_k, r_v <= LLA_MAX_RANK; n_max a multiple of 64; pos0 >= 0 and
 * pos0 + M <= n_max.
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_HIP.
 */
lla_status lla_encode(int dtype, int B, int M, int H, int T, int d_head, int r_k, int r_v,
                      const void* x_k, const void* x_v, const void* mu_k, const void* mu_v,
                      const void* wdt_k, const void* wdt_v, void* c_k, void* c_v,
                      int n_max, int pos0, void* stream);

/*
 * Workspace bytes lla_decode_attn needs to split the context of every
 * (b, h) across workgroups (split-K) for these sizes.  Depends only on the
 * arguments.  Host only.  Errors: LLA_ERR_INVALID_ARG.
 */
lla_status lla_decode_workspace_bytes(int B, int H, int r_v, int n_ctx, size_t* bytes);

/*
 * Number of workgroups lla_decode_attn and lla_decode_attn_rope split the
 * context of every (b, h) over for these sizes on the current device, with a
 * workspace (with_workspace != 0) or without one (then always 1).  Splitting
 * is chosen only when the (b, h) units alone leave compute units without 8
 * resident wavefronts (small batches, long contexts); the partial softmax
 * states (m, l, z) of the splits are merged as in the split-K step of the
 * decode (the softmax over a union of disjoint key ranges).  The ranks r_k,
 * r_v and the rotary width d_rope (0 without the rotary branch) are those of
 * the call: at large ranks bf16 contexts are split into longer slices.
 * Host only.  Errors: LLA_ERR_INVALID_ARG (also for ranks outside
 * [1, LLA_MAX_RANK] or d_rope outside [0, LLA_MAX_ROPE]).
 */
lla_status lla_decode_splits(int dtype, int B, int H, int n_ctx, int r_k, int r_v, int d_rope,
                             int with_workspace, int* splits);

/*
 * Loop-l decode attention over the latent cache, absorbed form (App. J):
 *   q~    = U_k^T q                                  [r_k]
 *   s_n   = scale * (q~ . c_k[n] + q . mu_k)         n < N_b
 *   a     = softmax(s)
 *   out   = U_v (sum_n a_n c_v[n]) + mu_v            [d_head]
 * which equals the teacher's attention over the Eq. 3 reconstructions
 * K_l[n] = U_k c_k[n] + mu_k, V_l[n] = U_v c_v[n] + mu_v.  The q . mu_k term
 * is the same for every n, so it cancels inside the softmax; the kernels do
 * not compute it (the result is the same in exact arithmetic).
 *
 *   q          [B][H][d_head]       loop-l queries
 *   c_k, c_v   latent caches (paged layout), ranks r_k / r_v, capacity n_max
 *   u_k        [H][d_head][r_k]     W^K_up,l  (Eq. 3's W_up,t for this loop)
 *   u_v        [H][d_head][r_v]     W^V_up,l
 *   mu_k, mu_v [H][d_head] or NULL  loop-l slices mu_t of the means
 *   ctx_len    device int32 [B] or NULL: N_b, the number of cached tokens
 *              sequence b attends (positions [0, N_b)); NULL means N_b = n_ctx
 *              for every b.  An entry outside [1, n_ctx] makes that
 *              sequence's outputs NaN.
 *   scale      softmax scale (the teacher's is 1/sqrt(d_head)); finite, > 0
 *   out        [B][H][d_head] of out_dtype (LLA_F32 or LLA_BF16)
 *   workspace  device buffer of ws_bytes >= lla_decode_workspace_bytes(), or
 *              NULL with ws_bytes == 0 (the context is then not split across
 *              workgroups).  Its first 4*B*H bytes are arrival counters that
 *              must be zero before the first call (zero the buffer once after
 *              allocating it); every call leaves them zero again.
 *
 * Requires 1 <= n_ctx <= n_max, n_max a multiple of 64, d_head a multiple of
 * 32 in [32, 256], 1 <= r_k, r_v <= LLA_MAX_RANK.
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_WORKSPACE, LLA_ERR_HIP.
 */
lla_status lla_decode_attn(int dtype, int out_dtype, int B, int H, int d_head, int r_k, int r_v,
                           int n_max, int n_ctx, const int32_t* ctx_len, const void* q,
                           const void* c_k, const void* c_v, const void* u_k, const void* u_v,
                           const void* mu_k, const void* mu_v, float scale, void* out,
                           void* workspace, size_t ws_bytes, void* stream);

/*
 * lla_decode_attn for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * arguments without the workspace, the same kernels, launch shape and
 * results.  When the context is split across workgroups, the arrival counters
 * and partial softmax states live in a static device array of
 * LLA_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends; the call clears the counters with a fill kernel
 * (no memset node) and never calls an allocating routine.  Every call on one
 * GPU shares that GPU's array and it keeps the last call's contents: calls
 * that may overlap on one GPU (different streams, or threads) race and must
 * be ordered by the caller.  The first call on a device resolves the array's
 * address (hipGetSymbolAddress).
 * Errors: as lla_decode_attn, and LLA_ERR_SCRATCH when the split the launch
 * heuristic chooses needs more than LLA_NOALLOC_SCRATCH_BYTES (4 bytes per
 * (b, h) unit rounded up to 256, plus 4 * (r_v + 2) bytes per unit and split;
 * on a 256-CU MI355X the default heuristic splits at most 768 unit-slices, so
 * it stays below 1.6 MiB at r_v = 512).
 */
lla_status lla_decode_attn_noalloc(int dtype, int out_dtype, int B, int H, int d_head, int r_k,
                                   int r_v, int n_max, int n_ctx, const int32_t* ctx_len,
                                   const void* q, const void* c_k, const void* c_v, const void* u_k,
                                   const void* u_v, const void* mu_k, const void* mu_v, float scale,
                                   void* out, void* stream);

/*
 * Causal prefill attention at loop l over the latent cache: query m of
 * sequence b sits at absolute position p0 + m and attends the cached tokens
 * n <= p0 + m, i.e. row m equals lla_decode_attn with N = p0 + m + 1 (pass 2
 * of the two-pass decoder of App. A reads the cache this way).  The cache
 * must already hold positions [0, p0 + M) (write them with lla_encode first);
 * later slots are not read.
 *
 *   q    [B][H][M][d_head]   loop-l queries
 *   out  [B][H][M][d_head]   of out_dtype
 *   workspace  device memory of ws_bytes >= lla_prefill_workspace_bytes() for
 *        these sizes (16-byte aligned, no initial contents needed, overwritten;
 *        calls sharing it must be ordered on the stream), or NULL with
 *        ws_bytes == 0 when that size is 0
 *   other arguments as for lla_decode_attn.
 *
 * Requires M >= 1, p0 >= 0, p0 + M <= n_max, and the decode size limits.
 * fp32 runs an fp32 scan (one workgroup per query).  bf16 runs one of two
 * kernels, each with fp32 accumulation:
 *  - r_k <= 95 and r_v <= 95 (d_head <= 128): the absorbed form of App. J,
 *    q~ = U_k^T q, s_n = q~ . c_k[n], z = sum_n p_n c_v[n], out = U_v z / l +
 *    mu_v, with no workspace.  The latent pages and U_v are converted from
 *    bf16 to fp16 (exact within fp16's range), and q~ * scale * log2(e), the
 *    softmax weights and z / l are rounded to fp16 before their products.
 *  - otherwise (d_head = 128, r_k and r_v multiples of 8 up to LLA_MAX_RANK):
 *    every head's K_l = c_k U_k^T and V_l = c_v U_v^T (Eq. 3) are rebuilt for
 *    positions [0, p0 + M) on MFMA into the workspace in fp16, then the
 *    teacher's attention runs over them; q * scale * log2(e) and the softmax
 *    weights enter its products in fp16.  The workspace holds
 *    4 * B * H * d_head * (p0 + M rounded up to 64) bytes.
 * fp16 range: the fp16 operands above (latent and U_v entries, rebuilt K and
 * V entries, scaled queries q~ or q) and the base-2 logits
 * scale * log2(e) * q . k (the running row maximum is held in fp16) must stay
 * below 65504 in magnitude; beyond it the affected outputs are not finite.
 * Non-finite data: a masked (future) key of a 64-key page enters the value
 * product with weight 0, and 0 * NaN is NaN, so a non-finite value latent at
 * position n may also make non-finite the outputs of the queries at positions
 * 64 * floor(n / 64) - 31 .. n - 1 (at most 95 before it); queries before
 * those are unaffected.  A non-finite key latent affects only the queries
 * that attend it.
 * Errors: LLA_ERR_INVALID_ARG; LLA_ERR_WORKSPACE (missing or too small);
 * LLA_ERR_UNSUPPORTED for bf16 shapes neither kernel takes, or more than
 * 65535 query blocks (256 queries) or (b, h) pairs on the rebuild path;
 * LLA_ERR_HIP.
 */
lla_status lla_prefill_attn(int dtype, int out_dtype, int B, int H, int M, int d_head, int r_k,
                            int r_v, int n_max, int p0, const void* q, const void* c_k,
                            const void* c_v, const void* u_k, const void* u_v, const void* mu_k,
                            const void* mu_v, float scale, void* out, void* workspace,
                            size_t ws_bytes, void* stream);

/* Workspace bytes lla_prefill_attn needs for these sizes: 0 when the call
 * takes none (fp32, or bf16 with both ranks <= 95 and d_head <= 128).  Host
 * only.  Errors: LLA_ERR_INVALID_ARG. */
lla_status lla_prefill_workspace_bytes(int dtype, int B, int H, int M, int d_head, int r_k, int r_v,
                                      int p0, size_t* bytes);

/*
 * Loop-l decode with full RoPE, reconstruct-then-attend (Sec. 3 "RoPE and
 * reconstruction"): the latent is fit to the pre-RoPE content projection and a
 * token's rotary phase, the same at every loop, is applied after the loop-l
 * reconstruction.  Every cached key is rebuilt and rotated at its position,
 *   K_l[n] = RoPE(U_k c_k[n] + mu_k, n)          (slot n holds position n)
 *   s_n    = scale * < RoPE(q, p_q), K_l[n] >     n < N_b
 *   out    = U_v (sum_n softmax(s)_n c_v[n]) + mu_v
 * Values carry no rotary phase, so the value side keeps the absorbed form of
 * App. J; the key side cannot (the rotation differs per key), so K is
 * reconstructed on chip (never written to memory).  RoPE is half-split over
 * the whole head (feature i pairs with i + d_head/2, angle p * base^(-2i/d_head)).
 *
 *   q        [B][H][d_head]  loop-l queries, NOT rotated (the kernel rotates)
 *   q_pos    device int32 [B] or NULL: the query position p_q of sequence b;
 *            NULL means N_b - 1 (the newest cached token)
 *   mu_k     [H][d_head] or NULL: added before the rotation (it does not
 *            cancel here)
 *   base     RoPE base (finite, > 1), e.g. 10000
 *   scale    softmax scale, the teacher's 1/sqrt(d_head)
 *   other arguments as for lla_decode_attn; the workspace is the one sized by
 *   lla_decode_workspace_bytes (the context may be split over workgroups).
 * bf16 with d_head = 128 and r_k <= 256 runs on bf16 MFMA (fp32 accumulation,
 * keys reconstructed exactly from bf16 operands); fp32 and other shapes run a
 * plain fp32 kernel.
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_WORKSPACE, LLA_ERR_HIP.
 */
lla_status lla_decode_attn_fullrope(int dtype, int out_dtype, int B, int H, int d_head, int r_k,
                                    int r_v, int n_max, int n_ctx, const int32_t* ctx_len,
                                    const int32_t* q_pos, const void* q, const void* c_k,
                                    const void* c_v, const void* u_k, const void* u_v,
                                    const void* mu_k, const void* mu_v, double base, float scale,
                                    void* out, void* workspace, size_t ws_bytes, void* stream);

/*
 * Decoupled rotary branch (App. J, "Absorbed attention"): RoPE prevents exact
 * absorption of the positional component, so a small explicit rotary key per
 * token joins the NoPE content path; it is shared across the loops (written
 * once per token) and, MLA-style, either shared by the heads (H_rope = 1) or
 * one per head (H_rope = H).  With it, the score of key n becomes
 *   scale * ( <q, K_l[n]> + <RoPE(q_r, p_q), RoPE(k_r[n], p_n)> ).
 * RoPE here is half-split: feature i pairs with feature i + d_rope/2 and turns
 * by the angle p * base^(-2i/d_rope) (the paper names no convention; this is
 * the one of Llama-family models).  d_rope is a multiple of 8 in
 * [8, LLA_MAX_ROPE].
 *
 * Rotary cache layout: like a latent cache of rank d_rope with H_rope heads,
 *   element (b, g, token n, feature i) at
 *     ((b*H_rope + g) * n_max + (n/64)*64) * d_rope + i*64 + (n % 64),
 * holding keys already rotated at their position (slot n = position n).
 */

/*
 * Rotate the rotary keys of M new tokens per sequence at positions
 * pos0 .. pos0+M-1 and write them into the rotary cache (App. J).
 *
 *   k_rope  [B][M][H_rope][d_rope]  raw (unrotated) rotary keys, dtype
 *   r_cache paged rotary cache (layout above), dtype, capacity n_max
 *   base    the RoPE base (e.g. 10000), > 1
 *
 * Requires 0 <= pos0, pos0 + M <= n_max, H_rope <= 65535.  Writes exactly the slots
 * [pos0, pos0 + M) of every (b, g); angles are formed in double precision and
 * the result rounded to dtype (RNE for bf16).
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_HIP.
 */
lla_status lla_rope_write(int dtype, int B, int M, int H_rope, int d_rope, const void* k_rope,
                          double base, void* r_cache, int n_max, int pos0, void* stream);

/*
 * Rotate query rotary parts (App. J) into a dense output:
 *   x, y  [B][G][M][d_rope] of dtype (y may not alias x)
 * Row (b, g, m) is rotated at position (pos ? pos[b] : pos0) + m, where pos is
 * an optional device int32 [B] (for decode: each sequence's newest position,
 * N_b - 1; for prefill: pos0 = p0 with M the new tokens).  G <= 65535.
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_HIP.
 */
lla_status lla_rope_rotate(int dtype, int B, int G, int M, int d_rope, const void* x,
                           const int32_t* pos, int pos0, double base, void* y, void* stream);

/*
 * lla_decode_attn with the decoupled rotary branch:
 *   q_rope   [B][H][d_rope]  the query's rotary part, already rotated at its
 *                            position (lla_rope_rotate)
 *   r_cache  rotary cache written by lla_rope_write (rotated keys)
 * Slot n of r_cache is key n of the context, as for the latents.  The softmax
 * scale is the caller's (the usual choice is 1/sqrt(d_head + d_rope)).
 * Extra limits: ceil8(r_k) + d_rope <= LLA_MAX_RANK; H_rope is 1 or H.
 * Errors: as lla_decode_attn.
 */
lla_status lla_decode_attn_rope(int dtype, int out_dtype, int B, int H, int d_head, int r_k,
                                int r_v, int d_rope, int H_rope, int n_max, int n_ctx,
                                const int32_t* ctx_len, const void* q, const void* q_rope,
                                const void* c_k, const void* c_v, const void* r_cache,
                                const void* u_k, const void* u_v, const void* mu_k,
                                const void* mu_v, float scale, void* out, void* workspace,
                                size_t ws_bytes, void* stream);

/*
 * lla_prefill_attn with the decoupled rotary branch (no workspace):
 *   q_rope  [B][H][M][d_rope]  rotary query parts rotated at p0 + m
 * bf16 runs the absorbed kernel only and requires r_k + d_rope <= 95 and
 * r_v <= 95 (else LLA_ERR_UNSUPPORTED); the rotary keys and query parts enter
 * its score product in fp16, under lla_prefill_attn's range and non-finite
 * rules.
 * Errors: as lla_prefill_attn.
 */
lla_status lla_prefill_attn_rope(int dtype, int out_dtype, int B, int H, int M, int d_head,
                                 int r_k, int r_v, int d_rope, int H_rope, int n_max, int p0,
                                 const void* q, const void* q_rope, const void* c_k,
                                 const void* c_v, const void* r_cache, const void* u_k,
                                 const void* u_v, const void* mu_k, const void* mu_v, float scale,
                                 void* out, void* stream);

/*
 * Sequence-axis eviction composed with the latent cache (App. J "Eviction and
 * long-context prefill"; tab:evict): a StreamingLLM-style budget keeps the
 * first `sink` tokens and the most recent `window` tokens.  The cache then
 * holds sink + window slots: position p lives in slot p when p < sink, else in
 * slot sink + (p - sink) % window (a ring).  Attention on the content path
 * does not depend on the order of the keys, so the decode entry points attend
 * slots [0, min(N, sink + window)) unchanged (pass that as n_ctx / ctx_len);
 * rotary keys are rotated at their true position before they are stored, so
 * the rotary branch composes too (rotate the query at its true position).
 */

/*
 * lla_encode writing position pos0 + m into its ring slot.
 * Requires sink >= 0, window >= 1, sink + window <= n_max, and the M tokens to
 * land in distinct slots: at most `window` of them at positions >= sink.
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_HIP.
 */
lla_status lla_encode_ring(int dtype, int B, int M, int H, int T, int d_head, int r_k, int r_v,
                           const void* x_k, const void* x_v, const void* mu_k, const void* mu_v,
                           const void* wdt_k, const void* wdt_v, void* c_k, void* c_v, int n_max,
                           int pos0, int sink, int window, void* stream);

/*
 * lla_rope_write rotating key m at its position pos0 + m and storing it in the
 * position's ring slot; the same slot requirements as lla_encode_ring.
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_HIP.
 */
lla_status lla_rope_write_ring(int dtype, int B, int M, int H_rope, int d_rope, const void* k_rope,
                               double base, void* r_cache, int n_max, int pos0, int sink,
                               int window, void* stream);

/*
 * LLA-2D (Sec. 3 "The LLA-2D variant (loop x head)"): one latent per token and
 * layer reconstructs all H heads, (r_k + r_v) scalars per token per layer, a
 * factor H below per-head LLA.  The down-projection input is the whole
 * loop-major, head-major stack x = [x_{1,1}; ...; x_{1,H}; ...; x_{T,H}] of
 * T*H*d_head values, and loop l, head h has its own up-projection slice
 * U_{k,l,h} [d_head][r_k] (likewise U_v).
 *
 * Cache layouts (one sequence b of capacity n_max):
 *   key latents   token-major: element (b, n, j) at (b*n_max + n)*r_k + j
 *   value latents paged feature-major, as a per-head cache with H = 1:
 *                 element (b, n, j) at (b*n_max + (n/64)*64)*r_v + j*64 + n%64
 * The write and the decode support bf16 only, H = 16, r_k a multiple of 32 and
 * r_v a multiple of 16, both <= LLA_MAX_RANK_2D (else LLA_ERR_UNSUPPORTED); the
 * prefill's limits are stated with it.
 */

/*
 * Write c = (x - mu) W_down of M new tokens per sequence into the LLA-2D
 * caches at positions pos0 .. pos0+M-1 (Eqs. 1-2 over the T*H*d_head stack).
 *   x_k, x_v      [B][M][T*H*d_head]
 *   mu_k, mu_v    [T*H*d_head] or NULL
 *   wdt_k, wdt_v  [r][T*H*d_head]  (W_down transposed)
 *   c_k, c_v      the 2D caches (layouts above), capacity n_max
 *   workspace     NULL (ws_bytes ignored), or a device buffer of ws_bytes >=
 *                 lla_encode_2d_workspace_bytes(): with at most 64 new tokens
 *                 and a stack of >= 2048 values, the contraction is then split
 *                 over the stack so the weights spread over every compute
 *                 unit (a decode step's write), in two launches that pass fp32
 *                 partial sums through the workspace (no initial contents
 *                 needed).  Calls that share a workspace must not overlap.
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_UNSUPPORTED, LLA_ERR_WORKSPACE, LLA_ERR_HIP.
 */
lla_status lla_encode_2d(int dtype, int B, int M, int H, int T, int d_head, int r_k, int r_v,
                         const void* x_k, const void* x_v, const void* mu_k, const void* mu_v,
                         const void* wdt_k, const void* wdt_v, void* c_k, void* c_v, int n_max,
                         int pos0, void* workspace, size_t ws_bytes, void* stream);

/* Workspace bytes lla_encode_2d uses for M new tokens per sequence (0: the
 * write is not split and takes no workspace).  Errors: LLA_ERR_INVALID_ARG. */
lla_status lla_encode_2d_workspace_bytes(int B, int M, int H, int T, int d_head, int r_k, int r_v,
                                         size_t* bytes);

/* Workspace bytes lla_decode_attn_2d needs (the absorbed queries and the split
 * partials).  Host only.  Errors: LLA_ERR_INVALID_ARG. */
lla_status lla_decode_2d_workspace_bytes(int B, int H, int r_k, int r_v, int n_ctx, size_t* bytes);

/*
 * Loop-l decode of all H heads of every sequence over its shared LLA-2D latents
 * (absorbed form of App. J applied per head): q~_h = U_{k,l,h}^T q_h, scores
 * q~_h . c_k[n] over n < N_b, softmax, z_h = sum_n p_n c_v[n],
 * out_h = U_{v,l,h} z_h + mu_{v,l,h}.
 *   q    [B][H][d_head];  u_k [H][d_head][r_k];  u_v [H][d_head][r_v]
 *   mu_k, mu_v [H][d_head] or NULL (mu_k cancels in the softmax)
 *   out  [B][H][d_head] of out_dtype
 *   workspace  device memory of at least lla_decode_2d_workspace_bytes (no
 *              initial contents needed; calls sharing it must be ordered)
 * ctx_len and n_ctx as for lla_decode_attn (NaN output for a bad length).
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_UNSUPPORTED, LLA_ERR_WORKSPACE, LLA_ERR_HIP.
 */
lla_status lla_decode_attn_2d(int dtype, int out_dtype, int B, int H, int d_head, int r_k, int r_v,
                              int n_max, int n_ctx, const int32_t* ctx_len, const void* q,
                              const void* c_k, const void* c_v, const void* u_k, const void* u_v,
                              const void* mu_k, const void* mu_v, float scale, void* out,
                              void* workspace, size_t ws_bytes, void* stream);

/* Workspace bytes lla_prefill_attn_2d needs when the keys span positions
 * 0 .. n_keys-1 (n_keys = p0 + M): every head's rebuilt keys and values in
 * fp16, 4 * B * H * d_head * (n_keys rounded up to 64) bytes.  Host only.
 * Errors: LLA_ERR_INVALID_ARG. */
lla_status lla_prefill_2d_workspace_bytes(int B, int H, int d_head, int n_keys, size_t* bytes);

/*
 * Loop-l causal prefill of all H heads over the shared LLA-2D latents, on the
 * full-memory path of App. J ("Per-head LLA versus LLA-2D at inference"):
 * every head's K_h = c_k U_{k,l,h}^T and V_h = c_v U_{v,l,h}^T (Eq. 3 with the
 * (l, h) slice of W_up) are rebuilt for positions 0 .. p0+M-1 into the
 * workspace, then query m of head h, at position p0 + m, attends the keys
 * n <= p0 + m:  out = softmax(scale * K_h q) V_h + mu_{v,l,h}.  The rebuilt
 * K and V, the query scaled by scale * log2(e) and the softmax weights enter
 * the products in fp16 (accumulation in fp32), and the running row maximum of
 * the base-2 logits scale * log2(e) * q.k is held in fp16: |q|, |K| and |V|
 * entries and those logits must stay below 65504 in magnitude, else the output
 * is not finite.  Non-finite latents follow lla_prefill_attn's rule (a value
 * latent at position n may also reach the queries at positions
 * 64 * floor(n / 64) - 31 .. n - 1).
 *   q    [B][H][M][d_head]; out [B][H][M][d_head] of out_dtype
 *   c_k, c_v  the 2D caches (layouts above) of capacity n_max, holding latents
 *        at positions 0 .. p0+M-1 (p0 + M <= n_max); later slots are not read
 *   u_k [H][d_head][r_k]; u_v [H][d_head][r_v]; mu_k, mu_v [H][d_head] or NULL
 *        (mu_k cancels in the softmax)
 *   workspace  device memory of at least lla_prefill_2d_workspace_bytes(B, H,
 *        d_head, p0 + M), 16-byte aligned; overwritten, no initial contents
 *        needed; calls sharing it must be ordered on the stream
 * Supported: bf16, d_head = 128, r_k and r_v multiples of 16 up to 512, any H
 * (else LLA_ERR_UNSUPPORTED).  B*H*M <= 2^30 and B <= 65535 (else
 * LLA_ERR_INVALID_ARG).
 * Errors: LLA_ERR_INVALID_ARG, LLA_ERR_UNSUPPORTED, LLA_ERR_WORKSPACE, LLA_ERR_HIP.
 */
lla_status lla_prefill_attn_2d(int dtype, int out_dtype, int B, int H, int M, int d_head, int r_k,
                               int r_v, int n_max, int p0, const void* q, const void* c_k,
                               const void* c_v, const void* u_k, const void* u_v, const void* mu_k,
                               const void* mu_v, float scale, void* out, void* workspace,
                               size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LLA_H_ */
