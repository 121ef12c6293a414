"""Plain float64 CPU oracle of Looped Latent Attention (LLA), arxiv 2607.15456.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  The product path
(the HIP library and its Python binding) never imports, links or calls it, and
this module imports nothing from the product package.

Every function is written straight from the paper's definitions, in float64,
with no blocking, fusion or reordering beyond what the definition states, so
that it can be checked against the paper by eye.  Notation follows the paper:

* T recurrence steps (loops), D layers, H heads of width d = d_head;
* per (layer, head, token, axis) the teacher emits T vectors x_1..x_T, stacked
  loop-major as x = [x_1; ...; x_T] of length T*d            (Sec. 3, Eq. 1);
* the codec stores c = (x - mu) W_down, c in R^r              (Sec. 3, Eq. 2);
* loop t is reconstructed as x_hat_t = c W_up,t^T + mu_t      (Sec. 3, Eq. 3);
* the exact compression ratio is rho = 2 T d / (r_k + r_v)   (Sec. 3, Eq. 4).

Loop indices here are 0-based (l = 0..T-1); the paper's t is l + 1.

Attention itself is the teacher's, unchanged (Sec. 1, caption of the
architecture figure: reconstruction happens before attention, which is left
unchanged): s_n = scale * <q, k_n>, a = softmax(s), o = sum_n a_n v_n.

Readings where the paper is silent:
* the softmax scale is a parameter; the teacher's 1/sqrt(d_head) is the default;
* no RoPE on the content path (the NoPE content path of App. J, where
  absorption is exact); the decoupled rotary branch of App. J is a separate
  per-token key, shared across loops, rotated half-split (pairs i, i + d_rope/2)
  with angle p * base^(-2i/d_rope), and its softmax scale defaults to
  1/sqrt(d_head + d_rope);
* full RoPE (the paper's accuracy path): the rotary phase of a token's position
  is applied to the loop-l reconstruction of its key (values carry none), with
  the same half-split convention over all d_head features;
* a decode query attends exactly the N cached latent entries [0, N);
* a prefill query at absolute position p attends keys n <= p.

Parity pins: see tests/test_oracle_pins.py.  Every function below is pinned
there by something other than itself (printed values, closed forms, brute
force in pure Python, special cases that reduce to textbook results).
"""

from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

__all__ = [
    "compression_ratio",
    "teacher_scalars_per_token_layer",
    "latent_scalars_per_token_layer",
    "cache_bytes",
    "stack_loops",
    "encode",
    "reconstruct",
    "softmax",
    "attention",
    "default_scale",
    "decode_attn",
    "decode_attn_absorbed",
    "prefill_attn",
    "split_partial",
    "split_merge",
    "decode_attn_batched",
    "prefill_attn_batched",
    "prefill_attn_2d",
    "prefill_attn_2d_batched",
    "encode_batched",
    "rope",
    "decode_attn_rope",
    "prefill_attn_rope",
    "decode_attn_rope_batched",
    "prefill_attn_rope_batched",
    "kept_positions",
    "ring_slot",
    "decode_attn_evict",
    "decode_attn_rope_evict",
    "stack_loops_heads",
    "decode_attn_2d",
    "decode_attn_2d_batched",
    "decode_attn_fullrope",
    "decode_attn_fullrope_batched",
]


# ---------------------------------------------------------------------------
# Sec. 3, Eq. 4 and the "Teacher cache" / "Cross-loop codec" paragraphs:
# scalar accounting of the cache.
# ---------------------------------------------------------------------------

def compression_ratio(T: int, d_head: int, r_k: int, r_v: int) -> Fraction:
    """Eq. 4: rho = 2 T H d / ((r_k + r_v) H) = 2 T d / (r_k + r_v), exact."""
    for name, v in (("T", T), ("d_head", d_head), ("r_k", r_k), ("r_v", r_v)):
        if int(v) != v or v <= 0:
            raise ValueError(f"{name} must be a positive integer, got {v!r}")
    return Fraction(2 * T * d_head, r_k + r_v)


def teacher_scalars_per_token_layer(T: int, H: int, d_head: int) -> int:
    """Sec. 3 "Teacher cache": K and V for every loop and head: 2 T H d scalars."""
    return 2 * T * H * d_head


def latent_scalars_per_token_layer(H: int, r_k: int, r_v: int) -> int:
    """Sec. 3 "Cross-loop codec": (r_k + r_v) H latent scalars per token per layer."""
    return (r_k + r_v) * H


def cache_bytes(layers: int, heads: int, T: int, d_head: int, r_k: int, r_v: int,
                tokens: int, elem_bytes: int, latent: bool) -> int:
    """Bytes of a D-layer cache holding ``tokens`` tokens (Sec. 3; tab:memory)."""
    per = (latent_scalars_per_token_layer(heads, r_k, r_v) if latent
           else teacher_scalars_per_token_layer(T, heads, d_head))
    return layers * per * elem_bytes * tokens


# ---------------------------------------------------------------------------
# Sec. 3, Eqs. 1-3: the codec.
# ---------------------------------------------------------------------------

def stack_loops(per_loop):
    """Eq. 1: x = [x_1; ...; x_T], loop-major along the last axis."""
    return np.concatenate([np.asarray(v, dtype=np.float64) for v in per_loop], axis=-1)


def encode(x, mu, w_down):
    """Eq. 2: c = (x - mu) W_down.

    x: [..., T*d] loop-stacked vectors; mu: [T*d] or None (zero mean);
    w_down: [T*d, r].  Returns c: [..., r].
    """
    x = np.asarray(x, dtype=np.float64)
    w_down = np.asarray(w_down, dtype=np.float64)
    if mu is not None:
        x = x - np.asarray(mu, dtype=np.float64)
    return x @ w_down


def reconstruct(c, w_up_t, mu_t):
    """Eq. 3: x_hat_t = c W_up,t^T + mu_t.

    c: [..., r]; w_up_t: [d, r] (the loop-t up-projection); mu_t: [d] or None
    (the loop-t slice of mu).  Returns x_hat_t: [..., d].
    """
    c = np.asarray(c, dtype=np.float64)
    w_up_t = np.asarray(w_up_t, dtype=np.float64)
    out = c @ w_up_t.T
    if mu_t is not None:
        out = out + np.asarray(mu_t, dtype=np.float64)
    return out


# ---------------------------------------------------------------------------
# The teacher's attention (unchanged by LLA).
# ---------------------------------------------------------------------------

def default_scale(d_head: int) -> float:
    """The teacher's softmax scale 1/sqrt(d_head) (reading: the paper leaves
    attention unchanged and states no other scale)."""
    return 1.0 / math.sqrt(d_head)


def softmax(s):
    """Softmax along the last axis, max-shifted."""
    s = np.asarray(s, dtype=np.float64)
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attention(q, K, V, scale):
    """One query against N keys/values: o = softmax(scale K q)^T V.

    q: [d]; K: [N, d]; V: [N, d_v].  Returns o: [d_v].
    """
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    if K.shape[0] == 0:
        raise ValueError("attention over an empty context is undefined")
    a = softmax(scale * (K @ q))
    return a @ V


# ---------------------------------------------------------------------------
# Loop-l decode over the latent cache.
# ---------------------------------------------------------------------------

def decode_attn(q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None):
    """Loop-l decode attention of one (batch, head) over N cached latents --
    the plain definition: reconstruct K_l and V_l with Eq. 3 for every cached
    token, then run the teacher's attention on them.

    q: [d]; c_k: [N, r_k]; c_v: [N, r_v]; u_k: [d, r_k] = W^K_up,l;
    u_v: [d, r_v] = W^V_up,l; mu_k, mu_v: [d] loop-l slices of the means, or
    None.  Returns o: [d].
    """
    d = np.asarray(q).shape[-1]
    if scale is None:
        scale = default_scale(d)
    K = reconstruct(c_k, u_k, mu_k)
    V = reconstruct(c_v, u_v, mu_v)
    return attention(q, K, V, scale)


def decode_attn_absorbed(q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None):
    """The same result through the absorbed identities of App. J
    ("Absorbed attention"): q^T (W_up c) = (W_up^T q)^T c for the score and
    sum_i a_i W^V_up c_i = W^V_up sum_i a_i c_i for the value.  With means,
    Eq. 3 adds q . mu_k to every score and mu_v to the output.
    """
    q = np.asarray(q, dtype=np.float64)
    c_k = np.asarray(c_k, dtype=np.float64)
    c_v = np.asarray(c_v, dtype=np.float64)
    u_k = np.asarray(u_k, dtype=np.float64)
    u_v = np.asarray(u_v, dtype=np.float64)
    if scale is None:
        scale = default_scale(q.shape[-1])
    q_tilde = u_k.T @ q                       # absorbed query, [r_k]
    s = c_k @ q_tilde
    if mu_k is not None:
        s = s + q @ np.asarray(mu_k, dtype=np.float64)
    a = softmax(scale * s)
    z = a @ c_v                               # attention-weighted latent, [r_v]
    o = u_v @ z
    if mu_v is not None:
        o = o + np.asarray(mu_v, dtype=np.float64)
    return o


def prefill_attn(Q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None, p0=0):
    """Causal prefill of M queries at absolute positions p0..p0+M-1 over the
    latent cache: query m attends keys n <= p0 + m (plain definition, row by
    row).  Q: [M, d]; c_k: [>= p0+M, r_k]; c_v likewise.  Returns [M, d]."""
    Q = np.asarray(Q, dtype=np.float64)
    out = np.empty_like(Q)
    for m in range(Q.shape[0]):
        n = p0 + m + 1
        out[m] = decode_attn(Q[m], c_k[:n], c_v[:n], u_k, u_v, mu_k, mu_v, scale)
    return out


# ---------------------------------------------------------------------------
# Split-context partials and their merge (the softmax over a union of
# disjoint key ranges, written as running max / sum / weighted latent).
# ---------------------------------------------------------------------------

def split_partial(q_tilde_scaled, c_k, c_v):
    """Partial softmax state of one key range: (m, l, z) with
    m = max_n s_n, l = sum_n exp(s_n - m), z = sum_n exp(s_n - m) c_v[n],
    where s_n = <q_tilde_scaled, c_k[n]> (the scale already folded in)."""
    s = np.asarray(c_k, dtype=np.float64) @ np.asarray(q_tilde_scaled, dtype=np.float64)
    m = float(np.max(s))
    e = np.exp(s - m)
    return m, float(np.sum(e)), e @ np.asarray(c_v, dtype=np.float64)


def split_merge(partials):
    """Merge (m_s, l_s, z_s) partials: m = max m_s, weights w_s = exp(m_s - m),
    l = sum w_s l_s, z = sum w_s z_s; returns the normalised latent z / l."""
    m = max(p[0] for p in partials)
    w = [math.exp(p[0] - m) for p in partials]
    l_tot = sum(wi * p[1] for wi, p in zip(w, partials))
    z = sum(wi * p[2] for wi, p in zip(w, partials))
    return z / l_tot


# ---------------------------------------------------------------------------
# Batched wrappers: plain loops over (batch, head).  Layouts are the logical
# ones (token-major latents); they say nothing about device layouts.
# ---------------------------------------------------------------------------

def encode_batched(x, mu, w_down_t):
    """Eq. 2 for every (batch, token, head).

    x: [B, M, H, T*d]; mu: [H, T*d] or None; w_down_t: [H, r, T*d]
    (W_down transposed, one per head).  Returns c: [B, H, M, r]."""
    x = np.asarray(x, dtype=np.float64)
    w_down_t = np.asarray(w_down_t, dtype=np.float64)
    B, M, H, _ = x.shape
    r = w_down_t.shape[1]
    c = np.empty((B, H, M, r))
    for b in range(B):
        for h in range(H):
            c[b, h] = encode(x[b, :, h, :], None if mu is None else mu[h], w_down_t[h].T)
    return c


def decode_attn_batched(q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None,
                        ctx_len=None, units=None):
    """decode_attn for every (b, h) (or only the (b, h) pairs in ``units``).

    q: [B, H, d]; c_k: [B, H, >=N, r_k]; c_v: [B, H, >=N, r_v];
    u_k: [H, d, r_k]; u_v: [H, d, r_v]; mu_k, mu_v: [H, d] or None;
    ctx_len: int or per-batch sequence of ints.  Returns [B, H, d] (entries
    not in ``units`` are NaN)."""
    q = np.asarray(q, dtype=np.float64)
    B, H, d = q.shape
    if ctx_len is None:
        ctx_len = c_k.shape[2]
    lens = [int(ctx_len)] * B if np.ndim(ctx_len) == 0 else [int(v) for v in ctx_len]
    out = np.full((B, H, d), np.nan)
    todo = units if units is not None else [(b, h) for b in range(B) for h in range(H)]
    for b, h in todo:
        n = lens[b]
        out[b, h] = decode_attn(q[b, h], c_k[b, h, :n], c_v[b, h, :n], u_k[h], u_v[h],
                                None if mu_k is None else mu_k[h],
                                None if mu_v is None else mu_v[h], scale)
    return out


def prefill_attn_batched(Q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None, p0=0,
                         units=None, rows=None):
    """prefill_attn for every (b, h) (or the given units), optionally only for
    the query rows in ``rows``.  Q: [B, H, M, d].  Returns [B, H, M, d]
    (entries not computed are NaN)."""
    Q = np.asarray(Q, dtype=np.float64)
    B, H, M, d = Q.shape
    out = np.full((B, H, M, d), np.nan)
    todo = units if units is not None else [(b, h) for b in range(B) for h in range(H)]
    row_list = range(M) if rows is None else rows
    for b, h in todo:
        for m in row_list:
            n = p0 + m + 1
            out[b, h, m] = decode_attn(Q[b, h, m], c_k[b, h, :n], c_v[b, h, :n], u_k[h], u_v[h],
                                       None if mu_k is None else mu_k[h],
                                       None if mu_v is None else mu_v[h], scale)
    return out


# ---------------------------------------------------------------------------
# App. J "Absorbed attention": the NoPE content path plus a small explicit
# rotary branch, shared across loops for each token (MLA-style decoupled RoPE).
# The score of key n becomes scale * (<q, K_l[n]> + <RoPE(q_r, p_q), RoPE(k_r[n], p_n)>).
# ---------------------------------------------------------------------------

def rope(x, pos, base=10000.0):
    """Rotary position embedding of x [..., d_rope] at position ``pos`` (scalar
    or broadcastable to x's leading shape).  Half-split convention: feature i
    pairs with feature i + d_rope/2 and turns by the angle pos * base^(-2i/d_rope)
    (reading: the paper names no convention)."""
    x = np.asarray(x, dtype=np.float64)
    dr = x.shape[-1]
    if dr % 2:
        raise ValueError("d_rope must be even")
    half = dr // 2
    inv_freq = base ** (-2.0 * np.arange(half) / dr)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv_freq
    c, s_ = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s_, x2 * c + x1 * s_], axis=-1)


def decode_attn_rope(q, q_rope, c_k, c_v, k_rope, u_k, u_v, mu_k=None, mu_v=None, scale=None,
                     base=10000.0, q_pos=None, k_pos=None):
    """Loop-l decode with the decoupled rotary branch, plain definition: the
    full key of token n is [K_l[n]; RoPE(k_rope[n], k_pos[n])] with K_l from
    Eq. 3, the query is [q; RoPE(q_rope, q_pos)], then the teacher's attention.

    q: [d]; q_rope: [d_rope] (unrotated); c_k: [N, r_k]; c_v: [N, r_v];
    k_rope: [N, d_rope] (unrotated); k_pos defaults to 0..N-1 (the cache slot
    is the position), q_pos to N - 1 (the newest token).  Returns [d]."""
    q = np.asarray(q, dtype=np.float64)
    k_rope = np.asarray(k_rope, dtype=np.float64)
    N = k_rope.shape[0]
    d, dr = q.shape[-1], k_rope.shape[-1]
    if scale is None:
        scale = default_scale(d + dr)
    if k_pos is None:
        k_pos = np.arange(N)
    if q_pos is None:
        q_pos = N - 1
    K = np.concatenate([reconstruct(c_k, u_k, mu_k), rope(k_rope, k_pos, base)], axis=-1)
    V = reconstruct(c_v, u_v, mu_v)
    qf = np.concatenate([q, rope(q_rope, q_pos, base)])
    return attention(qf, K, V, scale)


def prefill_attn_rope(Q, Q_rope, c_k, c_v, k_rope, u_k, u_v, mu_k=None, mu_v=None, scale=None,
                      base=10000.0, p0=0):
    """Causal prefill with the rotary branch: query m sits at position p0 + m
    and attends keys n <= p0 + m (plain definition, row by row)."""
    Q = np.asarray(Q, dtype=np.float64)
    out = np.empty_like(Q)
    for m in range(Q.shape[0]):
        n = p0 + m + 1
        out[m] = decode_attn_rope(Q[m], Q_rope[m], c_k[:n], c_v[:n], k_rope[:n], u_k, u_v, mu_k,
                                  mu_v, scale, base, q_pos=p0 + m)
    return out


def decode_attn_rope_batched(q, q_rope, c_k, c_v, k_rope, u_k, u_v, mu_k=None, mu_v=None,
                             scale=None, base=10000.0, ctx_len=None, units=None):
    """decode_attn_rope for every (b, h).  q: [B, H, d]; q_rope: [B, H, d_rope];
    k_rope: [B, Hr, >=N, d_rope] with Hr = 1 (one rotary key per token, shared
    by the heads) or Hr = H; other arguments as decode_attn_batched."""
    q = np.asarray(q, dtype=np.float64)
    B, H, d = q.shape
    Hr = k_rope.shape[1]
    if ctx_len is None:
        ctx_len = c_k.shape[2]
    lens = [int(ctx_len)] * B if np.ndim(ctx_len) == 0 else [int(v) for v in ctx_len]
    out = np.full((B, H, d), np.nan)
    todo = units if units is not None else [(b, h) for b in range(B) for h in range(H)]
    for b, h in todo:
        n = lens[b]
        hr = 0 if Hr == 1 else h
        out[b, h] = decode_attn_rope(q[b, h], q_rope[b, h], c_k[b, h, :n], c_v[b, h, :n],
                                     k_rope[b, hr, :n], u_k[h], u_v[h],
                                     None if mu_k is None else mu_k[h],
                                     None if mu_v is None else mu_v[h], scale, base)
    return out


def prefill_attn_rope_batched(Q, Q_rope, c_k, c_v, k_rope, u_k, u_v, mu_k=None, mu_v=None,
                              scale=None, base=10000.0, p0=0, units=None, rows=None):
    """prefill_attn_rope for every (b, h) (or the given units / rows).
    Q: [B, H, M, d]; Q_rope: [B, H, M, d_rope]; k_rope: [B, Hr, >=p0+M, d_rope]."""
    Q = np.asarray(Q, dtype=np.float64)
    B, H, M, d = Q.shape
    Hr = k_rope.shape[1]
    out = np.full((B, H, M, d), np.nan)
    todo = units if units is not None else [(b, h) for b in range(B) for h in range(H)]
    row_list = range(M) if rows is None else rows
    for b, h in todo:
        hr = 0 if Hr == 1 else h
        for m in row_list:
            n = p0 + m + 1
            out[b, h, m] = decode_attn_rope(Q[b, h, m], Q_rope[b, h, m], c_k[b, h, :n], c_v[b, h, :n],
                                            k_rope[b, hr, :n], u_k[h], u_v[h],
                                            None if mu_k is None else mu_k[h],
                                            None if mu_v is None else mu_v[h], scale, base,
                                            q_pos=p0 + m)
    return out


# ---------------------------------------------------------------------------
# Sequence-axis eviction composed with the latent cache (App. J "Eviction and
# long-context prefill"; tab:evict): a StreamingLLM-style budget keeps the
# first `sink` tokens and the most recent `window` tokens.
# ---------------------------------------------------------------------------

def kept_positions(N: int, sink: int, window: int):
    """Positions of a context of N tokens that a (sink, window) budget keeps."""
    if N <= sink + window:
        return list(range(N))
    return list(range(sink)) + list(range(N - window, N))


def ring_slot(p: int, sink: int, window: int) -> int:
    """Cache slot of position p when the window part is a ring of ``window`` slots
    after the ``sink`` fixed ones (reading: the paper does not say how the
    budget is laid out; any bijection of the kept positions onto the slots
    gives the same attention on the content path)."""
    return p if p < sink else sink + (p - sink) % window


def decode_attn_evict(q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None, sink=4, window=256):
    """Loop-l decode of the newest token over the tokens an eviction budget keeps
    (plain definition: select the kept positions of the full latent history, then
    decode_attn).  c_k, c_v: [N, r] for every position 0..N-1."""
    keep = kept_positions(np.asarray(c_k).shape[0], sink, window)
    c_k = np.asarray(c_k, dtype=np.float64)[keep]
    c_v = np.asarray(c_v, dtype=np.float64)[keep]
    return decode_attn(q, c_k, c_v, u_k, u_v, mu_k, mu_v, scale)


def decode_attn_rope_evict(q, q_rope, c_k, c_v, k_rope, u_k, u_v, mu_k=None, mu_v=None, scale=None,
                           base=10000.0, sink=4, window=256):
    """decode_attn_rope over the kept positions: the rotary keys keep their true
    positions, and the query sits at N - 1."""
    N = np.asarray(c_k).shape[0]
    keep = kept_positions(N, sink, window)
    return decode_attn_rope(q, q_rope, np.asarray(c_k, dtype=np.float64)[keep],
                            np.asarray(c_v, dtype=np.float64)[keep],
                            np.asarray(k_rope, dtype=np.float64)[keep], u_k, u_v, mu_k, mu_v, scale, base,
                            q_pos=N - 1, k_pos=np.asarray(keep))


# ---------------------------------------------------------------------------
# LLA-2D (Sec. 3 "The LLA-2D variant (loop x head)"): one latent per token and
# layer for all H heads.  The down-projection input is the full T*H*d stack,
# and loop l, head h is reconstructed from the shared latent with its own
# up-projection slice.
# ---------------------------------------------------------------------------

def stack_loops_heads(per_loop_head):
    """The LLA-2D stack: x = [x_{1,1}; ...; x_{1,H}; x_{2,1}; ...; x_{T,H}],
    loop-major then head-major (reading: Eq. 1's loop stacking, with each
    loop's vector being all heads' K (or V) concatenated).
    per_loop_head[t][h]: [..., d]."""
    return np.concatenate([np.asarray(v, dtype=np.float64) for loop in per_loop_head for v in loop], axis=-1)


def decode_attn_2d(q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None):
    """Loop-l decode of all H heads over one shared latent per token (plain
    definition): head h reconstructs K_{l,h} = c_k U_{k,l,h}^T + mu_{k,l,h} and
    V_{l,h} likewise (Eq. 3 with the (l, h) slice of W_up), then runs the
    teacher's attention.

    q: [H, d]; c_k: [N, r_k]; c_v: [N, r_v]; u_k: [H, d, r_k]; u_v: [H, d, r_v];
    mu_k, mu_v: [H, d] or None.  Returns [H, d]."""
    q = np.asarray(q, dtype=np.float64)
    H = q.shape[0]
    return np.stack([decode_attn(q[h], c_k, c_v, u_k[h], u_v[h],
                                 None if mu_k is None else mu_k[h],
                                 None if mu_v is None else mu_v[h], scale) for h in range(H)])


def decode_attn_2d_batched(q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None, ctx_len=None,
                           batches=None):
    """decode_attn_2d for every sequence b (or those in ``batches``).
    q: [B, H, d]; c_k: [B, >=N, r_k]; c_v: [B, >=N, r_v].  Returns [B, H, d]."""
    q = np.asarray(q, dtype=np.float64)
    B, H, d = q.shape
    if ctx_len is None:
        ctx_len = c_k.shape[1]
    lens = [int(ctx_len)] * B if np.ndim(ctx_len) == 0 else [int(v) for v in ctx_len]
    out = np.full((B, H, d), np.nan)
    for b in (range(B) if batches is None else batches):
        n = lens[b]
        out[b] = decode_attn_2d(q[b], c_k[b, :n], c_v[b, :n], u_k, u_v, mu_k, mu_v, scale)
    return out


def prefill_attn_2d(Q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None, p0=0):
    """LLA-2D causal prefill at loop l (plain definition): head h rebuilds
    K_{l,h} = c_k U_{k,l,h}^T + mu_{k,l,h} and V_{l,h} likewise from the shared
    latents (Eq. 3 with the (l, h) slice of W_up), and its query m, at absolute
    position p0 + m, attends keys n <= p0 + m with the teacher's attention.

    Q: [H, M, d]; c_k: [>= p0+M, r_k]; c_v: [>= p0+M, r_v]; u_k: [H, d, r_k];
    u_v: [H, d, r_v]; mu_k, mu_v: [H, d] or None.  Returns [H, M, d]."""
    Q = np.asarray(Q, dtype=np.float64)
    H, M, d = Q.shape
    if scale is None:
        scale = default_scale(d)
    n_all = p0 + M
    out = np.empty_like(Q)
    for h in range(H):
        K = reconstruct(c_k[:n_all], u_k[h], None if mu_k is None else mu_k[h])
        V = reconstruct(c_v[:n_all], u_v[h], None if mu_v is None else mu_v[h])
        for m in range(M):
            n = p0 + m + 1
            out[h, m] = attention(Q[h, m], K[:n], V[:n], scale)
    return out


def prefill_attn_2d_batched(Q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None, p0=0,
                            batches=None):
    """prefill_attn_2d for every sequence b (or those in ``batches``).
    Q: [B, H, M, d]; c_k: [B, >= p0+M, r_k]; c_v: [B, >= p0+M, r_v] (token-major).
    Returns [B, H, M, d] (sequences not computed are NaN)."""
    Q = np.asarray(Q, dtype=np.float64)
    out = np.full(Q.shape, np.nan)
    for b in (range(Q.shape[0]) if batches is None else batches):
        out[b] = prefill_attn_2d(Q[b], c_k[b], c_v[b], u_k, u_v, mu_k, mu_v, scale, p0)
    return out


# ---------------------------------------------------------------------------
# Sec. 3 "RoPE and reconstruction": the latent is fit to the pre-RoPE content
# projection, and since a token keeps its position at every recurrence step its
# rotary phase is applied after the loop-l reconstruction.  This is the full-RoPE
# path all main accuracy results use (App. J, tab:decoupled_char), read here as
# reconstruct-then-attend over the latent cache: the rotation differs per key
# position, so the key up-projection cannot move to the query side (App. J);
# values carry no rotary phase.
# ---------------------------------------------------------------------------

def decode_attn_fullrope(q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None, base=10000.0,
                         q_pos=None, k_pos=None):
    """Loop-l decode with full RoPE, plain definition: every cached key is
    reconstructed with Eq. 3 and then rotated at its position,
    K_l[n] = RoPE(c_k[n] U_k^T + mu_k, k_pos[n]); values V_l[n] = c_v[n] U_v^T + mu_v
    are not rotated; the query is RoPE(q, q_pos); then the teacher's attention
    with its scale 1/sqrt(d_head).

    q: [d] (unrotated); c_k: [N, r_k]; c_v: [N, r_v]; u_k: [d, r_k]; u_v: [d, r_v];
    mu_k, mu_v: [d] or None.  k_pos defaults to 0..N-1 (cache slot n holds
    position n), q_pos to N - 1 (the newest cached token).  Returns [d]."""
    q = np.asarray(q, dtype=np.float64)
    N = np.asarray(c_k).shape[0]
    d = q.shape[-1]
    if scale is None:
        scale = default_scale(d)
    if k_pos is None:
        k_pos = np.arange(N)
    if q_pos is None:
        q_pos = N - 1
    K = rope(reconstruct(c_k, u_k, mu_k), k_pos, base)
    V = reconstruct(c_v, u_v, mu_v)
    return attention(rope(q, q_pos, base), K, V, scale)


def decode_attn_fullrope_batched(q, c_k, c_v, u_k, u_v, mu_k=None, mu_v=None, scale=None,
                                 base=10000.0, ctx_len=None, q_pos=None, units=None):
    """decode_attn_fullrope for every (b, h) (or the pairs in ``units``).
    q: [B, H, d]; c_k: [B, H, >=N, r_k]; c_v: [B, H, >=N, r_v]; u_k: [H, d, r_k];
    u_v: [H, d, r_v]; ctx_len: int or per-batch ints; q_pos: None (N_b - 1 for
    every sequence) or per-batch ints.  Returns [B, H, d] (NaN where not computed)."""
    q = np.asarray(q, dtype=np.float64)
    B, H, d = q.shape
    if ctx_len is None:
        ctx_len = c_k.shape[2]
    lens = [int(ctx_len)] * B if np.ndim(ctx_len) == 0 else [int(v) for v in ctx_len]
    qp = [n - 1 for n in lens] if q_pos is None else [int(v) for v in q_pos]
    out = np.full((B, H, d), np.nan)
    todo = units if units is not None else [(b, h) for b in range(B) for h in range(H)]
    for b, h in todo:
        n = lens[b]
        out[b, h] = decode_attn_fullrope(q[b, h], c_k[b, h, :n], c_v[b, h, :n], u_k[h], u_v[h],
                                         None if mu_k is None else mu_k[h],
                                         None if mu_v is None else mu_v[h], scale, base,
                                         q_pos=qp[b])
    return out
