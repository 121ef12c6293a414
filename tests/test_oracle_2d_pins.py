"""Pins of the oracle's LLA-2D variant (Sec. 3 "The LLA-2D variant (loop x
head)": one latent per token and layer reconstructs all H heads).

A block-diagonal 2D codec (each head's per-head codec in its own block of the
latent) must reproduce per-head LLA exactly: that ties the 2D stacking order,
the shared-latent encode and the per-(loop, head) up-projection slices to the
already-pinned per-head oracle.  The cache accounting is pinned against the
paper's statement (a factor H below per-head LLA) and the printed 2D ratios;
the attention against pure-Python brute force."""

import math

import numpy as np
import pytest

import oracle


def test_2d_ratio_and_cache_are_a_factor_h_below_per_head():
    # Ouro-1.4B: T 4, H 16, d 128.  The printed LLA-2D operating points 5.33x and 21.33x
    # (tab:isocache) need rank sums 3072 and 768 for a single latent per token.
    T, H, d = 4, 16, 128
    assert oracle.compression_ratio(T, H * d, 1152, 1920) == oracle.compression_ratio(T, d, 72, 120)
    assert f"{float(oracle.compression_ratio(T, H * d, 1152, 1920)):.2f}" == "5.33"
    assert f"{float(oracle.compression_ratio(T, H * d, 288, 480)):.2f}" == "21.33"
    per_head = oracle.cache_bytes(24, 16, T, d, 288, 480, 1, 2, latent=True)
    two_d = oracle.cache_bytes(24, 1, T, d, 288, 480, 1, 2, latent=True)
    assert per_head == 16 * two_d


def test_stack_is_loop_major_then_head_major():
    x = [[np.full(2, 10 * t + h) for h in range(3)] for t in range(2)]
    assert list(oracle.stack_loops_heads(x)) == [0, 0, 1, 1, 2, 2, 10, 10, 11, 11, 12, 12]


def test_block_diagonal_2d_codec_is_per_head_lla():
    g = np.random.default_rng(1)
    T, H, d, rk, rv, N = 2, 3, 4, 2, 3, 6
    # per-head codecs: W_down,h [T*d, r], loop-l up-projections U_{l,h} [d, r]
    wdk = g.standard_normal((H, T * d, rk))
    wdv = g.standard_normal((H, T * d, rv))
    xk = g.standard_normal((N, T, H, d))   # token n, loop t, head h
    xv = g.standard_normal((N, T, H, d))
    ck_h = np.stack([oracle.encode(oracle.stack_loops([xk[:, t, h] for t in range(T)]), None, wdk[h])
                     for h in range(H)])   # [H, N, rk]
    cv_h = np.stack([oracle.encode(oracle.stack_loops([xv[:, t, h] for t in range(T)]), None, wdv[h])
                     for h in range(H)])
    # the 2D down-projection: row (t, h, i) of the T*H*d stack feeds latent block h
    Wk = np.zeros((T * H * d, H * rk))
    Wv = np.zeros((T * H * d, H * rv))
    for t in range(T):
        for h in range(H):
            Wk[(t * H + h) * d:(t * H + h + 1) * d, h * rk:(h + 1) * rk] = wdk[h, t * d:(t + 1) * d]
            Wv[(t * H + h) * d:(t * H + h + 1) * d, h * rv:(h + 1) * rv] = wdv[h, t * d:(t + 1) * d]
    ck2 = oracle.encode(oracle.stack_loops_heads([[xk[:, t, h] for h in range(H)] for t in range(T)]), None, Wk)
    cv2 = oracle.encode(oracle.stack_loops_heads([[xv[:, t, h] for h in range(H)] for t in range(T)]), None, Wv)
    assert np.max(np.abs(ck2 - np.concatenate(list(ck_h), axis=1))) < 1e-12
    assert np.max(np.abs(cv2 - np.concatenate(list(cv_h), axis=1))) < 1e-12
    # loop-l up-projections of the 2D codec: head h's block only
    uk_h, uv_h = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    Uk2, Uv2 = np.zeros((H, d, H * rk)), np.zeros((H, d, H * rv))
    for h in range(H):
        Uk2[h, :, h * rk:(h + 1) * rk] = uk_h[h]
        Uv2[h, :, h * rv:(h + 1) * rv] = uv_h[h]
    mk, mv = g.standard_normal((H, d)), g.standard_normal((H, d))
    q = g.standard_normal((H, d))
    got = oracle.decode_attn_2d(q, ck2, cv2, Uk2, Uv2, mk, mv, scale=0.3)
    for h in range(H):
        ref = oracle.decode_attn(q[h], ck_h[h], cv_h[h], uk_h[h], uv_h[h], mk[h], mv[h], scale=0.3)
        assert np.max(np.abs(got[h] - ref)) < 1e-12


def test_decode_2d_bruteforce():
    g = np.random.default_rng(2)
    H, d, rk, rv, N = 2, 3, 4, 2, 5
    q = g.standard_normal((H, d))
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    Uk, Uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    got = oracle.decode_attn_2d(q, ck, cv, Uk, Uv, scale=0.7)
    for h in range(H):
        K = [[sum(ck[n, j] * Uk[h, i, j] for j in range(rk)) for i in range(d)] for n in range(N)]
        V = [[sum(cv[n, j] * Uv[h, i, j] for j in range(rv)) for i in range(d)] for n in range(N)]
        s = [0.7 * sum(q[h, i] * K[n][i] for i in range(d)) for n in range(N)]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        ref = [sum(e[n] * V[n][i] for n in range(N)) / sum(e) for i in range(d)]
        assert np.max(np.abs(got[h] - np.array(ref))) < 1e-12


def test_decode_2d_batched_lengths():
    g = np.random.default_rng(3)
    B, H, d, rk, rv, N = 2, 2, 4, 3, 2, 7
    q = g.standard_normal((B, H, d))
    ck, cv = g.standard_normal((B, N, rk)), g.standard_normal((B, N, rv))
    Uk, Uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    out = oracle.decode_attn_2d_batched(q, ck, cv, Uk, Uv, ctx_len=[7, 3])
    assert np.array_equal(out[1], oracle.decode_attn_2d(q[1], ck[1, :3], cv[1, :3], Uk, Uv))
    assert np.array_equal(out[0], oracle.decode_attn_2d(q[0], ck[0], cv[0], Uk, Uv))
