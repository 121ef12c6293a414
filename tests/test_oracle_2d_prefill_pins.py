"""Pins of the oracle's LLA-2D causal prefill (Sec. 3 "The LLA-2D variant
(loop x head)": one latent per token reconstructs all H heads; App. J
"Per-head LLA versus LLA-2D at inference").

Independent formulations: pure-Python brute force (reconstruction and
attention written out with math.exp); each query row must be the 2D decode of
a context that ends at the query's own position; a block-diagonal 2D codec
must reproduce the per-head prefill of each head's own latents; causality is
checked by changing latents past and before a query's position.  Planted
mistakes (attending the whole prompt, dropping the query's own key, taking
another head's up-projection, forgetting the offset p0) must fail the pins.
"""

import math

import numpy as np
import pytest

import oracle


def _case(g, H=2, M=4, p0=3, d=4, rk=3, rv=5):
    n = p0 + M
    Q = g.standard_normal((H, M, d))
    ck, cv = g.standard_normal((n, rk)), g.standard_normal((n, rv))
    uk, uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    muk, muv = g.standard_normal((H, d)), g.standard_normal((H, d))
    return Q, ck, cv, uk, uv, muk, muv


def _bruteforce(Q, ck, cv, uk, uv, muk, muv, scale, p0):
    H, M, d = Q.shape
    out = np.zeros((H, M, d))
    for h in range(H):
        for m in range(M):
            n_vis = p0 + m + 1
            K = [[sum(ck[n][j] * uk[h][i][j] for j in range(len(ck[n]))) + muk[h][i] for i in range(d)]
                 for n in range(n_vis)]
            V = [[sum(cv[n][j] * uv[h][i][j] for j in range(len(cv[n]))) + muv[h][i] for i in range(d)]
                 for n in range(n_vis)]
            s = [scale * sum(Q[h][m][i] * K[n][i] for i in range(d)) for n in range(n_vis)]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            tot = sum(e)
            for i in range(d):
                out[h, m, i] = sum(e[n] * V[n][i] for n in range(n_vis)) / tot
    return out


def test_prefill_2d_matches_pure_python_bruteforce():
    g = np.random.default_rng(11)
    for p0 in (0, 3):
        args = _case(g, p0=p0)
        ref = _bruteforce(*args, 0.41, p0)
        got = oracle.prefill_attn_2d(*args, scale=0.41, p0=p0)
        assert np.max(np.abs(got - ref)) < 1e-12


def test_each_row_is_the_2d_decode_at_its_position():
    g = np.random.default_rng(12)
    Q, ck, cv, uk, uv, muk, muv = _case(g, H=3, M=5, p0=6, d=8, rk=4, rv=6)
    out = oracle.prefill_attn_2d(Q, ck, cv, uk, uv, muk, muv, p0=6)
    for m in range(5):
        n = 6 + m + 1
        ref = oracle.decode_attn_2d(Q[:, m], ck[:n], cv[:n], uk, uv, muk, muv)
        assert np.max(np.abs(out[:, m] - ref)) < 1e-13


def test_block_diagonal_2d_codec_gives_per_head_prefill():
    # the shared latent holds head h's own latent in block h; head h's 2D
    # up-projection reads only its block, so the 2D prefill is per-head LLA
    g = np.random.default_rng(13)
    H, M, p0, d, rk, rv = 3, 4, 2, 4, 2, 3
    n = p0 + M
    ck_h, cv_h = g.standard_normal((H, n, rk)), g.standard_normal((H, n, rv))
    uk_h, uv_h = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    Q = g.standard_normal((H, M, d))
    ck2 = np.concatenate(list(ck_h), axis=1)
    cv2 = np.concatenate(list(cv_h), axis=1)
    uk2 = np.zeros((H, d, H * rk))
    uv2 = np.zeros((H, d, H * rv))
    for h in range(H):
        uk2[h, :, h * rk:(h + 1) * rk] = uk_h[h]
        uv2[h, :, h * rv:(h + 1) * rv] = uv_h[h]
    got = oracle.prefill_attn_2d(Q, ck2, cv2, uk2, uv2, scale=0.5, p0=p0)
    for h in range(H):
        ref = oracle.prefill_attn(Q[h], ck_h[h], cv_h[h], uk_h[h], uv_h[h], scale=0.5, p0=p0)
        assert np.max(np.abs(got[h] - ref)) < 1e-12


def test_prefill_2d_is_causal():
    g = np.random.default_rng(14)
    Q, ck, cv, uk, uv, muk, muv = _case(g, H=2, M=6, p0=2, d=4)
    a = oracle.prefill_attn_2d(Q, ck, cv, uk, uv, muk, muv, p0=2)
    ck2, cv2 = ck.copy(), cv.copy()
    ck2[5] += 3.0
    cv2[5] -= 2.0
    b = oracle.prefill_attn_2d(Q, ck2, cv2, uk, uv, muk, muv, p0=2)
    # token 5 is visible to rows m with 2 + m >= 5, i.e. m >= 3
    assert np.max(np.abs(a[:, :3] - b[:, :3])) == 0.0
    assert np.min(np.max(np.abs(a[:, 3:] - b[:, 3:]), axis=-1)) > 1e-6


def test_prefill_2d_batched():
    g = np.random.default_rng(15)
    B, H, M, p0, d, rk, rv = 2, 2, 3, 1, 4, 3, 2
    Q = g.standard_normal((B, H, M, d))
    ck, cv = g.standard_normal((B, p0 + M + 2, rk)), g.standard_normal((B, p0 + M + 2, rv))
    uk, uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    out = oracle.prefill_attn_2d_batched(Q, ck, cv, uk, uv, scale=0.3, p0=p0)
    z = np.zeros((H, d))
    for b in range(B):
        ref = _bruteforce(Q[b], ck[b], cv[b], uk, uv, z, z, 0.3, p0)
        assert np.max(np.abs(out[b] - ref)) < 1e-12
    part = oracle.prefill_attn_2d_batched(Q, ck, cv, uk, uv, scale=0.3, p0=p0, batches=[1])
    assert np.all(np.isnan(part[0])) and np.max(np.abs(part[1] - out[1])) == 0.0


# ---------------------------------------------------------------------------
# planted mistakes must fail the brute-force pin
# ---------------------------------------------------------------------------

def _not_causal(Q, ck, cv, uk, uv, muk, muv, scale, p0):
    H, M, d = Q.shape
    n = p0 + M
    return np.stack([np.stack([oracle.attention(Q[h, m], oracle.reconstruct(ck[:n], uk[h], muk[h]),
                                                oracle.reconstruct(cv[:n], uv[h], muv[h]), scale)
                               for m in range(M)]) for h in range(H)])


def _drops_own_key(Q, ck, cv, uk, uv, muk, muv, scale, p0):
    H, M, d = Q.shape
    out = np.zeros((H, M, d))
    for h in range(H):
        for m in range(M):
            n = max(p0 + m, 1)
            out[h, m] = oracle.attention(Q[h, m], oracle.reconstruct(ck[:n], uk[h], muk[h]),
                                         oracle.reconstruct(cv[:n], uv[h], muv[h]), scale)
    return out


def _other_heads_slice(Q, ck, cv, uk, uv, muk, muv, scale, p0):
    return oracle.prefill_attn_2d(Q, ck, cv, uk[::-1], uv, muk, muv, scale, p0)


def _no_offset(Q, ck, cv, uk, uv, muk, muv, scale, p0):
    return oracle.prefill_attn_2d(Q, ck, cv, uk, uv, muk, muv, scale, 0)


@pytest.mark.parametrize("mutant", [_not_causal, _drops_own_key, _other_heads_slice, _no_offset])
def test_bruteforce_pin_rejects_planted_mistakes(mutant):
    g = np.random.default_rng(16)
    args = _case(g, p0=3)
    ref = _bruteforce(*args, 0.41, 3)
    assert np.max(np.abs(oracle.prefill_attn_2d(*args, scale=0.41, p0=3) - ref)) < 1e-12
    wrong = mutant(*args, 0.41, 3)
    assert np.max(np.abs(wrong - ref)) > 1e-4
