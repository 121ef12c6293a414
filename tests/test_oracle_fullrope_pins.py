"""Pins of the oracle's full-RoPE reconstruct-then-attend decode (Sec. 3 "RoPE
and reconstruction": the latent is fit to the pre-RoPE content projection, and
the rotary phase, shared by the loops because a token's position does not
change across recurrence steps, is applied after reconstruction).

Independent formulations: pure-Python brute force (each half-split pair
rotated as a complex number with cmath, attention with math.exp); the
lossless orthogonal codec, where the result must be the teacher's own RoPE
attention over its pre-RoPE keys; position 0 everywhere, which must reduce to
the NoPE content path pinned elsewhere; and relative-position invariance.
Planted mistakes (rotating the values, adding the mean after the rotation, an
unrotated query, interleaved pairs, absorbing the key projection into the
query as if there were no rotation) must fail these pins.
"""

import cmath
import math

import numpy as np
import pytest

import oracle


def _rng(seed):
    return np.random.default_rng(seed)


def _py_rope(x, p, base):
    d = len(x)
    h = d // 2
    out = [0.0] * d
    for i in range(h):
        z = complex(x[i], x[i + h]) * cmath.exp(1j * p * base ** (-2.0 * i / d))
        out[i], out[i + h] = z.real, z.imag
    return out


def _py_attention(q, K, V, scale):
    s = [scale * sum(qi * ki for qi, ki in zip(q, k)) for k in K]
    m = max(s)
    e = [math.exp(x - m) for x in s]
    tot = sum(e)
    return [sum(e[n] * V[n][i] for n in range(len(V))) / tot for i in range(len(V[0]))]


def _case(g, d=8, rk=3, rv=5, N=7):
    q = g.standard_normal(d)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    Uk, Uv = g.standard_normal((d, rk)), g.standard_normal((d, rv))
    muk, muv = g.standard_normal(d), g.standard_normal(d)
    return q, ck, cv, Uk, Uv, muk, muv


def _bruteforce(q, ck, cv, Uk, Uv, muk, muv, scale, base, qpos, kpos=None):
    d, rk, rv, N = len(q), ck.shape[1], cv.shape[1], ck.shape[0]
    kpos = list(range(N)) if kpos is None else list(kpos)
    K = [_py_rope([sum(ck[n, j] * Uk[i, j] for j in range(rk)) + muk[i] for i in range(d)], kpos[n], base)
         for n in range(N)]
    V = [[sum(cv[n, j] * Uv[i, j] for j in range(rv)) + muv[i] for i in range(d)] for n in range(N)]
    return np.array(_py_attention(_py_rope(list(q), qpos, base), K, V, scale))


def test_fullrope_matches_pure_python_bruteforce():
    g = _rng(1)
    args = _case(g)
    for base, qpos in ((10000.0, 6), (50.0, 6), (10000.0, 40)):
        ref = _bruteforce(*args, 0.37, base, qpos)
        got = oracle.decode_attn_fullrope(*args, scale=0.37, base=base, q_pos=qpos)
        assert np.max(np.abs(got - ref)) < 1e-12


def test_fullrope_default_position_and_scale():
    g = _rng(2)
    args = _case(g, d=8, N=9)
    ref = _bruteforce(*args, 1.0 / math.sqrt(8), 10000.0, 8)  # newest token, 1/sqrt(d_head)
    assert np.max(np.abs(oracle.decode_attn_fullrope(*args) - ref)) < 1e-12


def test_fullrope_at_position_zero_is_the_content_path():
    g = _rng(3)
    q, ck, cv, Uk, Uv, muk, muv = _case(g, N=9)
    got = oracle.decode_attn_fullrope(q, ck, cv, Uk, Uv, muk, muv, scale=0.3, q_pos=0, k_pos=np.zeros(9))
    ref = oracle.decode_attn(q, ck, cv, Uk, Uv, muk, muv, scale=0.3)
    assert np.max(np.abs(got - ref)) < 1e-13


def test_fullrope_depends_on_relative_positions_only():
    g = _rng(4)
    args = _case(g, d=16, N=11)
    a = oracle.decode_attn_fullrope(*args, scale=0.5, q_pos=10)
    for s in (1, 64, 4093, 100000):
        b = oracle.decode_attn_fullrope(*args, scale=0.5, q_pos=10 + s, k_pos=np.arange(11) + s)
        assert np.max(np.abs(a - b)) < 1e-9
    c = oracle.decode_attn_fullrope(*args, scale=0.5, q_pos=30)  # a different query position matters
    assert np.max(np.abs(a - c)) > 1e-4


def test_orthogonal_codec_gives_the_teachers_rope_attention():
    """r = T*d with an orthogonal W_down and W_up,t = its loop slices is
    lossless, so full-RoPE latent attention at loop l equals the teacher's
    RoPE attention over its own pre-RoPE loop-l keys (pure Python)."""
    g = _rng(5)
    T, d, N = 3, 4, 6
    r = T * d
    qm, rm = np.linalg.qr(g.standard_normal((r, r)))
    Wk = qm * np.sign(np.diag(rm))
    qm, rm = np.linalg.qr(g.standard_normal((r, r)))
    Wv = qm * np.sign(np.diag(rm))
    xk, xv = g.standard_normal((N, r)), g.standard_normal((N, r))  # loop-stacked pre-RoPE K, V
    muk, muv = g.standard_normal(r), g.standard_normal(r)
    ck, cv = oracle.encode(xk, muk, Wk), oracle.encode(xv, muv, Wv)
    q = g.standard_normal(d)
    for l in range(T):
        sl = slice(l * d, (l + 1) * d)
        K = [_py_rope(list(xk[n, sl]), n, 10000.0) for n in range(N)]
        ref = _py_attention(_py_rope(list(q), N - 1, 10000.0), K, xv[:, sl].tolist(), 0.5)
        got = oracle.decode_attn_fullrope(q, ck, cv, Wk[sl, :], Wv[sl, :], muk[sl], muv[sl], 0.5)
        assert np.max(np.abs(got - np.array(ref))) < 1e-12


def test_fullrope_batched_positions_and_lengths():
    g = _rng(6)
    B, H, d, rk, rv, N = 2, 3, 8, 3, 4, 9
    q = g.standard_normal((B, H, d))
    ck, cv = g.standard_normal((B, H, N, rk)), g.standard_normal((B, H, N, rv))
    Uk, Uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    lens = [9, 4]
    out = oracle.decode_attn_fullrope_batched(q, ck, cv, Uk, Uv, scale=0.4, ctx_len=lens)
    out2 = oracle.decode_attn_fullrope_batched(q, ck, cv, Uk, Uv, scale=0.4, ctx_len=lens, q_pos=[20, 3])
    for b in range(B):
        for h in range(H):
            n = lens[b]
            z = np.zeros(d)
            ref = _bruteforce(q[b, h], ck[b, h, :n], cv[b, h, :n], Uk[h], Uv[h], z, z, 0.4, 10000.0, n - 1)
            assert np.max(np.abs(out[b, h] - ref)) < 1e-12
            ref2 = _bruteforce(q[b, h], ck[b, h, :n], cv[b, h, :n], Uk[h], Uv[h], z, z, 0.4, 10000.0,
                               [20, 3][b])
            assert np.max(np.abs(out2[b, h] - ref2)) < 1e-12


def test_key_mean_no_longer_cancels():
    # without rotation q . mu_k is the same for every key and cancels; with it,
    # q . R(n - p) mu_k depends on n, so the mean must be added before rotating
    g = _rng(7)
    q, ck, cv, Uk, Uv, muk, muv = _case(g, N=9)
    a = oracle.decode_attn_fullrope(q, ck, cv, Uk, Uv, muk, muv, scale=1.0)
    b = oracle.decode_attn_fullrope(q, ck, cv, Uk, Uv, None, muv, scale=1.0)
    assert np.max(np.abs(a - b)) > 1e-3
    c = oracle.decode_attn(q, ck, cv, Uk, Uv, muk, muv, scale=1.0)
    d = oracle.decode_attn(q, ck, cv, Uk, Uv, None, muv, scale=1.0)
    assert np.max(np.abs(c - d)) < 1e-13


# ---------------------------------------------------------------------------
# planted mistakes must fail the brute-force pin
# ---------------------------------------------------------------------------

def _rotate_values_too(q, ck, cv, Uk, Uv, muk, muv, scale, base, qpos):
    N, d = ck.shape[0], len(q)
    K = oracle.rope(oracle.reconstruct(ck, Uk, muk), np.arange(N), base)
    V = oracle.rope(oracle.reconstruct(cv, Uv, muv), np.arange(N), base)
    return oracle.attention(oracle.rope(q, qpos, base), K, V, scale)


def _mean_after_rotation(q, ck, cv, Uk, Uv, muk, muv, scale, base, qpos):
    N = ck.shape[0]
    K = oracle.rope(oracle.reconstruct(ck, Uk, None), np.arange(N), base) + muk
    V = oracle.reconstruct(cv, Uv, muv)
    return oracle.attention(oracle.rope(q, qpos, base), K, V, scale)


def _unrotated_query(q, ck, cv, Uk, Uv, muk, muv, scale, base, qpos):
    return oracle.decode_attn_fullrope(q, ck, cv, Uk, Uv, muk, muv, scale, base, q_pos=0)


def _interleaved_pairs(q, ck, cv, Uk, Uv, muk, muv, scale, base, qpos):
    def rope_il(x, pos):
        x = np.asarray(x, dtype=np.float64)
        dd = x.shape[-1]
        ang = np.asarray(pos, dtype=np.float64)[..., None] * base ** (-2.0 * np.arange(dd // 2) / dd)
        out = x.copy()
        out[..., 0::2] = x[..., 0::2] * np.cos(ang) - x[..., 1::2] * np.sin(ang)
        out[..., 1::2] = x[..., 1::2] * np.cos(ang) + x[..., 0::2] * np.sin(ang)
        return out
    N = ck.shape[0]
    K = rope_il(oracle.reconstruct(ck, Uk, muk), np.arange(N))
    V = oracle.reconstruct(cv, Uv, muv)
    return oracle.attention(rope_il(q, qpos), K, V, scale)


def _absorbed_as_if_nope(q, ck, cv, Uk, Uv, muk, muv, scale, base, qpos):
    return oracle.decode_attn_absorbed(oracle.rope(q, qpos, base), ck, cv, Uk, Uv, muk, muv, scale)


@pytest.mark.parametrize("mutant", [_rotate_values_too, _mean_after_rotation, _unrotated_query,
                                    _interleaved_pairs, _absorbed_as_if_nope])
def test_bruteforce_pin_rejects_planted_mistakes(mutant):
    g = _rng(8)
    args = _case(g)
    ref = _bruteforce(*args, 0.37, 10000.0, 6)
    assert np.max(np.abs(oracle.decode_attn_fullrope(*args, scale=0.37, q_pos=6) - ref)) < 1e-12
    wrong = mutant(*args, 0.37, 10000.0, 6)
    assert np.max(np.abs(wrong - ref)) > 1e-4
