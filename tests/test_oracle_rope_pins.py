"""Pins of the oracle's decoupled rotary branch (App. J "Absorbed attention":
a NoPE content path plus a small explicit rotary branch shared across loops).

The rotation is pinned by an independent formulation (each half-split pair
(x_i, x_{i+h}) is the complex number x_i + j x_{i+h}, multiplied by
exp(j p base^(-2i/d)) with Python's cmath), by the group properties of a
rotation (identity at position 0, composition, norm preservation, relative
position), and the attention with the branch by pure-Python brute force and by
special cases.  Planted mistakes at the end must fail these pins.
"""

import cmath
import math

import numpy as np
import pytest

import oracle


def _rng(seed):
    return np.random.default_rng(seed)


def _py_rope(x, p, base):
    """Half-split rotary embedding in pure Python via complex multiplication."""
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


# ---------------------------------------------------------------------------
# the rotation itself
# ---------------------------------------------------------------------------

def test_rope_position_zero_is_identity():
    x = _rng(1).standard_normal((5, 8))
    assert np.array_equal(oracle.rope(x, 0.0), x)


def test_rope_unit_vectors_show_half_split_pairing():
    # d = 4, base b: feature 0 pairs with feature 2 (angle p), feature 1 with 3 (angle p / sqrt(b))
    p, b = 0.7, 100.0
    e = np.eye(4)
    assert np.allclose(oracle.rope(e[0], p, b), [math.cos(p), 0, math.sin(p), 0], atol=1e-15)
    assert np.allclose(oracle.rope(e[2], p, b), [-math.sin(p), 0, math.cos(p), 0], atol=1e-15)
    a1 = p / math.sqrt(b)
    assert np.allclose(oracle.rope(e[1], p, b), [0, math.cos(a1), 0, math.sin(a1)], atol=1e-15)


@pytest.mark.parametrize("d,p,base", [(2, 3.0, 10000.0), (8, 17.0, 10000.0), (64, 4095.0, 10000.0),
                                      (32, 262143.0, 500000.0)])
def test_rope_is_complex_multiplication(d, p, base):
    x = _rng(d).standard_normal(d)
    ref = _py_rope(list(x), p, base)
    assert np.max(np.abs(oracle.rope(x, p, base) - np.array(ref))) < 1e-9


def test_rope_preserves_norm_and_composes():
    g = _rng(2)
    x = g.standard_normal((7, 16))
    a, b = 11.0, 250.0
    r = oracle.rope(x, a)
    assert np.allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    assert np.allclose(oracle.rope(r, b), oracle.rope(x, a + b), atol=1e-12)


def test_rope_scores_depend_on_relative_position_only():
    g = _rng(3)
    q, k = g.standard_normal(64), g.standard_normal(64)
    for m, n, s in [(10, 3, 100), (0, 0, 4096), (5000, 17, 31)]:
        s0 = oracle.rope(q, m) @ oracle.rope(k, n)
        s1 = oracle.rope(q, m + s) @ oracle.rope(k, n + s)
        assert abs(s0 - s1) < 1e-9


def test_rope_per_row_positions():
    g = _rng(4)
    x = g.standard_normal((3, 8))
    pos = np.array([0.0, 5.0, 9.0])
    got = oracle.rope(x, pos)
    for i in range(3):
        assert np.allclose(got[i], oracle.rope(x[i], pos[i]), atol=1e-15)


# ---------------------------------------------------------------------------
# attention with the rotary branch
# ---------------------------------------------------------------------------

def _case(g, d=4, dr=4, rk=3, rv=5, N=6):
    q, qr = g.standard_normal(d), g.standard_normal(dr)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    kr = g.standard_normal((N, dr))
    Uk, Uv = g.standard_normal((d, rk)), g.standard_normal((d, rv))
    muk, muv = g.standard_normal(d), g.standard_normal(d)
    return q, qr, ck, cv, kr, Uk, Uv, muk, muv


def _bruteforce(q, qr, ck, cv, kr, Uk, Uv, muk, muv, scale, base, qpos):
    d, rk, rv, N = len(q), ck.shape[1], cv.shape[1], ck.shape[0]
    K = [[sum(ck[n, j] * Uk[i, j] for j in range(rk)) + muk[i] for i in range(d)]
         + _py_rope(list(kr[n]), n, base) for n in range(N)]
    V = [[sum(cv[n, j] * Uv[i, j] for j in range(rv)) + muv[i] for i in range(d)] for n in range(N)]
    return np.array(_py_attention(list(q) + _py_rope(list(qr), qpos, base), K, V, scale))


def test_decode_rope_matches_pure_python_bruteforce():
    g = _rng(5)
    args = _case(g)
    for base in (10000.0, 50.0):
        ref = _bruteforce(*args, 0.41, base, 5)
        got = oracle.decode_attn_rope(*args, scale=0.41, base=base)
        assert np.max(np.abs(got - ref)) < 1e-12


def test_decode_rope_default_position_and_scale():
    g = _rng(6)
    args = _case(g, d=8, dr=4, N=9)
    ref = _bruteforce(*args, 1.0 / math.sqrt(12), 10000.0, 8)  # the newest token, 1/sqrt(d + d_rope)
    assert np.max(np.abs(oracle.decode_attn_rope(*args) - ref)) < 1e-12


def test_zero_rotary_branch_is_the_content_path():
    g = _rng(7)
    q, qr, ck, cv, kr, Uk, Uv, muk, muv = _case(g, N=9)
    got = oracle.decode_attn_rope(q, np.zeros_like(qr), ck, cv, kr, Uk, Uv, muk, muv, scale=0.3)
    ref = oracle.decode_attn(q, ck, cv, Uk, Uv, muk, muv, scale=0.3)
    assert np.max(np.abs(got - ref)) < 1e-13


def test_rotary_only_attention_is_shift_invariant():
    # with the content path switched off (U_k = 0), only relative positions matter
    g = _rng(8)
    q, qr, ck, cv, kr, Uk, Uv, muk, muv = _case(g, d=4, dr=8, N=7)
    Uk = np.zeros_like(Uk)
    a = oracle.decode_attn_rope(q, qr, ck, cv, kr, Uk, Uv, None, muv, scale=1.0)
    b = oracle.decode_attn_rope(q, qr, ck, cv, kr, Uk, Uv, None, muv, scale=1.0,
                                q_pos=6 + 1000, k_pos=np.arange(7) + 1000)
    assert np.max(np.abs(a - b)) < 1e-10


def test_prefill_rope_rows_are_decodes():
    g = _rng(9)
    d, dr, rk, rv, p0, M = 4, 4, 3, 2, 3, 4
    Q, QR = g.standard_normal((M, d)), g.standard_normal((M, dr))
    ck, cv = g.standard_normal((p0 + M, rk)), g.standard_normal((p0 + M, rv))
    kr = g.standard_normal((p0 + M, dr))
    Uk, Uv = g.standard_normal((d, rk)), g.standard_normal((d, rv))
    out = oracle.prefill_attn_rope(Q, QR, ck, cv, kr, Uk, Uv, scale=0.5, p0=p0)
    for m in range(M):
        n = p0 + m + 1
        ref = _bruteforce(Q[m], QR[m], ck[:n], cv[:n], kr[:n], Uk, Uv, np.zeros(d), np.zeros(d), 0.5,
                          10000.0, p0 + m)
        assert np.max(np.abs(out[m] - ref)) < 1e-12


def test_shared_rotary_key_equals_replicated_heads():
    g = _rng(10)
    B, H, d, dr, rk, rv, N = 2, 3, 4, 4, 3, 2, 5
    q, qr = g.standard_normal((B, H, d)), g.standard_normal((B, H, dr))
    ck, cv = g.standard_normal((B, H, N, rk)), g.standard_normal((B, H, N, rv))
    kr1 = g.standard_normal((B, 1, N, dr))
    Uk, Uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    a = oracle.decode_attn_rope_batched(q, qr, ck, cv, kr1, Uk, Uv)
    b = oracle.decode_attn_rope_batched(q, qr, ck, cv, np.repeat(kr1, H, axis=1), Uk, Uv)
    assert np.array_equal(a, b)
    for bb in range(B):
        for h in range(H):
            ref = oracle.decode_attn_rope(q[bb, h], qr[bb, h], ck[bb, h], cv[bb, h], kr1[bb, 0], Uk[h], Uv[h])
            assert np.array_equal(a[bb, h], ref)
    P = oracle.prefill_attn_rope_batched(q[:, :, None], qr[:, :, None], ck, cv, kr1, Uk, Uv, p0=N - 1)
    assert np.max(np.abs(P[:, :, 0] - a)) < 1e-13


# ---------------------------------------------------------------------------
# planted mistakes must fail the pins above
# ---------------------------------------------------------------------------

def _rope_interleaved(x, pos, base=10000.0):
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    inv = base ** (-2.0 * np.arange(d // 2) / d)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv
    out = x.copy()
    out[..., 0::2] = x[..., 0::2] * np.cos(ang) - x[..., 1::2] * np.sin(ang)
    out[..., 1::2] = x[..., 1::2] * np.cos(ang) + x[..., 0::2] * np.sin(ang)
    return out


def _rope_wrong_sign(x, pos, base=10000.0):
    return oracle.rope(x, -np.asarray(pos, dtype=np.float64), base)


def _rope_wrong_freq(x, pos, base=10000.0):
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    inv = base ** (-1.0 * np.arange(d // 2) / d)  # exponent -i/d instead of -2i/d
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv
    h = d // 2
    return np.concatenate([x[..., :h] * np.cos(ang) - x[..., h:] * np.sin(ang),
                           x[..., h:] * np.cos(ang) + x[..., :h] * np.sin(ang)], axis=-1)


def _pins_pass(rope_fn):
    try:
        e = np.eye(4)
        p, b = 0.7, 100.0
        if not np.allclose(rope_fn(e[0], p, b), [math.cos(p), 0, math.sin(p), 0], atol=1e-15):
            return False
        if not np.allclose(rope_fn(e[1], p, b), [0, math.cos(p / 10), 0, math.sin(p / 10)], atol=1e-15):
            return False
        x = _rng(8).standard_normal(8)
        return np.max(np.abs(rope_fn(x, 17.0, 10000.0) - np.array(_py_rope(list(x), 17.0, 10000.0)))) < 1e-9
    except Exception:
        return False


def test_rope_pins_accept_the_oracle():
    assert _pins_pass(oracle.rope)


@pytest.mark.parametrize("mutant", [_rope_interleaved, _rope_wrong_sign, _rope_wrong_freq])
def test_rope_pins_reject_planted_mistakes(mutant):
    assert not _pins_pass(mutant)


def test_decode_pin_rejects_unrotated_query():
    g = _rng(11)
    q, qr, ck, cv, kr, Uk, Uv, muk, muv = _case(g)
    ref = _bruteforce(q, qr, ck, cv, kr, Uk, Uv, muk, muv, 0.41, 10000.0, 5)
    # a slip that rotates the keys but feeds the query unrotated (position 0)
    wrong = oracle.decode_attn_rope(q, qr, ck, cv, kr, Uk, Uv, muk, muv, scale=0.41, q_pos=0)
    assert np.max(np.abs(wrong - ref)) > 1e-3


# ---------------------------------------------------------------------------
# the batched prefill wrapper: every row of several queries past an offset,
# against the brute force above, with one rotary key per token (shared by the
# heads) and one per head
# ---------------------------------------------------------------------------

def _batched_prefill_case(g, Hr):
    B, H, d, dr, rk, rv, p0, M = 2, 3, 4, 4, 3, 2, 5, 6
    Q, QR = g.standard_normal((B, H, M, d)), g.standard_normal((B, H, M, dr))
    ck, cv = g.standard_normal((B, H, p0 + M, rk)), g.standard_normal((B, H, p0 + M, rv))
    kr = g.standard_normal((B, Hr, p0 + M, dr))
    Uk, Uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    muk, muv = g.standard_normal((H, d)), g.standard_normal((H, d))
    return Q, QR, ck, cv, kr, Uk, Uv, muk, muv, p0


def _batched_prefill_pin_passes(fn, Hr):
    g = _rng(40 + Hr)
    Q, QR, ck, cv, kr, Uk, Uv, muk, muv, p0 = _batched_prefill_case(g, Hr)
    B, H, M, _ = Q.shape
    out = fn(Q, QR, ck, cv, kr, Uk, Uv, muk, muv, 0.45, 500.0, p0)
    for b in range(B):
        for h in range(H):
            hr = 0 if Hr == 1 else h
            for m in range(M):
                n = p0 + m + 1
                ref = _bruteforce(Q[b, h, m], QR[b, h, m], ck[b, h, :n], cv[b, h, :n], kr[b, hr, :n],
                                  Uk[h], Uv[h], muk[h], muv[h], 0.45, 500.0, p0 + m)
                if not np.max(np.abs(out[b, h, m] - ref)) < 1e-12:
                    return False
    return True


def _oracle_batched(Q, QR, ck, cv, kr, Uk, Uv, muk, muv, scale, base, p0):
    return oracle.prefill_attn_rope_batched(Q, QR, ck, cv, kr, Uk, Uv, muk, muv, scale, base, p0)


def _batched_mutant(q_pos_of, n_of):
    """The batched wrapper with one slip in the query position or the causal length."""
    def fn(Q, QR, ck, cv, kr, Uk, Uv, muk, muv, scale, base, p0):
        B, H, M, d = Q.shape
        Hr = kr.shape[1]
        out = np.empty((B, H, M, d))
        for b in range(B):
            for h in range(H):
                hr = 0 if Hr == 1 else h
                for m in range(M):
                    n = n_of(p0, m)
                    out[b, h, m] = oracle.decode_attn_rope(Q[b, h, m], QR[b, h, m], ck[b, h, :n], cv[b, h, :n],
                                                           kr[b, hr, :n], Uk[h], Uv[h], muk[h], muv[h], scale,
                                                           base, q_pos=q_pos_of(p0, m))
        return out
    return fn


@pytest.mark.parametrize("Hr", [1, 3])
def test_prefill_rope_batched_rows_match_bruteforce(Hr):
    assert _batched_prefill_pin_passes(_oracle_batched, Hr)


@pytest.mark.parametrize("Hr", [1, 3])
@pytest.mark.parametrize("slip", ["q_pos=p0", "n=p0+1", "q_pos=m", "n=m+1"])
def test_prefill_rope_batched_pin_rejects_slips(Hr, slip):
    good_q, good_n = (lambda p0, m: p0 + m), (lambda p0, m: p0 + m + 1)
    mutants = {
        "q_pos=p0": _batched_mutant(lambda p0, m: p0, good_n),
        "n=p0+1": _batched_mutant(good_q, lambda p0, m: p0 + 1),
        "q_pos=m": _batched_mutant(lambda p0, m: m, good_n),
        "n=m+1": _batched_mutant(good_q, lambda p0, m: m + 1),
    }
    assert _batched_prefill_pin_passes(_batched_mutant(good_q, good_n), Hr)  # the harness itself
    assert not _batched_prefill_pin_passes(mutants[slip], Hr)
