"""Pins of the float64 CPU oracle against things other than itself.

Each test fixes part of the oracle with something the paper or the mathematics
determines independently: values the paper prints (tests/golden/), brute force
in pure Python (math.exp, no numpy) on tiny inputs, closed forms, and special
cases that reduce to textbook results (an orthogonal codec is lossless; the
SVD codec obeys Eckart-Young).  The planted-mistake tests at the end show that
plausible slips in the oracle (a dropped term, a wrong index or sign, a
transposed operand) fail these pins.
"""

import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


# ---------------------------------------------------------------------------
# Eq. 4 and the bytes accounting (printed values).
# ---------------------------------------------------------------------------

def test_rho_matches_printed_tiers():
    n = 0
    for T, d, rk, rv, printed, dec, *_ in _rows("rho_tiers.txt"):
        rho = oracle.compression_ratio(int(T), int(d), int(rk), int(rv))
        assert isinstance(rho, Fraction)
        assert f"{float(rho):.{int(dec)}f}" == printed, (rk, rv, rho)
        n += 1
    assert n == 8


def test_rho_exact_fractions_of_extreme_tiers():
    # 10.67x and 21.33x are printed (tab:scale, tab:isocache); with the 3:5 split
    # of every printed tier they are (36, 60) and (18, 30): 1024/96 and 1024/48.
    assert oracle.compression_ratio(4, 128, 36, 60) == Fraction(32, 3)
    assert oracle.compression_ratio(4, 128, 18, 30) == Fraction(64, 3)
    assert f"{float(Fraction(32, 3)):.2f}" == "10.67"
    assert f"{float(Fraction(64, 3)):.2f}" == "21.33"
    assert f"{float(Fraction(64, 3)):.1f}" == "21.3"


def test_rho_huginn_rows_share_one_geometry():
    # tab:huginn: rho * (r_k + r_v) must be the same 2*R*d_head on every row.
    prods = {int(rho) * (int(rk) + int(rv)) for rho, rk, rv, *_ in _rows("huginn_ranks.txt")}
    assert len(prods) == 1
    (p,) = prods
    d = Fraction(p, 2 * 32)
    # and the oracle's Eq. 4 reproduces each printed ratio at that geometry
    for rho, rk, rv, *_ in _rows("huginn_ranks.txt"):
        assert oracle.compression_ratio(32, int(d), int(rk), int(rv)) == int(rho)


def test_rho_rejects_nonpositive():
    for bad in [(0, 128, 96, 160), (4, 0, 96, 160), (4, 128, 0, 160), (4, 128, 96, -1)]:
        with pytest.raises(ValueError):
            oracle.compression_ratio(*bad)


UNIT = {"KiB": 1024, "MiB": 1024 ** 2, "GiB": 1024 ** 3}


def test_cache_bytes_match_tab_memory():
    n = 0
    for layers, tokens, rk, rv, val, unit, *_ in _rows("cache_bytes.txt"):
        latent = int(rk) > 0
        b = oracle.cache_bytes(int(layers), 16, 4, 128, int(rk), int(rv), int(tokens), 2, latent)
        assert b == int(val) * UNIT[unit], (layers, tokens, rk, rv)
        n += 1
    assert n == 10


def test_cache_ratio_equals_rho():
    for rk, rv in [(96, 160), (192, 320), (36, 60), (18, 30), (120, 200)]:
        t = oracle.cache_bytes(24, 16, 4, 128, rk, rv, 1, 2, False)
        l = oracle.cache_bytes(24, 16, 4, 128, rk, rv, 1, 2, True)
        assert Fraction(t, l) == oracle.compression_ratio(4, 128, rk, rv)


# ---------------------------------------------------------------------------
# Pure-Python brute force (no numpy in the computation) on tiny inputs.
# ---------------------------------------------------------------------------

def _py_attention(q, K, V, scale):
    s = [scale * sum(qi * ki for qi, ki in zip(q, k)) for k in K]
    m = max(s)
    e = [math.exp(x - m) for x in s]
    tot = sum(e)
    return [sum(e[n] * V[n][i] for n in range(len(V))) / tot for i in range(len(V[0]))]


def _rng(seed):
    return np.random.default_rng(seed)


def test_encode_matches_elementwise_sum():
    g = _rng(1)
    T, d, r, M = 3, 4, 5, 6
    x = g.standard_normal((M, T * d))
    mu = g.standard_normal(T * d)
    W = g.standard_normal((T * d, r))
    c = oracle.encode(x, mu, W)
    for m in range(M):
        for j in range(r):
            ref = sum((x[m, i] - mu[i]) * W[i, j] for i in range(T * d))
            assert abs(c[m, j] - ref) < 1e-12


def test_stack_loops_is_loop_major():
    a, b = np.arange(3.0), np.arange(3.0) + 10
    assert list(oracle.stack_loops([a, b])) == [0, 1, 2, 10, 11, 12]


def test_reconstruct_matches_elementwise_sum():
    g = _rng(2)
    d, r, N = 4, 3, 5
    c = g.standard_normal((N, r))
    U = g.standard_normal((d, r))
    mu = g.standard_normal(d)
    x = oracle.reconstruct(c, U, mu)
    for n in range(N):
        for i in range(d):
            ref = sum(c[n, j] * U[i, j] for j in range(r)) + mu[i]
            assert abs(x[n, i] - ref) < 1e-12


def test_decode_matches_pure_python_bruteforce():
    g = _rng(3)
    d, rk, rv, N = 4, 3, 5, 7
    q = g.standard_normal(d)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    Uk, Uv = g.standard_normal((d, rk)), g.standard_normal((d, rv))
    muk, muv = g.standard_normal(d), g.standard_normal(d)
    scale = 0.37
    K = [[sum(ck[n, j] * Uk[i, j] for j in range(rk)) + muk[i] for i in range(d)] for n in range(N)]
    V = [[sum(cv[n, j] * Uv[i, j] for j in range(rv)) + muv[i] for i in range(d)] for n in range(N)]
    ref = _py_attention(list(q), K, V, scale)
    got = oracle.decode_attn(q, ck, cv, Uk, Uv, muk, muv, scale)
    assert np.max(np.abs(got - np.array(ref))) < 1e-12
    got_abs = oracle.decode_attn_absorbed(q, ck, cv, Uk, Uv, muk, muv, scale)
    assert np.max(np.abs(got_abs - np.array(ref))) < 1e-12


def test_default_scale_is_teachers():
    assert oracle.default_scale(128) == 1.0 / math.sqrt(128)
    g = _rng(4)
    d, N = 8, 5
    q = g.standard_normal(d)
    ck, cv = g.standard_normal((N, d)), g.standard_normal((N, d))
    I = np.eye(d)
    ref = _py_attention(list(q), ck.tolist(), cv.tolist(), 1.0 / math.sqrt(d))
    got = oracle.decode_attn(q, ck, cv, I, I)
    assert np.max(np.abs(got - np.array(ref))) < 1e-12


# ---------------------------------------------------------------------------
# App. J identities: absorbed form == reconstruct-then-attend, to fp64 rounding.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d,rk,rv,N", [(128, 96, 160, 64), (16, 3, 5, 33), (32, 36, 60, 1)])
def test_absorbed_equals_plain(d, rk, rv, N):
    g = _rng(5 + N)
    q = g.standard_normal(d)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    Uk = g.standard_normal((d, rk)) / math.sqrt(rk)
    Uv = g.standard_normal((d, rv)) / math.sqrt(rv)
    muk, muv = g.standard_normal(d), g.standard_normal(d)
    a = oracle.decode_attn(q, ck, cv, Uk, Uv, muk, muv)
    b = oracle.decode_attn_absorbed(q, ck, cv, Uk, Uv, muk, muv)
    assert np.linalg.norm(a - b) <= 1e-12 * np.linalg.norm(a)


# ---------------------------------------------------------------------------
# Textbook special cases of the codec (Sec. 3 "Initialization and conversion").
# ---------------------------------------------------------------------------

def _orthogonal(n, g):
    qm, rm = np.linalg.qr(g.standard_normal((n, n)))
    return qm * np.sign(np.diag(rm))


def test_full_rank_orthogonal_codec_is_lossless_attention():
    """r = T*d with an orthogonal W_down and W_up,t = its loop slices: every
    loop's K/V is reconstructed exactly, so latent attention at loop l equals
    the teacher's attention over its own loop-l K/V (computed in pure Python)."""
    g = _rng(7)
    T, d, N = 3, 4, 6
    r = T * d
    Wk, Wv = _orthogonal(r, g), _orthogonal(r, g)
    xk = g.standard_normal((N, T * d))        # loop-stacked teacher keys (Eq. 1)
    xv = g.standard_normal((N, T * d))
    muk, muv = g.standard_normal(T * d), g.standard_normal(T * d)
    ck, cv = oracle.encode(xk, muk, Wk), oracle.encode(xv, muv, Wv)
    q = g.standard_normal(d)
    for l in range(T):
        sl = slice(l * d, (l + 1) * d)
        Ukl, Uvl = Wk[sl, :], Wv[sl, :]      # loop slices of W_down
        assert np.max(np.abs(oracle.reconstruct(ck, Ukl, muk[sl]) - xk[:, sl])) < 1e-12
        ref = _py_attention(list(q), xk[:, sl].tolist(), xv[:, sl].tolist(), 0.5)
        got = oracle.decode_attn(q, ck, cv, Ukl, Uvl, muk[sl], muv[sl], 0.5)
        assert np.max(np.abs(got - np.array(ref))) < 1e-12


def test_svd_codec_obeys_eckart_young():
    """W_down = top-r right singular vectors of the centred stacked-loop matrix,
    W_up,t = loop slices (Sec. 3; App. A): encode-then-reconstruct is the
    orthogonal projector onto the top-r subspace, its error is the energy of
    the discarded singular values, and the projector is idempotent."""
    g = _rng(8)
    T, d, n, r = 4, 6, 200, 7
    X = g.standard_normal((n, T * d)) @ g.standard_normal((T * d, T * d))
    mu = X.mean(axis=0)
    _, S, Vt = np.linalg.svd(X - mu, full_matrices=False)
    Wd = Vt[:r].T                             # [T*d, r]
    C = oracle.encode(X, mu, Wd)
    Xhat = np.concatenate([oracle.reconstruct(C, Wd[l * d:(l + 1) * d, :], mu[l * d:(l + 1) * d])
                           for l in range(T)], axis=1)
    err = np.linalg.norm(X - Xhat)
    assert abs(err - math.sqrt(float(np.sum(S[r:] ** 2)))) < 1e-9 * np.linalg.norm(X)
    C2 = oracle.encode(Xhat, mu, Wd)
    assert np.max(np.abs(C2 - C)) < 1e-9 * np.max(np.abs(C))


# ---------------------------------------------------------------------------
# Closed forms of the attention.
# ---------------------------------------------------------------------------

def _codec(g, d, rk, rv):
    return (g.standard_normal((d, rk)) / math.sqrt(rk), g.standard_normal((d, rv)) / math.sqrt(rv),
            g.standard_normal(d), g.standard_normal(d))


@pytest.mark.parametrize("fn", [oracle.decode_attn, oracle.decode_attn_absorbed])
def test_single_token_context(fn):
    g = _rng(9)
    d, rk, rv = 16, 6, 10
    Uk, Uv, muk, muv = _codec(g, d, rk, rv)
    ck, cv = g.standard_normal((1, rk)), g.standard_normal((1, rv))
    q = g.standard_normal(d)
    o = fn(q, ck, cv, Uk, Uv, muk, muv)
    assert np.max(np.abs(o - (Uv @ cv[0] + muv))) < 1e-12


@pytest.mark.parametrize("fn", [oracle.decode_attn, oracle.decode_attn_absorbed])
def test_zero_query_is_uniform_average(fn):
    g = _rng(10)
    d, rk, rv, N = 16, 6, 10, 9
    Uk, Uv, muk, muv = _codec(g, d, rk, rv)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    o = fn(np.zeros(d), ck, cv, Uk, Uv, muk, muv)
    assert np.max(np.abs(o - (Uv @ cv.mean(axis=0) + muv))) < 1e-12


@pytest.mark.parametrize("fn", [oracle.decode_attn, oracle.decode_attn_absorbed])
def test_dominant_key_selects_its_value(fn):
    g = _rng(11)
    d, rk, rv, N = 16, 16, 10, 9
    Uk = np.eye(d)                             # K_l = c_k exactly
    _, Uv, _, muv = _codec(g, d, rk, rv)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    star = 4
    q = 1e3 * ck[star] / np.linalg.norm(ck[star]) ** 2 * 10
    o = fn(q, ck, cv, Uk, Uv, None, muv, 1.0)
    assert np.max(np.abs(o - (Uv @ cv[star] + muv))) < 1e-9


@pytest.mark.parametrize("fn", [oracle.decode_attn, oracle.decode_attn_absorbed])
def test_mean_terms(fn):
    """mu_k adds q.mu_k to every score, which softmax ignores; mu_v adds to the
    output because the weights sum to one (Eq. 3)."""
    g = _rng(12)
    d, rk, rv, N = 16, 6, 10, 11
    Uk, Uv, muk, muv = _codec(g, d, rk, rv)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    q = g.standard_normal(d)
    base = fn(q, ck, cv, Uk, Uv, None, None)
    assert np.max(np.abs(fn(q, ck, cv, Uk, Uv, muk, None) - base)) < 1e-12
    assert np.max(np.abs(fn(q, ck, cv, Uk, Uv, None, muv) - (base + muv))) < 1e-12


def test_empty_context_rejected():
    g = _rng(13)
    with pytest.raises(ValueError):
        oracle.decode_attn(g.standard_normal(4), np.zeros((0, 2)), np.zeros((0, 3)),
                           g.standard_normal((4, 2)), g.standard_normal((4, 3)))


# ---------------------------------------------------------------------------
# Prefill and split-merge structure.
# ---------------------------------------------------------------------------

def test_prefill_rows_are_decodes():
    g = _rng(14)
    d, rk, rv, p0, M = 8, 3, 5, 4, 6
    Uk, Uv, muk, muv = _codec(g, d, rk, rv)
    ck, cv = g.standard_normal((p0 + M, rk)), g.standard_normal((p0 + M, rv))
    Q = g.standard_normal((M, d))
    P = oracle.prefill_attn(Q, ck, cv, Uk, Uv, muk, muv, 0.3, p0)
    for m in range(M):
        K = [[sum(ck[n, j] * Uk[i, j] for j in range(rk)) + muk[i] for i in range(d)]
             for n in range(p0 + m + 1)]
        V = [[sum(cv[n, j] * Uv[i, j] for j in range(rv)) + muv[i] for i in range(d)]
             for n in range(p0 + m + 1)]
        ref = _py_attention(list(Q[m]), K, V, 0.3)
        assert np.max(np.abs(P[m] - np.array(ref))) < 1e-12
    # the causal boundary: row 0 sees exactly p0+1 keys, so a key after it has no influence
    ck2 = ck.copy()
    ck2[p0 + 1:] += 100.0
    P2 = oracle.prefill_attn(Q[:1], ck2, cv, Uk, Uv, muk, muv, 0.3, p0)
    assert np.max(np.abs(P2[0] - P[0])) < 1e-12


def test_split_merge_equals_whole():
    g = _rng(15)
    N, rk, rv = 100, 6, 9
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    qt = 2.0 * g.standard_normal(rk)
    a = oracle.softmax(ck @ qt)
    whole = a @ cv
    # brute-force weights in pure Python for one component
    s = [sum(ck[n, j] * qt[j] for j in range(rk)) for n in range(N)]
    m = max(s)
    e = [math.exp(x - m) for x in s]
    ref0 = sum(e[n] * cv[n, 0] for n in range(N)) / sum(e)
    assert abs(whole[0] - ref0) < 1e-12
    for cuts in ([0, 100], [0, 1, 100], [0, 37, 38, 90, 100], list(range(0, 101, 10))):
        parts = [oracle.split_partial(qt, ck[a_:b_], cv[a_:b_]) for a_, b_ in zip(cuts, cuts[1:])]
        assert np.max(np.abs(oracle.split_merge(parts) - whole)) < 1e-12


def test_batched_wrappers_agree_with_unit_calls():
    g = _rng(16)
    B, H, d, rk, rv, N, T = 2, 3, 8, 3, 5, 7, 2
    q = g.standard_normal((B, H, d))
    ck, cv = g.standard_normal((B, H, N, rk)), g.standard_normal((B, H, N, rv))
    Uk, Uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    muk, muv = g.standard_normal((H, d)), g.standard_normal((H, d))
    out = oracle.decode_attn_batched(q, ck, cv, Uk, Uv, muk, muv, 0.5, ctx_len=[7, 4])
    for b in range(B):
        n = [7, 4][b]
        for h in range(H):
            ref = oracle.decode_attn(q[b, h], ck[b, h, :n], cv[b, h, :n], Uk[h], Uv[h], muk[h], muv[h], 0.5)
            assert np.max(np.abs(out[b, h] - ref)) == 0.0
    x = g.standard_normal((B, 4, H, T * d))
    mu = g.standard_normal((H, T * d))
    wdt = g.standard_normal((H, rk, T * d))
    c = oracle.encode_batched(x, mu, wdt)
    for b in range(B):
        for h in range(H):
            for m in range(4):
                for j in range(rk):
                    ref = sum((x[b, m, h, i] - mu[h, i]) * wdt[h, j, i] for i in range(T * d))
                    assert abs(c[b, h, m, j] - ref) < 1e-12
    Q = g.standard_normal((B, H, 3, d))
    P = oracle.prefill_attn_batched(Q, ck, cv, Uk, Uv, muk, muv, 0.5, p0=2, rows=[0, 2])
    assert np.all(np.isnan(P[:, :, 1]))
    ref = oracle.decode_attn(Q[1, 2, 2], ck[1, 2, :5], cv[1, 2, :5], Uk[2], Uv[2], muk[2], muv[2], 0.5)
    assert np.max(np.abs(P[1, 2, 2] - ref)) == 0.0


# ---------------------------------------------------------------------------
# Planted mistakes: each variant of the oracle below carries one plausible slip.
# The pins above, re-run against the variant, must reject it.
# ---------------------------------------------------------------------------

def _decode_pins_pass(decode_fn):
    """The orthogonal-codec pin above (against pure-Python attention), packaged
    so it can be run against a variant; T=1 makes the up-projection square."""
    for T, d in ((2, 4), (1, 5)):
        g = _rng(21 + T)
        N = 6
        r = T * d
        Wk, Wv = _orthogonal(r, g), _orthogonal(r, g)
        xk, xv = g.standard_normal((N, r)), g.standard_normal((N, r))
        muk, muv = g.standard_normal(r), g.standard_normal(r)
        ck, cv = oracle.encode(xk, muk, Wk), oracle.encode(xv, muv, Wv)
        q = g.standard_normal(d)
        for l in range(T):
            sl = slice(l * d, (l + 1) * d)
            ref = np.array(_py_attention(list(q), xk[:, sl].tolist(), xv[:, sl].tolist(), 0.5))
            try:
                got = decode_fn(q, ck, cv, Wk[sl, :], Wv[sl, :], muk[sl], muv[sl], 0.5)
            except ValueError:
                return False
            if not np.max(np.abs(got - ref)) < 1e-9:
                return False
    return True


def _mutant_no_mu_v(q, ck, cv, Uk, Uv, muk, muv, scale):
    return oracle.decode_attn(q, ck, cv, Uk, Uv, muk, None, scale)


def _mutant_no_scale(q, ck, cv, Uk, Uv, muk, muv, scale):
    return oracle.decode_attn(q, ck, cv, Uk, Uv, muk, muv, 1.0)


def _mutant_transposed_up(q, ck, cv, Uk, Uv, muk, muv, scale):
    # Eq. 3 with W_up where W_up^T belongs (only type-checks when W_up is square)
    K = np.asarray(ck) @ np.asarray(Uk) + muk
    V = oracle.reconstruct(cv, Uv, muv)
    return oracle.attention(q, K, V, scale)


def _mutant_swapped_up(q, ck, cv, Uk, Uv, muk, muv, scale):
    return oracle.decode_attn_absorbed(q, ck, cv, Uv, Uk, muk, muv, scale)


def _mutant_sign(q, ck, cv, Uk, Uv, muk, muv, scale):
    return oracle.decode_attn(q, ck, cv, Uk, Uv, muk, muv, -scale)


def _mutant_unnormalised(q, ck, cv, Uk, Uv, muk, muv, scale):
    K = oracle.reconstruct(ck, Uk, muk)
    V = oracle.reconstruct(cv, Uv, muv)
    s = scale * (K @ q)
    return np.exp(s - s.max()) @ V


def _mutant_wrong_loop_mu(q, ck, cv, Uk, Uv, muk, muv, scale):
    return oracle.decode_attn(q, ck, cv, Uk, Uv, muk, np.roll(muv, 1), scale)


def _mutant_absorbed_drops_mu_v(q, ck, cv, Uk, Uv, muk, muv, scale):
    return oracle.decode_attn_absorbed(q, ck, cv, Uk, Uv, muk, None, scale)


def test_pins_accept_the_oracle():
    assert _decode_pins_pass(oracle.decode_attn)
    assert _decode_pins_pass(oracle.decode_attn_absorbed)


@pytest.mark.parametrize("mutant", [_mutant_no_mu_v, _mutant_no_scale, _mutant_transposed_up,
                                    _mutant_swapped_up, _mutant_sign, _mutant_unnormalised,
                                    _mutant_wrong_loop_mu, _mutant_absorbed_drops_mu_v])
def test_pins_reject_planted_mistakes(mutant):
    assert not _decode_pins_pass(mutant)


# ---------------------------------------------------------------------------
# The batched prefill wrapper, every row against pure-Python brute force at an
# offset p0 > 0; slips in the causal length must fail.
# ---------------------------------------------------------------------------

def _py_prefill_row(q, ck, cv, Uk, Uv, muk, muv, n, scale):
    d, rk, rv = len(q), ck.shape[1], cv.shape[1]
    K = [[sum(ck[t, j] * Uk[i, j] for j in range(rk)) + muk[i] for i in range(d)] for t in range(n)]
    V = [[sum(cv[t, j] * Uv[i, j] for j in range(rv)) + muv[i] for i in range(d)] for t in range(n)]
    return np.array(_py_attention(list(q), K, V, scale))


def _prefill_batched_pin_passes(fn):
    g = _rng(41)
    B, H, d, rk, rv, p0, M = 2, 2, 4, 3, 5, 3, 5
    Q = g.standard_normal((B, H, M, d))
    ck, cv = g.standard_normal((B, H, p0 + M, rk)), g.standard_normal((B, H, p0 + M, rv))
    Uk, Uv = g.standard_normal((H, d, rk)), g.standard_normal((H, d, rv))
    muk, muv = g.standard_normal((H, d)), g.standard_normal((H, d))
    out = fn(Q, ck, cv, Uk, Uv, muk, muv, 0.6, p0)
    for b in range(B):
        for h in range(H):
            for m in range(M):
                ref = _py_prefill_row(Q[b, h, m], ck[b, h], cv[b, h], Uk[h], Uv[h], muk[h], muv[h],
                                      p0 + m + 1, 0.6)
                if not np.max(np.abs(out[b, h, m] - ref)) < 1e-12:
                    return False
    return True


def _prefill_batched_mutant(n_of):
    def fn(Q, ck, cv, Uk, Uv, muk, muv, scale, p0):
        B, H, M, d = Q.shape
        out = np.empty(Q.shape)
        for b in range(B):
            for h in range(H):
                for m in range(M):
                    n = n_of(p0, m)
                    out[b, h, m] = oracle.decode_attn(Q[b, h, m], ck[b, h, :n], cv[b, h, :n], Uk[h], Uv[h],
                                                      muk[h], muv[h], scale)
        return out
    return fn


def test_prefill_batched_rows_match_bruteforce():
    assert _prefill_batched_pin_passes(
        lambda Q, ck, cv, Uk, Uv, muk, muv, s, p0: oracle.prefill_attn_batched(Q, ck, cv, Uk, Uv, muk, muv, s,
                                                                               p0=p0))


@pytest.mark.parametrize("n_of", [lambda p0, m: p0 + 1, lambda p0, m: m + 1, lambda p0, m: p0 + m,
                                  lambda p0, m: p0 + m + 2])
def test_prefill_batched_pin_rejects_slips(n_of):
    assert _prefill_batched_pin_passes(_prefill_batched_mutant(lambda p0, m: p0 + m + 1))
    assert not _prefill_batched_pin_passes(_prefill_batched_mutant(n_of))
