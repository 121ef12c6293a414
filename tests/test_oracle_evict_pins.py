"""Pins of the oracle's eviction composition (App. J "Eviction and long-context
prefill"; tab:evict: a StreamingLLM-style sink + window budget on top of the
latent cache).  The budget is pinned by the paper's printed 36 MiB for the
1M-context Ouro-1.4B cache at 21.3x with a 1024-token budget, the kept set by
enumeration, the ring layout by its bijection property, and the attention by
reduction to the full decode and by brute force."""

import math

import numpy as np
import pytest

import oracle


def test_budget_caps_the_printed_cache_size():
    # App. J: LLA-21.3x with a 1024-token eviction budget caps the 1M-context
    # Ouro-1.4B cache (24 layers, 16 heads, T 4, d 128, bf16) at 36 MiB.
    kept = len(oracle.kept_positions(1 << 20, 4, 1020))
    assert kept == 1024
    b = oracle.cache_bytes(24, 16, 4, 128, 18, 30, kept, 2, latent=True)
    assert b == 36 * (1 << 20)


def test_kept_positions_enumeration():
    assert oracle.kept_positions(10, 4, 256) == list(range(10))
    assert oracle.kept_positions(260, 4, 256) == list(range(260))
    k = oracle.kept_positions(1000, 4, 256)
    assert k == [0, 1, 2, 3] + list(range(744, 1000))
    assert len(k) == 260 and len(set(k)) == 260


@pytest.mark.parametrize("sink,window", [(4, 256), (0, 64), (4, 1020), (7, 3)])
def test_ring_slots_are_a_bijection_of_the_kept_positions(sink, window):
    for N in (1, sink + window, sink + window + 1, 3 * window + sink + 5):
        keep = oracle.kept_positions(N, sink, window)
        slots = [oracle.ring_slot(p, sink, window) for p in keep]
        assert sorted(slots) == list(range(len(keep)))
    for p in range(sink, sink + 4 * window):
        assert oracle.ring_slot(p, sink, window) == oracle.ring_slot(p + window, sink, window)


def test_short_context_is_the_full_decode():
    g = np.random.default_rng(1)
    d, rk, rv, N = 8, 3, 5, 9
    q = g.standard_normal(d)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    Uk, Uv = g.standard_normal((d, rk)), g.standard_normal((d, rv))
    a = oracle.decode_attn_evict(q, ck, cv, Uk, Uv, scale=0.3, sink=4, window=8)
    b = oracle.decode_attn(q, ck, cv, Uk, Uv, scale=0.3)
    assert np.array_equal(a, b)


def test_evicted_decode_bruteforce_and_ring_storage():
    g = np.random.default_rng(2)
    d, rk, rv, N, S, W = 4, 3, 2, 23, 2, 5
    q = g.standard_normal(d)
    ck, cv = g.standard_normal((N, rk)), g.standard_normal((N, rv))
    Uk, Uv = g.standard_normal((d, rk)), g.standard_normal((d, rv))
    got = oracle.decode_attn_evict(q, ck, cv, Uk, Uv, scale=0.5, sink=S, window=W)
    # brute force in pure Python over positions {0, 1} and {18, ..., 22}
    keep = [0, 1, 18, 19, 20, 21, 22]
    s = [0.5 * sum(q[i] * sum(ck[n, j] * Uk[i, j] for j in range(rk)) for i in range(d)) for n in keep]
    m = max(s)
    e = [math.exp(x - m) for x in s]
    ref = [sum(e[t] * sum(cv[n, j] * Uv[i, j] for j in range(rv)) for t, n in enumerate(keep)) / sum(e)
           for i in range(d)]
    assert np.max(np.abs(got - np.array(ref))) < 1e-12
    # writing every position into its ring slot in order leaves exactly the kept tokens
    slots_k, slots_v = np.zeros((S + W, rk)), np.zeros((S + W, rv))
    for p in range(N):
        slots_k[oracle.ring_slot(p, S, W)] = ck[p]
        slots_v[oracle.ring_slot(p, S, W)] = cv[p]
    ring = oracle.decode_attn(q, slots_k, slots_v, Uk, Uv, scale=0.5)
    assert np.max(np.abs(ring - got)) < 1e-12


def test_evicted_rotary_decode_uses_true_positions():
    g = np.random.default_rng(3)
    d, dr, rk, rv, N, S, W = 4, 4, 3, 2, 30, 2, 6
    q, qr = g.standard_normal(d), g.standard_normal(dr)
    ck, cv, kr = g.standard_normal((N, rk)), g.standard_normal((N, rv)), g.standard_normal((N, dr))
    Uk, Uv = g.standard_normal((d, rk)), g.standard_normal((d, rv))
    got = oracle.decode_attn_rope_evict(q, qr, ck, cv, kr, Uk, Uv, scale=0.4, sink=S, window=W)
    keep = oracle.kept_positions(N, S, W)
    K = np.concatenate([ck[keep] @ Uk.T, np.stack([oracle.rope(kr[n], n) for n in keep])], axis=1)
    V = cv[keep] @ Uv.T
    ref = oracle.attention(np.concatenate([q, oracle.rope(qr, N - 1)]), K, V, 0.4)
    assert np.max(np.abs(got - ref)) < 1e-12
    # a slip that rotates the kept keys at their slot index instead of their position differs
    Kw = np.concatenate([ck[keep] @ Uk.T, np.stack([oracle.rope(kr[n], t) for t, n in enumerate(keep)])], axis=1)
    wrong = oracle.attention(np.concatenate([q, oracle.rope(qr, N - 1)]), Kw, V, 0.4)
    assert np.max(np.abs(wrong - ref)) > 1e-3
