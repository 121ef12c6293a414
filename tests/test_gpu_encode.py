"""GPU parity of lla_encode (Eq. 2 cache write) against the float64 oracle,
called through the C ABI, plus an encode -> decode chain."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_15456_amd import lla, workloads as W
from tests.helpers import assert_close, assert_units_close, f64, f64_dev, log, round_bf16

pytestmark = pytest.mark.gpu

DEV = "cuda"
SENTINEL = 7.0


def _inputs(wl, r_k, r_v, B, M, means, dtype):
    xk = W.stacked_kv(wl, "k", 0, B=B, M=M, device=DEV, dtype=dtype)
    xv = W.stacked_kv(wl, "v", 0, B=B, M=M, device=DEV, dtype=dtype)
    wk = W.down_projection(wl, r_k, "k", 0, DEV, dtype)
    wv = W.down_projection(wl, r_v, "v", 0, DEV, dtype)
    muk = W.stacked_mean(wl, "k", 0, DEV, dtype) if means else None
    muv = W.stacked_mean(wl, "v", 0, DEV, dtype) if means else None
    return xk, xv, wk, wv, muk, muv


def _run(wl, r_k, r_v, B, M, pos0, n_max, means, dtype):
    xk, xv, wk, wv, muk, muv = _inputs(wl, r_k, r_v, B, M, means, dtype)
    ck = torch.full((B, wl.H, n_max // 64, r_k, 64), SENTINEL, dtype=dtype, device=DEV)
    cv = torch.full((B, wl.H, n_max // 64, r_v, 64), SENTINEL, dtype=dtype, device=DEV)
    lla.encode(xk, xv, wk, wv, ck, cv, T=wl.T, pos0=pos0, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    return (xk, xv, wk, wv, muk, muv), ck, cv


def _check(wl, inputs, ck, cv, pos0, M, dtype, what):
    xk, xv, wk, wv, muk, muv = inputs
    for x, w, mu, c, name in ((xk, wk, muk, ck, "K"), (xv, wv, muv, cv, "V")):
        ref = oracle.encode_batched(f64(x), None if mu is None else f64(mu), f64(w))
        got = f64(lla.from_paged(c))
        assert_close(got[:, :, pos0:pos0 + M], ref, dtype, f"{what} {name}")
        untouched = np.concatenate([got[:, :, :pos0].ravel(), got[:, :, pos0 + M:].ravel()])
        assert np.all(untouched == SENTINEL), f"{what} {name}: slots outside [pos0, pos0+M) changed"


def test_tiny_fp32_encode():
    wl = W.WORKLOADS["tiny_fp32"]
    r_k, r_v = wl.ranks[0]
    for means in (False, True):
        log(f"tiny_fp32 encode means={means}")
        inputs, ck, cv = _run(wl, r_k, r_v, wl.B, wl.N, 0, wl.N, means, torch.float32)
        _check(wl, inputs, ck, cv, 0, wl.N, torch.float32, f"means={means}")


SMALL = W.Workload("enc_small", 1, 3, 128, 4, 3, 0, ((18, 30),), torch.bfloat16)


@pytest.mark.parametrize("r_k,r_v", [(18, 30), (36, 60), (96, 160), (192, 320), (7, 9), (1, 512)])
@pytest.mark.parametrize("M,pos0", [(1, 0), (1, 63), (11, 5), (21, 40), (100, 37), (64, 64), (129, 0)])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_encode_ragged(r_k, r_v, M, pos0, dtype):
    n_max = 256
    log(f"encode r=({r_k},{r_v}) M={M} pos0={pos0} {dtype}")
    inputs, ck, cv = _run(SMALL, r_k, r_v, 3, M, pos0, n_max, True, dtype)
    _check(SMALL, inputs, ck, cv, pos0, M, dtype, f"M={M} pos0={pos0}")


def test_other_head_widths():
    for d, T in ((64, 4), (96, 2), (256, 1)):
        wl = W.Workload(f"enc_d{d}", 1, 2, d, T, 2, 0, ((18, 30),), torch.bfloat16)
        log(f"encode d_head={d} T={T}")
        inputs, ck, cv = _run(wl, 18, 30, 2, 70, 5, 128, True, torch.bfloat16)
        _check(wl, inputs, ck, cv, 5, 70, torch.bfloat16, f"d={d}")


def test_decode_time_write_ouro14b_shape():
    """One new token per sequence at position 4096 (the decode step's cache write)."""
    wl = W.WORKLOADS["ouro14b_decode"]
    r_k, r_v = wl.ranks[0]
    inputs, ck, cv = _run(wl, r_k, r_v, wl.B, 1, 4096, 4160, False, torch.bfloat16)
    _check(wl, inputs, ck, cv, 4096, 1, torch.bfloat16, "M=1 at 4096")


@pytest.mark.slow
def test_full_prefill_write_encode():
    """Workload 5's cache write at full size: 4 x 8192 tokens, every latent
    checked (against the oracle's Eq. 2 rounded to bf16 like the cache)."""
    wl = W.WORKLOADS["prefill_write"]
    r_k, r_v = wl.ranks[0]
    log("prefill_write encode full size")
    xk, xv, wk, wv, _, _ = _inputs(wl, r_k, r_v, wl.B, wl.N, False, torch.bfloat16)
    ck = lla.alloc_cache(wl.B, wl.H, wl.N, r_k)
    cv = lla.alloc_cache(wl.B, wl.H, wl.N, r_v)
    lla.encode(xk, xv, wk, wv, ck, cv, T=wl.T, pos0=0)
    torch.cuda.synchronize()
    for x, w, c, name in ((xk, wk, ck, "K"), (xv, wv, cv, "V")):
        got = f64_dev(lla.from_paged(c))            # [B, H, M, r]
        w64 = f64(w)
        for b in range(wl.B):
            ref = oracle.encode_batched(f64_dev(x[b:b + 1]), None, w64)
            assert_units_close(got[b:b + 1], round_bf16(ref), f"{name} sequence {b}: every (h, token)")


def test_encode_then_decode_chain_fp32():
    """Workload 1: encode 512 tokens' loop-stacked K/V, then decode at every loop."""
    wl = W.WORKLOADS["tiny_fp32"]
    r_k, r_v = wl.ranks[0]
    inputs, ck, cv = _run(wl, r_k, r_v, wl.B, wl.N, 0, wl.N, True, torch.float32)
    xk, xv, wk, wv, muk, muv = inputs
    c_k = oracle.encode_batched(f64(xk), f64(muk), f64(wk))
    c_v = oracle.encode_batched(f64(xv), f64(muv), f64(wv))
    for loop in range(wl.T):
        q = W.queries(wl, 0, loop, device=DEV, dtype=torch.float32)
        uk, uv, _, _ = W.codec_loop(wl, r_k, r_v, 0, loop, DEV, torch.float32)
        sl = slice(loop * wl.d, (loop + 1) * wl.d)
        mk, mv = muk[:, sl].contiguous(), muv[:, sl].contiguous()
        out = lla.decode_attn(q, ck, cv, uk, uv, n_ctx=wl.N, mu_k=mk, mu_v=mv,
                              workspace=lla.new_workspace(wl.B, wl.H, r_v, wl.N))
        torch.cuda.synchronize()
        ref = oracle.decode_attn_batched(f64(q), c_k, c_v, f64(uk), f64(uv), f64(mk), f64(mv))
        assert_close(f64(out), ref, torch.float32, f"chain loop {loop}")


@pytest.mark.parametrize("r_k,r_v,T,d,B,M,pos0", [
    (18, 30, 4, 128, 3, 2900, 7),     # K = 512, 16-row tiles x 2, ragged last block
    (33, 64, 4, 128, 2, 4100, 0),     # four 16-row tiles per wave
    (5, 17, 2, 128, 1, 8200, 60),     # K = 256
])
def test_encode_many_tokens(r_k, r_v, T, d, B, M, pos0):
    """Prefill-sized writes (>= 8192 tokens): the resident-weight streaming path."""
    wl = W.Workload(f"enc_many_{T}_{d}", 1, 4, d, T, B, 0, ((r_k, r_v),), torch.bfloat16)
    n_max = ((pos0 + M + 63) // 64) * 64 + 64
    log(f"encode many tokens r=({r_k},{r_v}) K={T * d} B={B} M={M} pos0={pos0}")
    inputs, ck, cv = _run(wl, r_k, r_v, B, M, pos0, n_max, True, torch.bfloat16)
    _check(wl, inputs, ck, cv, pos0, M, torch.bfloat16, f"M={M}")


@pytest.mark.parametrize("r_k,r_v,T,d,B,M,pos0", [
    (96, 160, 4, 128, 2, 300, 5),      # the 4x tier, K = 512, ragged token block
    (288, 480, 4, 128, 1, 1000, 64),   # the 1.33x tier
    (120, 200, 4, 128, 3, 257, 0),     # row blocks of 96 with ragged ends
    (96, 160, 2, 128, 1, 513, 7),      # K = 256
    (200, 8, 4, 96, 2, 400, 0),        # K = 384, one rank above 64
])
@pytest.mark.parametrize("means", [False, True])
def test_encode_many_tokens_tier_ranks(r_k, r_v, T, d, B, M, pos0, means):
    """Prompt-sized writes at the paper's per-head rank tiers: the MFMA GEMM path."""
    wl = W.Workload(f"enc_tier_{T}_{d}", 1, 4, d, T, B, 0, ((r_k, r_v),), torch.bfloat16)
    n_max = ((pos0 + M + 63) // 64) * 64 + 64
    log(f"encode tier ranks r=({r_k},{r_v}) K={T * d} B={B} M={M} pos0={pos0} means={means}")
    inputs, ck, cv = _run(wl, r_k, r_v, B, M, pos0, n_max, means, torch.bfloat16)
    _check(wl, inputs, ck, cv, pos0, M, torch.bfloat16, f"M={M}")


@pytest.mark.parametrize("r_k,r_v,T,d,H,B,M,pos0,runs", [
    # 3 row blocks x 48 token blocks x 15 heads: 2 heads per workgroup, the last group 1
    (96, 160, 4, 128, 15, 2, 6000, 5, 2),
    # 8 row blocks x 24 token blocks x 16 heads: 3 heads per workgroup, the last group 1
    (288, 480, 4, 128, 16, 1, 4100, 64, 3),
    # K = 192: an odd chunk count per head, so one head per workgroup
    (96, 160, 3, 64, 16, 1, 12000, 0, 1),
])
@pytest.mark.parametrize("means", [False, True])
def test_encode_gemm_head_runs(r_k, r_v, T, d, H, B, M, pos0, runs, means):
    """Prompt-sized per-head writes where a GEMM workgroup walks a run of heads
    (as many as keep 1024 workgroups), including a last run shorter than the
    others; every latent is checked against the oracle."""
    ntb = (B * M + 255) // 256
    blocks = ((r_k + 95) // 96 + (r_v + 95) // 96) * ((ntb + 7) // 8 * 8)
    nkc = T * d // 64
    assert runs == (1 if nkc % 2 else max(1, min(H, H * blocks // 1024))), "case no longer takes the intended runs"
    wl = W.Workload(f"enc_runs_{T}_{d}_{H}", 1, H, d, T, B, 0, ((r_k, r_v),), torch.bfloat16)
    n_max = ((pos0 + M + 63) // 64) * 64 + 64
    log(f"encode head runs r=({r_k},{r_v}) K={T * d} H={H} B={B} M={M} pos0={pos0} runs={runs} means={means}")
    inputs, ck, cv = _run(wl, r_k, r_v, B, M, pos0, n_max, means, torch.bfloat16)
    _check(wl, inputs, ck, cv, pos0, M, torch.bfloat16, f"H={H} M={M}")


@pytest.mark.parametrize("r_k,r_v,means", [(96, 160, False), (200, 8, True)])
def test_encode_gemm_ring_slots(r_k, r_v, means):
    """Prompt-sized chunks at ranks above 64 (the GEMM write) streamed into a
    sink + window ring cache whose positions wrap: every kept position's slot
    holds the oracle's latent of that token (later tokens overwrite earlier ones)."""
    sink, window, chunks = 4, 512, [300, 500, 260]  # at most `window` tokens per call
    wl = W.Workload("enc_ring_gemm", 1, 4, 128, 4, 2, 0, ((r_k, r_v),), torch.bfloat16)
    B, H, K = wl.B, wl.H, wl.T * wl.d
    n_max = ((sink + window + 63) // 64) * 64
    wk = W.down_projection(wl, r_k, "k", 0, DEV, torch.bfloat16)
    wv = W.down_projection(wl, r_v, "v", 0, DEV, torch.bfloat16)
    muk = W.stacked_mean(wl, "k", 0, DEV, torch.bfloat16) if means else None
    muv = W.stacked_mean(wl, "v", 0, DEV, torch.bfloat16) if means else None
    ck = lla.alloc_cache(B, H, n_max, r_k, device=DEV)
    cv = lla.alloc_cache(B, H, n_max, r_v, device=DEV)
    refs_k, refs_v, pos = [], [], 0
    for i, M in enumerate(chunks):
        xk = W.normal((B, M, H, K), ("enc_ring_gemm", "x_k", i), 1.0, torch.bfloat16, DEV)
        xv = W.normal((B, M, H, K), ("enc_ring_gemm", "x_v", i), 1.0, torch.bfloat16, DEV)
        log(f"ring GEMM write r=({r_k},{r_v}) chunk {i}: M={M} pos0={pos} means={means}")
        lla.encode(xk, xv, wk, wv, ck, cv, T=wl.T, pos0=pos, mu_k=muk, mu_v=muv, evict=(sink, window))
        refs_k.append(oracle.encode_batched(f64(xk), None if muk is None else f64(muk), f64(wk)))
        refs_v.append(oracle.encode_batched(f64(xv), None if muv is None else f64(muv), f64(wv)))
        pos += M
    torch.cuda.synchronize()
    keep = oracle.kept_positions(pos, sink, window)
    slots = [oracle.ring_slot(p, sink, window) for p in keep]
    assert sorted(slots) == list(range(sink + window)), "kept positions must fill every slot once"
    for refs, c, name in ((refs_k, ck, "K"), (refs_v, cv, "V")):
        ref = np.concatenate(refs, axis=2)[:, :, keep]          # [B, H, kept, r]
        got = f64(lla.from_paged(c))[:, :, slots]
        assert_close(got, ref, torch.bfloat16, f"ring GEMM write {name}")
