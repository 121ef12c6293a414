"""GPU parity of lla_prefill_attn (causal prefill over the latent cache) against
the float64 oracle, through the C ABI."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_15456_amd import lla, workloads as W
from tests.helpers import assert_close, assert_units_close, f64, f64_dev, log

pytestmark = pytest.mark.gpu

DEV = "cuda"
SMALL = W.Workload("pf_small", 1, 3, 128, 4, 2, 0, ((18, 30),), torch.bfloat16)


def _paged(c, n_max, poison):
    """Paged cache of the latents c [B, H, N, r]; slots past N hold NaN when poisoned
    (they must not leak into any output), zeros otherwise."""
    B, H, N, r = c.shape
    full = c.new_full((B, H, n_max, r), float("nan") if poison else 0.0)
    full[:, :, :N] = c
    return full.view(B, H, n_max // 64, 64, r).transpose(-1, -2).contiguous()


def _case(wl, r_k, r_v, B, M, p0, dtype, means=True, poison=True, n_max=None, qmul=1.0, kramp=0.0):
    N = p0 + M
    n_max = n_max or ((N + 63) // 64) * 64 + 64
    ck = W.latents(wl, r_k, "k", 0, B=B, N=N, device=DEV, dtype=torch.float32)
    cv = W.latents(wl, r_v, "v", 0, B=B, N=N, device=DEV, dtype=torch.float32)
    if kramp:  # latents growing along the context: later keys score higher (forces rescales)
        ck = ck * (1.0 + kramp * torch.arange(N, device=DEV, dtype=torch.float32)[None, None, :, None] / N)
    ck, cv = ck.to(dtype), cv.to(dtype)
    q = W.queries(wl, 0, 2, B=B, M=M, device=DEV, dtype=torch.float32)
    q = (q * qmul).to(dtype)
    uk, uv, muk, muv = W.codec_loop(wl, r_k, r_v, 0, 2, DEV, dtype, means=means)
    pk, pv = _paged(ck, n_max, poison), _paged(cv, n_max, poison)
    return q, ck, cv, uk, uv, muk, muv, pk, pv


def _oracle(q, ck, cv, uk, uv, muk, muv, p0, rows=None, units=None, scale=None):
    return oracle.prefill_attn_batched(f64(q), f64(ck), f64(cv), f64(uk), f64(uv),
                                       None if muk is None else f64(muk),
                                       None if muv is None else f64(muv), scale, p0=p0,
                                       rows=rows, units=units)


@pytest.mark.parametrize("r_k,r_v", [(18, 30), (36, 60), (7, 9), (64, 95), (32, 31), (33, 64), (1, 1),
                                     (95, 95), (80, 40), (31, 95), (63, 20)])
@pytest.mark.parametrize("M,p0", [(1, 0), (33, 0), (128, 0), (200, 5), (77, 100), (130, 64)])
def test_bf16_prefill(r_k, r_v, M, p0):
    log(f"prefill bf16 r=({r_k},{r_v}) M={M} p0={p0}")
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(SMALL, r_k, r_v, 2, M, p0, torch.bfloat16)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=p0, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    assert_close(f64(out), _oracle(q, ck, cv, uk, uv, muk, muv, p0), torch.bfloat16, "prefill")


@pytest.mark.parametrize("M,p0", [(1, 0), (65, 3), (130, 64)])
def test_fp32_prefill(M, p0):
    log(f"prefill fp32 M={M} p0={p0}")
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(SMALL, 36, 60, 2, M, p0, torch.float32)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=p0, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    assert_close(f64(out), _oracle(q, ck, cv, uk, uv, muk, muv, p0), torch.float32, "prefill fp32")


def test_bf16_out_and_custom_scale():
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(SMALL, 18, 30, 2, 150, 20, torch.bfloat16, means=False)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=20, scale=0.2, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert out.dtype == torch.bfloat16
    assert_close(f64(out), _oracle(q, ck, cv, uk, uv, None, None, 20, scale=0.2), torch.bfloat16, "bf16 out",
                 out_bf16=True)


@pytest.mark.parametrize("qmul,kramp", [(4.0, 0.0), (1.0, 6.0), (3.0, 4.0)])
def test_peaked_and_rising_scores(qmul, kramp):
    """Peaked softmax rows and keys whose scores rise along the context: the
    running max is raised page after page (lazy rescale path)."""
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(SMALL, 18, 30, 2, 600, 0, torch.bfloat16, qmul=qmul,
                                                kramp=kramp)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=0, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    assert_close(f64(out), _oracle(q, ck, cv, uk, uv, muk, muv, 0), torch.bfloat16, f"q x{qmul} ramp {kramp}")


def test_prefill_rows_match_decode():
    """Row m of a prefill equals a decode over the first p0 + m + 1 tokens."""
    M, p0 = 96, 40
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(SMALL, 36, 60, 2, M, p0, torch.bfloat16, poison=False)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=p0, mu_k=muk, mu_v=muv)
    for m in (0, 31, 32, 95):
        n = p0 + m + 1
        dec = lla.decode_attn(q[:, :, m].contiguous(), pk, pv, uk, uv, n_ctx=n, mu_k=muk, mu_v=muv)
        torch.cuda.synchronize()
        assert_close(f64(out[:, :, m]), f64(dec), torch.bfloat16, f"row {m}")


@pytest.mark.slow
def test_full_prefill_write():
    """Workload 5 at full size: encode 4 x 8192 tokens into the (18, 30) cache,
    then causal prefill at every loop.  Every (b, h) unit is checked at the
    first and last row of every 256-query block (and a few more rows) against
    the absorbed oracle over the row's prefix (App. J; a prefill row is the
    decode of the context that ends at its position), and three units at ten
    rows against the plain definition."""
    wl = W.WORKLOADS["prefill_write"]
    r_k, r_v = wl.ranks[0]
    B, M, H = wl.B, wl.N, wl.H
    log("prefill_write full size: encode")
    xk = W.stacked_kv(wl, "k", 0, device=DEV)
    xv = W.stacked_kv(wl, "v", 0, device=DEV)
    wk = W.down_projection(wl, r_k, "k", 0, DEV)
    wv = W.down_projection(wl, r_v, "v", 0, DEV)
    ck = lla.alloc_cache(B, H, M, r_k)
    cv = lla.alloc_cache(B, H, M, r_v)
    lla.encode(xk, xv, wk, wv, ck, cv, T=wl.T, pos0=0)
    del xk, xv
    plain_units = [(0, 0), (1, 7), (3, 15)]
    plain_rows = [0, 1, 63, 64, 127, 128, 4095, 5000, 8190, 8191]
    rows = sorted(set(plain_rows) | {256 * qb + e for qb in range(M // 256) for e in (0, 255)})
    lat_k = f64_dev(lla.from_paged(ck))
    lat_v = f64_dev(lla.from_paged(cv))
    for loop in range(wl.T):
        log(f"prefill_write full size: loop {loop}")
        q = W.queries(wl, 0, loop, M=M, device=DEV)
        uk, uv, _, _ = W.codec_loop(wl, r_k, r_v, 0, loop, DEV)
        out = lla.prefill_attn(q, ck, cv, uk, uv, p0=0)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(out).all())
        o = f64_dev(out[:, :, rows])
        q64 = f64_dev(q[:, :, rows])
        uk64, uv64 = f64(uk), f64(uv)
        ref = np.empty_like(o)
        for b in range(B):
            for h in range(H):
                for i, m in enumerate(rows):
                    ref[b, h, i] = oracle.decode_attn_absorbed(q64[b, h, i], lat_k[b, h, :m + 1], lat_v[b, h, :m + 1],
                                                               uk64[h], uv64[h])
        assert_units_close(o, ref, f"loop {loop}: every (b, h) at {len(rows)} rows")
        for (b, h) in plain_units:
            idx = [rows.index(m) for m in plain_rows]
            plain = np.stack([oracle.decode_attn(q64[b, h, i], lat_k[b, h, :rows[i] + 1], lat_v[b, h, :rows[i] + 1],
                                                 uk64[h], uv64[h]) for i in idx])
            assert_close(o[b, h, idx], plain, torch.bfloat16, f"loop {loop} unit ({b},{h}) plain definition")


# ---------------------------------------------------------------------------
# bf16 at the paper's per-head rank tiers (tab:tier4, ranks above the absorbed
# kernel's 95): each head's K_l and V_l are rebuilt (Eq. 3) into the
# workspace, then attended.  Rows are checked against the absorbed oracle
# (App. J; pinned against the plain definition), and a sample against the
# plain definition (K and V rebuilt once, the teacher's attention per row).
# ---------------------------------------------------------------------------

def _rows_absorbed(q, ck, cv, uk, uv, muk, muv, p0, scale=None, rows=None):
    q64, k64, v64, uk64, uv64 = f64(q), f64(ck), f64(cv), f64(uk), f64(uv)
    mk = None if muk is None else f64(muk)
    mv = None if muv is None else f64(muv)
    B, H, M, _ = q64.shape
    rows = range(M) if rows is None else rows
    return np.stack([np.stack([np.stack([
        oracle.decode_attn_absorbed(q64[b, h, m], k64[b, h, :p0 + m + 1], v64[b, h, :p0 + m + 1], uk64[h], uv64[h],
                                    None if mk is None else mk[h], None if mv is None else mv[h], scale)
        for m in rows]) for h in range(H)]) for b in range(B)])


TIERS = [(96, 160), (120, 200), (144, 240), (192, 320), (240, 400), (288, 480)]


@pytest.mark.parametrize("r_k,r_v", TIERS + [(512, 512), (8, 504), (128, 96)])
@pytest.mark.parametrize("M,p0", [(1, 0), (37, 0), (130, 5), (300, 64), (257, 200)])
def test_bf16_prefill_tier_ranks(r_k, r_v, M, p0):
    log(f"prefill bf16 rebuild r=({r_k},{r_v}) M={M} p0={p0}")
    assert lla.prefill_workspace_bytes(torch.bfloat16, 2, SMALL.H, M, 128, r_k, r_v, p0) > 0
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(SMALL, r_k, r_v, 2, M, p0, torch.bfloat16)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=p0, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    assert_close(f64(out), _rows_absorbed(q, ck, cv, uk, uv, muk, muv, p0), torch.bfloat16, "prefill rebuild")


def test_bf16_prefill_tier_plain_definition_bf16_out_and_scale():
    r_k, r_v, M, p0 = 192, 320, 200, 33
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(SMALL, r_k, r_v, 2, M, p0, torch.bfloat16, means=False)
    ws = torch.empty(lla.prefill_workspace_bytes(torch.bfloat16, 2, SMALL.H, M, 128, r_k, r_v, p0),
                     dtype=torch.uint8, device=DEV)
    for scale, out_dtype in ((None, torch.float32), (0.2, torch.bfloat16)):
        out = lla.prefill_attn(q, pk, pv, uk, uv, p0=p0, scale=scale, out_dtype=out_dtype, workspace=ws)
        torch.cuda.synchronize()
        ref = np.stack([oracle.prefill_attn_2d(f64(q)[b, h:h + 1], f64(ck)[b, h], f64(cv)[b, h], f64(uk)[h:h + 1],
                                               f64(uv)[h:h + 1], scale=scale, p0=p0)[0]
                        for b in range(2) for h in range(SMALL.H)]).reshape(2, SMALL.H, M, 128)
        assert_close(f64(out), ref, torch.bfloat16, f"plain definition scale={scale}",
                     out_bf16=out_dtype == torch.bfloat16)


@pytest.mark.parametrize("qmul,kramp", [(4.0, 0.0), (1.0, 6.0)])
def test_bf16_prefill_tier_peaked_and_rising(qmul, kramp):
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(SMALL, 96, 160, 2, 600, 0, torch.bfloat16, qmul=qmul, kramp=kramp)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=0, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    assert_close(f64(out), _rows_absorbed(q, ck, cv, uk, uv, muk, muv, 0), torch.bfloat16,
                 f"q x{qmul} ramp {kramp}")


@pytest.mark.slow
@pytest.mark.parametrize("r_k,r_v", [(96, 160), (288, 480)])
def test_full_prefill_tier(r_k, r_v):
    """4 x 8192 new tokens, 16 heads, at the 4x and 1.33x tiers: every (b, h) at
    the first and last row of every 256-query block."""
    wl = W.WORKLOADS["prefill_write"]
    B, M, H = wl.B, wl.N, wl.H
    log(f"full-size rebuild prefill r=({r_k},{r_v})")
    ck = lla.to_paged(W.latents(wl, r_k, "k", 0, device=DEV), M)
    cv = lla.to_paged(W.latents(wl, r_v, "v", 0, device=DEV), M)
    q = W.queries(wl, 0, 1, M=M, device=DEV)
    uk, uv, _, _ = W.codec_loop(wl, r_k, r_v, 0, 1, DEV)
    out = lla.prefill_attn(q, ck, cv, uk, uv, p0=0)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all())
    rows = sorted({256 * qb + e for qb in range(M // 256) for e in (0, 255)})
    o = f64_dev(out[:, :, rows])
    q64, uk64, uv64 = f64_dev(q[:, :, rows]), f64(uk), f64(uv)
    ref = np.empty_like(o)
    for b in range(B):
        k64 = f64_dev(lla.from_paged(ck[b:b + 1]))[0]
        v64 = f64_dev(lla.from_paged(cv[b:b + 1]))[0]
        for h in range(H):
            for i, m in enumerate(rows):
                ref[b, h, i] = oracle.decode_attn_absorbed(q64[b, h, i], k64[h, :m + 1], v64[h, :m + 1], uk64[h], uv64[h])
    assert_units_close(o, ref, f"every (b, h) at {len(rows)} rows")


@pytest.mark.parametrize("d", [32, 64, 96])
def test_bf16_prefill_other_head_widths(d):
    wl = W.Workload(f"pf_d{d}", 1, 3, d, 4, 2, 0, ((18, 30),), torch.bfloat16)
    q, ck, cv, uk, uv, muk, muv, pk, pv = _case(wl, 18, 30, 2, 150, 7, torch.bfloat16)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=7, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    assert_close(f64(out), _oracle(q, ck, cv, uk, uv, muk, muv, 7), torch.bfloat16, f"d_head={d}")
