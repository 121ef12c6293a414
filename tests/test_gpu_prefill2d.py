"""GPU parity of the LLA-2D causal prefill (Sec. 3 "The LLA-2D variant (loop x
head)"; App. J "Per-head LLA versus LLA-2D at inference") against the float64
oracle, through the C ABI: every head's K and V rebuilt from the shared
latents, then causal attention of the M new queries at positions p0 .. p0+M-1.
Cache slots past p0 + M hold NaN, so a read past the prompt would show."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_15456_amd import lla, workloads as W
from tests.helpers import assert_close, f64, log

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _wl(H):
    return W.Workload("prefill_2d_test", 1, H, 128, 4, 2, 0, ((288, 480),), torch.bfloat16)


def _caches(ck, cv, n_max):
    """Token-major [B, N, r] latents -> the 2D caches (keys token-major, values
    paged feature-major), NaN past N."""
    B, N, rk = ck.shape
    rv = cv.shape[2]
    k = ck.new_full((B, n_max, rk), float("nan"))
    k[:, :N] = ck
    v = cv.new_full((B, n_max, rv), float("nan"))
    v[:, :N] = cv
    return k, v.view(B, n_max // 64, 64, rv).transpose(-1, -2).contiguous()


def _run(B, H, M, p0, r_k, r_v, *, seed=0, mu=False, out_dtype=torch.float32, scale=None, n_max=None,
         workspace=None):
    wl = _wl(H)
    n = p0 + M
    if n_max is None:
        n_max = ((n + 63) // 64) * 64 + 64
    ck = W.latents_2d(wl, r_k, "k", seed, B=B, N=n, device=DEV)
    cv = W.latents_2d(wl, r_v, "v", seed, B=B, N=n, device=DEV)
    q = W.queries(wl, seed, 1, B=B, M=M, device=DEV)
    uk, uv = W.codec_loop_2d(wl, r_k, r_v, seed, 1, DEV)
    # means ~ N(0, 1/4): outputs stay below 4, where one bf16 ulp (2^-6) of an
    # output rounded the other way stays inside the 2e-2 bar
    muk = W.normal((H, 128), ("prefill_2d_test", "mu_k", seed), 0.25, torch.bfloat16, DEV) if mu else None
    muv = W.normal((H, 128), ("prefill_2d_test", "mu_v", seed), 0.25, torch.bfloat16, DEV) if mu else None
    kc, vc = _caches(ck, cv, n_max)
    out = lla.prefill_attn_2d(q, kc, vc, uk, uv, p0=p0, mu_k=muk, mu_v=muv, scale=scale, out_dtype=out_dtype,
                              workspace=workspace)
    torch.cuda.synchronize()
    host = dict(q=f64(q), ck=f64(ck), cv=f64(cv), uk=f64(uk), uv=f64(uv),
                muk=None if muk is None else f64(muk), muv=None if muv is None else f64(muv))
    return f64(out), host


@pytest.mark.parametrize("r_k,r_v", [(288, 480), (32, 16), (64, 96), (160, 272), (512, 512), (16, 496)])
@pytest.mark.parametrize("M,p0", [(1, 0), (37, 0), (130, 5), (300, 64), (257, 200)])
def test_prefill_2d(r_k, r_v, M, p0):
    B, H = 2, 3
    log(f"prefill 2d r=({r_k},{r_v}) M={M} p0={p0}")
    got, h = _run(B, H, M, p0, r_k, r_v)
    ref = oracle.prefill_attn_2d_batched(h["q"], h["ck"], h["cv"], h["uk"], h["uv"], p0=p0)
    assert_close(got, ref, torch.bfloat16, f"prefill 2d r=({r_k},{r_v}) M={M} p0={p0}")


def test_prefill_2d_sixteen_heads_means_bf16_out():
    B, H, M, p0 = 2, 16, 200, 40
    log("prefill 2d H=16 with means, bf16 out")
    got, h = _run(B, H, M, p0, 288, 480, seed=1, mu=True, out_dtype=torch.bfloat16)
    ref = oracle.prefill_attn_2d_batched(h["q"], h["ck"], h["cv"], h["uk"], h["uv"], h["muk"], h["muv"], p0=p0)
    assert_close(got, ref, torch.bfloat16, "H=16 means", out_bf16=True)


def test_prefill_2d_sharp_scores():
    """A larger softmax scale makes rows peaked: the running max moves often and
    the weights span many binades."""
    B, H, M, p0 = 1, 2, 190, 3
    log("prefill 2d sharp scores")
    got, h = _run(B, H, M, p0, 288, 480, seed=2, scale=0.35)
    ref = oracle.prefill_attn_2d_batched(h["q"], h["ck"], h["cv"], h["uk"], h["uv"], scale=0.35, p0=p0)
    assert_close(got, ref, torch.bfloat16, "sharp")


def test_prefill_2d_full_cache_and_shared_workspace():
    """p0 + M = n_max exactly; then a second, smaller call on the same workspace."""
    B, H = 2, 2
    ws = torch.empty(lla.prefill_2d_workspace_bytes(B, H, 128, 512), dtype=torch.uint8, device=DEV)
    log("prefill 2d full cache")
    got, h = _run(B, H, 320, 192, 96, 160, seed=3, n_max=512, workspace=ws)
    ref = oracle.prefill_attn_2d_batched(h["q"], h["ck"], h["cv"], h["uk"], h["uv"], p0=192)
    assert_close(got, ref, torch.bfloat16, "full cache")
    log("prefill 2d second call, smaller")
    got, h = _run(B, H, 70, 0, 96, 160, seed=4, workspace=ws)
    ref = oracle.prefill_attn_2d_batched(h["q"], h["ck"], h["cv"], h["uk"], h["uv"], p0=0)
    assert_close(got, ref, torch.bfloat16, "second call")


@pytest.mark.parametrize("B,H,M,p0,n_max", [(1, 1, 100, 27, 128), (1, 2, 1, 255, 256), (3, 1, 64, 0, 64),
                                              (1, 5, 129, 0, 192)])
def test_prefill_2d_edges(B, H, M, p0, n_max):
    """One head or one sequence, a prompt that ends mid-page or at the cache's
    last slot, a one-token prompt at the end of a long cached prefix, exactly
    one page, one query past a 128-query block."""
    log(f"prefill 2d edges B={B} H={H} M={M} p0={p0} n_max={n_max}")
    got, h = _run(B, H, M, p0, 288, 480, seed=5, n_max=n_max)
    ref = oracle.prefill_attn_2d_batched(h["q"], h["ck"], h["cv"], h["uk"], h["uv"], p0=p0)
    assert_close(got, ref, torch.bfloat16, f"edges B={B} H={H} M={M} p0={p0}")


def test_prefill_2d_rejects_small_workspace():
    B, H, M = 1, 2, 70
    wl = _wl(H)
    ck = W.latents_2d(wl, 96, "k", 6, B=B, N=M, device=DEV)
    cv = W.latents_2d(wl, 160, "v", 6, B=B, N=M, device=DEV)
    kc, vc = _caches(ck, cv, 128)
    q = W.queries(wl, 6, 1, B=B, M=M, device=DEV)
    uk, uv = W.codec_loop_2d(wl, 96, 160, 6, 1, DEV)
    need = lla.prefill_2d_workspace_bytes(B, H, 128, M)
    ws = torch.empty(need - 16, dtype=torch.uint8, device=DEV)
    with pytest.raises(lla.LLAError):
        lla.prefill_attn_2d(q, kc, vc, uk, uv, p0=0, workspace=ws)


@pytest.mark.slow
def test_prefill_2d_full_size_sampled_rows():
    """The benchmark's shape (4 sequences x 8192 new tokens, 16 heads, (288, 480)):
    sampled query rows of sampled sequences against the oracle's 2D decode of the
    same row's context (each prefill row is that decode)."""
    B, H, M, r_k, r_v = 4, 16, 8192, 288, 480
    wl = W.Workload("prefill_2d", 1, H, 128, 4, B, M, ((r_k, r_v),), torch.bfloat16)
    log("prefill 2d full size")
    ck = W.latents_2d(wl, r_k, "k", 0, device=DEV)
    cv = W.latents_2d(wl, r_v, "v", 0, device=DEV)
    q = W.queries(wl, 0, 3, M=M, device=DEV)
    uk, uv = W.codec_loop_2d(wl, r_k, r_v, 0, 3, DEV)
    kc, vc = _caches(ck, cv, M)
    out = lla.prefill_attn_2d(q, kc, vc, uk, uv, p0=0)
    torch.cuda.synchronize()
    got = out[:, :, [0, 1, 63, 64, 127, 128, 1000, 4095, 8191]].cpu().double().numpy()
    hq, hk, hv, huk, huv = f64(q), f64(ck), f64(cv), f64(uk), f64(uv)
    for b in (0, 3):
        for i, m in enumerate((0, 1, 63, 64, 127, 128, 1000, 4095, 8191)):
            ref = oracle.decode_attn_2d(hq[b, :, m], hk[b, :m + 1], hv[b, :m + 1], huk, huv)
            assert_close(got[b, :, i], ref, torch.bfloat16, f"b={b} row {m}")


def test_prefill_2d_large_logits():
    """scale 1.0: base-2 logits of tens, the running maximum (held in fp16)
    raised on many pages and shifted inside the score product."""
    B, H, M, p0 = 1, 2, 260, 30
    log("prefill 2d large logits")
    got, h = _run(B, H, M, p0, 96, 160, seed=7, scale=1.0)
    ref = oracle.prefill_attn_2d_batched(h["q"], h["ck"], h["cv"], h["uk"], h["uv"], scale=1.0, p0=p0)
    assert_close(got, ref, torch.bfloat16, "large logits")
