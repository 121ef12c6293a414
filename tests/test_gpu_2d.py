"""GPU parity of LLA-2D (Sec. 3 "The LLA-2D variant (loop x head)": one latent
per token and layer for all heads) against the float64 oracle, through the C
ABI: the 2D cache write and the decode of all heads over the shared latents."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_15456_amd import lla, workloads as W
from tests.helpers import assert_close, f64, log

pytestmark = pytest.mark.gpu

DEV = "cuda"
WL = W.Workload("two_d", 1, 16, 128, 4, 3, 0, ((288, 480),), torch.bfloat16)


def _paged_v(cv, n_max):
    """[B, N, r] token-major -> the paged [B, n_max/64, r, 64] value cache (NaN past N)."""
    B, N, r = cv.shape
    full = cv.new_full((B, n_max, r), float("nan"))
    full[:, :N] = cv
    return full.view(B, n_max // 64, 64, r).transpose(-1, -2).contiguous()


def _keys(ck, n_max):
    B, N, r = ck.shape
    full = ck.new_full((B, n_max, r), float("nan"))
    full[:, :N] = ck
    return full


@pytest.mark.parametrize("r_k,r_v", [(288, 480), (64, 96), (32, 16), (576, 960), (1024, 1024), (160, 272)])
@pytest.mark.parametrize("N", [1, 63, 700, 4096])
def test_decode_2d(r_k, r_v, N):
    B = 3
    n_max = ((N + 63) // 64) * 64 + 64
    log(f"decode 2d r=({r_k},{r_v}) N={N}")
    ck = W.latents_2d(WL, r_k, "k", 0, B=B, N=N, device=DEV)
    cv = W.latents_2d(WL, r_v, "v", 0, B=B, N=N, device=DEV)
    q = W.queries(WL, 0, 1, B=B, device=DEV)
    uk, uv = W.codec_loop_2d(WL, r_k, r_v, 0, 1, DEV)
    muv = W.normal((WL.H, WL.d), ("two_d", "mu_v"), 1.0, torch.bfloat16, DEV)
    out = lla.decode_attn_2d(q, _keys(ck, n_max), _paged_v(cv, n_max), uk, uv, n_ctx=N, mu_v=muv)
    torch.cuda.synchronize()
    ref = oracle.decode_attn_2d_batched(f64(q), f64(ck), f64(cv), f64(uk), f64(uv), None, f64(muv))
    assert_close(f64(out), ref, torch.bfloat16, "decode 2d")


def test_decode_2d_ctx_len_and_bad_lengths():
    B, N, r_k, r_v = 4, 1500, 288, 480
    n_max = 1536
    ck = W.latents_2d(WL, r_k, "k", 1, B=B, N=N, device=DEV)
    cv = W.latents_2d(WL, r_v, "v", 1, B=B, N=N, device=DEV)
    q = W.queries(WL, 1, 0, B=B, device=DEV)
    uk, uv = W.codec_loop_2d(WL, r_k, r_v, 1, 0, DEV)
    lens = torch.tensor([1500, 65, 0, 1501], dtype=torch.int32, device=DEV)
    out = lla.decode_attn_2d(q, _keys(ck, n_max), _paged_v(cv, n_max), uk, uv, n_ctx=N, ctx_len=lens,
                             out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    got = f64(out)
    for b, n in ((0, 1500), (1, 65)):
        ref = oracle.decode_attn_2d(f64(q)[b], f64(ck)[b, :n], f64(cv)[b, :n], f64(uk), f64(uv))
        assert_close(got[b], ref, torch.bfloat16, f"b={b} N={n}", out_bf16=True)
    assert np.all(np.isnan(got[2])) and np.all(np.isnan(got[3])), "bad lengths must give NaN"


@pytest.mark.parametrize("M,pos0", [(1, 0), (1, 4095), (37, 100), (300, 0)])
def test_encode_2d_then_decode(M, pos0):
    """The 2D cache write (x stacked loop-major then head-major, Eq. 2 over T*H*d)
    and a decode over what it wrote."""
    B, T, H, d, r_k, r_v = 2, 4, 16, 128, 288, 480
    n_max = ((pos0 + M + 63) // 64) * 64
    K = T * H * d
    xk = W.normal((B, M, K), ("two_d", "x_k", M), 1.0, torch.bfloat16, DEV)
    xv = W.normal((B, M, K), ("two_d", "x_v", M), 1.0, torch.bfloat16, DEV)
    wk = W.normal((r_k, K), ("two_d", "Wd_k", r_k), 1.0 / K, torch.bfloat16, DEV)
    wv = W.normal((r_v, K), ("two_d", "Wd_v", r_v), 1.0 / K, torch.bfloat16, DEV)
    muk = W.normal((K,), ("two_d", "mu_k"), 1.0, torch.bfloat16, DEV)
    ck, cv = lla.alloc_cache_2d(B, n_max, r_k, r_v, device=DEV)
    ck.fill_(7.0)
    cv.fill_(7.0)
    lla.encode_2d(xk, xv, wk, wv, ck, cv, T=T, H=H, pos0=pos0, mu_k=muk)
    torch.cuda.synchronize()
    refk = np.stack([oracle.encode(f64(xk)[b], f64(muk), f64(wk).T) for b in range(B)])
    refv = np.stack([oracle.encode(f64(xv)[b], None, f64(wv).T) for b in range(B)])
    gk = f64(ck)
    gv = f64(cv).transpose(0, 1, 3, 2).reshape(B, n_max, r_v)
    assert_close(gk[:, pos0:pos0 + M], refk, torch.bfloat16, "2d keys")
    assert_close(gv[:, pos0:pos0 + M], refv, torch.bfloat16, "2d values")
    assert np.all(gk[:, :pos0] == 7.0) and np.all(gk[:, pos0 + M:] == 7.0)
    if pos0 == 0:
        q = W.queries(WL, 0, 2, B=B, device=DEV)
        uk, uv = W.codec_loop_2d(WL, r_k, r_v, 0, 2, DEV)
        out = lla.decode_attn_2d(q, ck, cv, uk, uv, n_ctx=M)
        torch.cuda.synchronize()
        ref = oracle.decode_attn_2d_batched(f64(q), gk[:, :M], gv[:, :M], f64(uk), f64(uv))
        assert_close(f64(out), ref, torch.bfloat16, "encode -> decode")


@pytest.mark.parametrize("B,M,pos0,r_k,r_v", [(2, 520, 64, 288, 480), (3, 256, 0, 96, 160), (1, 1000, 24, 576, 400)])
def test_encode_2d_prompt_write_with_means(B, M, pos0, r_k, r_v):
    """A prompt-sized 2D write (the tiled GEMM over the loop x head stack): token
    blocks straddle sequences, row blocks are partial at r = 400, 576, both means."""
    T, H, d = 4, 16, 128
    n_max = ((pos0 + M + 63) // 64) * 64 + 64
    K = T * H * d
    log(f"encode 2d prompt write B={B} M={M} pos0={pos0} r=({r_k},{r_v})")
    xk = W.normal((B, M, K), ("two_d", "px_k", M), 1.0, torch.bfloat16, DEV)
    xv = W.normal((B, M, K), ("two_d", "px_v", M), 1.0, torch.bfloat16, DEV)
    # variance 1/(16 K): latents ~ N(0, 1/8), so a one-ulp bf16 rounding flip stays below 2e-2
    wk = W.normal((r_k, K), ("two_d", "pWd_k", r_k), 1.0 / (16 * K), torch.bfloat16, DEV)
    wv = W.normal((r_v, K), ("two_d", "pWd_v", r_v), 1.0 / (16 * K), torch.bfloat16, DEV)
    muk = W.normal((K,), ("two_d", "pmu_k"), 1.0, torch.bfloat16, DEV)
    muv = W.normal((K,), ("two_d", "pmu_v"), 1.0, torch.bfloat16, DEV)
    ck, cv = lla.alloc_cache_2d(B, n_max, r_k, r_v, device=DEV)
    ck.fill_(7.0)
    cv.fill_(7.0)
    lla.encode_2d(xk, xv, wk, wv, ck, cv, T=T, H=H, pos0=pos0, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    refk = np.stack([oracle.encode(f64(xk)[b], f64(muk), f64(wk).T) for b in range(B)])
    refv = np.stack([oracle.encode(f64(xv)[b], f64(muv), f64(wv).T) for b in range(B)])
    gk = f64(ck)
    gv = f64(cv).transpose(0, 1, 3, 2).reshape(B, n_max, r_v)
    assert_close(gk[:, pos0:pos0 + M], refk, torch.bfloat16, "2d keys", out_bf16=True)
    assert_close(gv[:, pos0:pos0 + M], refv, torch.bfloat16, "2d values", out_bf16=True)
    assert np.all(gk[:, :pos0] == 7.0) and np.all(gk[:, pos0 + M:] == 7.0)
    assert np.all(gv[:, :pos0] == 7.0) and np.all(gv[:, pos0 + M:] == 7.0)


@pytest.mark.parametrize("B,M,T,d", [(32, 1, 4, 128), (5, 3, 4, 128), (33, 1, 4, 128), (64, 1, 2, 64),
                                     (2, 1, 4, 256)])
def test_encode_2d_split_write(B, M, T, d):
    """A decode step's write (few tokens, a long loop x head stack): the contraction
    is split over the stack and the fp32 partials are added by a second launch.
    Two calls in a row on one workspace."""
    H, r_k, r_v = 16, 288, 480
    K = T * H * d
    ws = lla.new_encode_2d_workspace(B, M, H, T, d, r_k, r_v, device=DEV)
    assert ws is not None
    n_max = 128
    # variance 1/(16 K): latents ~ N(0, 1/8), so a one-ulp bf16 rounding flip stays below 2e-2
    wk = W.normal((r_k, K), ("two_d", "Wd_k", K), 1.0 / (16 * K), torch.bfloat16, DEV)
    wv = W.normal((r_v, K), ("two_d", "Wd_v", K), 1.0 / (16 * K), torch.bfloat16, DEV)
    mu = W.normal((K,), ("two_d", "mu", K), 1.0, torch.bfloat16, DEV)
    ck, cv = lla.alloc_cache_2d(B, n_max, r_k, r_v, device=DEV)
    ck.fill_(7.0)
    cv.fill_(7.0)
    for call, pos0 in enumerate((5, 70)):
        log(f"encode 2d split B={B} M={M} K={K} call {call}")
        xk = W.normal((B, M, K), ("two_d", "sx_k", call), 1.0, torch.bfloat16, DEV)
        xv = W.normal((B, M, K), ("two_d", "sx_v", call), 1.0, torch.bfloat16, DEV)
        lla.encode_2d(xk, xv, wk, wv, ck, cv, T=T, H=H, pos0=pos0, mu_k=mu, mu_v=mu, workspace=ws)
        torch.cuda.synchronize()
        refk = np.stack([oracle.encode(f64(xk)[b], f64(mu), f64(wk).T) for b in range(B)])
        refv = np.stack([oracle.encode(f64(xv)[b], f64(mu), f64(wv).T) for b in range(B)])
        gk = f64(ck)
        gv = f64(cv).transpose(0, 1, 3, 2).reshape(B, n_max, r_v)
        assert_close(gk[:, pos0:pos0 + M], refk, torch.bfloat16, f"split keys call {call}", out_bf16=True)
        assert_close(gv[:, pos0:pos0 + M], refv, torch.bfloat16, f"split values call {call}", out_bf16=True)
    written = np.zeros(n_max, bool)
    written[5:5 + M] = written[70:70 + M] = True
    assert np.all(f64(ck)[:, ~written] == 7.0), "slots outside the writes changed"


def test_graph_replay_matches_eager():
    """The decode and the split write captured in a HIP graph and replayed three
    times, with eager work in between, give the eager results bit for bit."""
    B, T, H, d, r_k, r_v, N = 4, 4, 16, 128, 288, 480, 700
    n_max = 768
    K = T * H * d
    ck = W.latents_2d(WL, r_k, "k", 2, B=B, N=N, device=DEV)
    cv = W.latents_2d(WL, r_v, "v", 2, B=B, N=N, device=DEV)
    kc, vc = _keys(ck, n_max), _paged_v(cv, n_max)
    q = W.queries(WL, 2, 3, B=B, device=DEV)
    uk, uv = W.codec_loop_2d(WL, r_k, r_v, 2, 3, DEV)
    ws = torch.empty(lla.decode_2d_workspace_bytes(B, H, r_k, r_v, N), dtype=torch.uint8, device=DEV)
    xk = W.normal((B, 1, K), ("two_d", "gx_k"), 1.0, torch.bfloat16, DEV)
    xv = W.normal((B, 1, K), ("two_d", "gx_v"), 1.0, torch.bfloat16, DEV)
    wk = W.normal((r_k, K), ("two_d", "gWd_k"), 1.0 / (16 * K), torch.bfloat16, DEV)
    wv = W.normal((r_v, K), ("two_d", "gWd_v"), 1.0 / (16 * K), torch.bfloat16, DEV)
    ews = lla.new_encode_2d_workspace(B, 1, H, T, d, r_k, r_v, device=DEV)
    eager = lla.decode_attn_2d(q, kc, vc, uk, uv, n_ctx=N, workspace=ws)
    ek, ev = lla.alloc_cache_2d(B, 128, r_k, r_v, device=DEV)
    ek.zero_()
    ev.zero_()
    lla.encode_2d(xk, xv, wk, wv, ek, ev, T=T, H=H, pos0=70, workspace=ews)
    torch.cuda.synchronize()
    out = torch.empty_like(eager)
    gk, gv = torch.zeros_like(ek), torch.zeros_like(ev)
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=cap):
        lla.decode_attn_2d(q, kc, vc, uk, uv, n_ctx=N, out=out, workspace=ws)
        lla.encode_2d(xk, xv, wk, wv, gk, gv, T=T, H=H, pos0=70, workspace=ews)
    for rep in range(3):
        log(f"graph replay {rep}")
        out.fill_(float("nan"))
        gk.zero_()
        gv.zero_()
        ws.fill_(0xff)  # the workspace's contents must not matter
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"decode replay {rep}"
        assert torch.equal(gk, ek) and torch.equal(gv, ev), f"write replay {rep}"
