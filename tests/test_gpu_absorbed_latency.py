"""The two decodes that tab:absorbed_latency compares (App. J), at its shapes:
Ouro-1.4B geometry at the 4x tier (r_k, r_v) = (96, 160) with a 64-wide
decoupled rotary key (tab:decoupled_char), contexts 32k, 131k and 262k, one
sequence of 16 heads.  The absorbed decode with the rotary branch and the
full-RoPE reconstruct-then-attend decode each run through the C ABI in the
launch configuration the benchmark times (split-K workspace), and one sampled
(b, h) unit per context is checked against the float64 oracle."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_15456_amd import lla, workloads as W
from tests.helpers import assert_close, f64, f64_dev, log

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

DEV = "cuda"
WL = W.Workload("absorbed_latency", 1, 16, 128, 4, 1, 0, ((96, 160),), torch.bfloat16)
R_K, R_V, D_ROPE = 96, 160, 64


@pytest.mark.parametrize("N,unit", [(32768, 3), (131072, 9), (262144, 15)])
def test_absorbed_and_fullrope_at_paper_contexts(N, unit):
    B, H = 1, WL.H
    log(f"absorbed-latency geometry N={N}")
    ck = W.latents(WL, R_K, "k", 0, B=B, N=N, device=DEV)
    cv = W.latents(WL, R_V, "v", 0, B=B, N=N, device=DEV)
    kr = W.rotary_keys(WL, D_ROPE, 1, 0, B=B, N=N, device=DEV)
    q = W.queries(WL, 0, 2, B=B, device=DEV)
    qr = W.rotary_queries(WL, D_ROPE, 0, 2, B=B, device=DEV)
    uk, uv, _, _ = W.codec_loop(WL, R_K, R_V, 0, 2, DEV)
    pk, pv = lla.to_paged(ck, N), lla.to_paged(cv, N)
    rc = lla.alloc_cache(B, 1, N, D_ROPE, device=DEV)
    lla.rope_write(kr, rc, pos0=0)
    q_rot = lla.rope_rotate(qr, pos0=N - 1)            # the query is the newest token
    ws = lla.new_workspace(B, H, R_V, N)
    out_abs = lla.decode_attn(q, pk, pv, uk, uv, n_ctx=N, workspace=ws, q_rope=q_rot, r_cache=rc)
    out_full = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, workspace=ws)
    torch.cuda.synchronize()
    h = unit
    ck64, cv64 = f64_dev(ck[0, h]), f64_dev(cv[0, h])
    ref_abs = oracle.decode_attn_rope(f64(q[0, h]), f64(qr[0, h]), ck64, cv64, f64_dev(kr[0, :, 0]), f64(uk[h]),
                                      f64(uv[h]), q_pos=N - 1)
    ref_full = oracle.decode_attn_fullrope(f64(q[0, h]), ck64, cv64, f64(uk[h]), f64(uv[h]), q_pos=N - 1)
    assert_close(f64(out_abs[0, h]), ref_abs, torch.bfloat16, f"absorbed + rotary, unit (0,{h})")
    assert_close(f64(out_full[0, h]), ref_full, torch.bfloat16, f"full RoPE, unit (0,{h})")
    assert bool(torch.isfinite(out_abs).all()) and bool(torch.isfinite(out_full).all())
