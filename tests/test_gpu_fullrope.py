"""GPU parity of lla_decode_attn_fullrope (full-RoPE reconstruct-then-attend,
Sec. 3 "RoPE and reconstruction") against the float64 oracle's plain
definition: keys reconstructed with Eq. 3 and rotated at their positions, the
query rotated at its position, teacher attention.  Called through the C ABI.

The bf16 MFMA kernel reconstructs the keys exactly from bf16 operands in fp32
and rotates them in fp32, so besides the stated bf16 tolerance the tests also
hold it to relative L2 <= 1e-4 (fp32 rounding over a few thousand tokens),
which a wrong feature, frequency or position would break.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_15456_amd import lla, workloads as W
from tests.helpers import assert_close, errors, f64, log

pytestmark = pytest.mark.gpu

DEV = "cuda"
SMALL = W.Workload("small_fullrope", 1, 4, 128, 4, 3, 0, ((96, 160),), torch.bfloat16)


def _case(wl, r_k, r_v, B, N, n_max, layer, loop, means, dtype, d=None):
    ck = W.latents(wl, r_k, "k", layer, B=B, N=N, device=DEV, dtype=dtype)
    cv = W.latents(wl, r_v, "v", layer, B=B, N=N, device=DEV, dtype=dtype)
    if d is None or d == wl.d:
        q = W.queries(wl, layer, loop, B=B, device=DEV, dtype=dtype)
        uk, uv, muk, muv = W.codec_loop(wl, r_k, r_v, layer, loop, DEV, dtype, means=means)
    else:
        q = W.normal((B, wl.H, d), (wl.name, "q_d", d, layer, loop), 1.0, dtype, DEV)
        uk = W.normal((wl.H, d, r_k), (wl.name, "Uk_d", d, layer, loop), 1.0 / r_k, dtype, DEV)
        uv = W.normal((wl.H, d, r_v), (wl.name, "Uv_d", d, layer, loop), 1.0 / r_v, dtype, DEV)
        muk = W.normal((wl.H, d), (wl.name, "muk_d", d), 1.0, dtype, DEV) if means else None
        muv = W.normal((wl.H, d), (wl.name, "muv_d", d), 1.0, dtype, DEV) if means else None
    return ck, cv, q, uk, uv, muk, muv, lla.to_paged(ck, n_max), lla.to_paged(cv, n_max)


def _oracle(q, ck, cv, uk, uv, muk, muv, scale=None, ctx_len=None, q_pos=None, base=10000.0, units=None):
    return oracle.decode_attn_fullrope_batched(f64(q), f64(ck), f64(cv), f64(uk), f64(uv),
                                               None if muk is None else f64(muk),
                                               None if muv is None else f64(muv), scale, base,
                                               ctx_len=ctx_len, q_pos=q_pos, units=units)


def _tight(got, ref, what, bound=1e-4):
    _, rel = errors(np.asarray(got, dtype=np.float64), ref)
    assert rel <= bound, (what, rel)


# ---------------------------------------------------------------------------
# fp32 (plain kernel): the tiny workload's shape, every loop, 1e-5.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("means", [False, True])
def test_tiny_fp32_every_loop(means):
    wl = W.WORKLOADS["tiny_fp32"]
    r_k, r_v = wl.ranks[0]
    for loop in range(wl.T):
        log(f"fullrope tiny_fp32 loop={loop} means={means}")
        ck, cv, q, uk, uv, muk, muv, pk, pv = _case(wl, r_k, r_v, wl.B, wl.N, wl.N, 0, loop, means,
                                                    torch.float32)
        out = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=wl.N, mu_k=muk, mu_v=muv)
        torch.cuda.synchronize()
        assert_close(f64(out), _oracle(q, ck, cv, uk, uv, muk, muv), torch.float32, f"loop {loop}")


def test_fp32_positions_lengths_and_base():
    B, N = 3, 300
    ck, cv, q, uk, uv, muk, muv, pk, pv = _case(SMALL, 36, 60, B, N, 320, 0, 1, True, torch.float32)
    lens, qp = [300, 1, 131], [299, 5000, 7]
    ctx = torch.tensor(lens, dtype=torch.int32, device=DEV)
    qpos = torch.tensor(qp, dtype=torch.int32, device=DEV)
    for base in (10000.0, 500000.0):
        log(f"fullrope fp32 lengths base={base}")
        out = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, ctx_len=ctx, q_pos=qpos, mu_k=muk,
                                       mu_v=muv, base=base)
        torch.cuda.synchronize()
        assert_close(f64(out), _oracle(q, ck, cv, uk, uv, muk, muv, ctx_len=lens, q_pos=qp, base=base),
                     torch.float32, f"base {base}")


# ---------------------------------------------------------------------------
# bf16 MFMA kernel: ranks (incl. ones that are not multiples of 8 or 16),
# ragged contexts, with and without the split workspace.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("r_k,r_v", [(96, 160), (192, 320), (36, 60), (18, 30), (288, 480), (120, 200),
                                     (7, 9), (256, 512)])
@pytest.mark.parametrize("N", [1, 63, 65, 777])
def test_bf16_ragged(r_k, r_v, N):
    n_max = ((N + 63) // 64) * 64 + 64
    log(f"fullrope bf16 r=({r_k},{r_v}) N={N}")
    ck, cv, q, uk, uv, muk, muv, pk, pv = _case(SMALL, r_k, r_v, 3, N, n_max, 0, 1, True, torch.bfloat16)
    ref = _oracle(q, ck, cv, uk, uv, muk, muv)
    ws = lla.new_workspace(3, SMALL.H, r_v, N)
    for w in (None, ws):
        out = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, mu_k=muk, mu_v=muv, workspace=w)
        torch.cuda.synchronize()
        tag = f"ws={'yes' if w is not None else 'no'}"
        assert_close(f64(out), ref, torch.bfloat16, tag)
        _tight(f64(out), ref, tag)


def test_bf16_long_context_split_positions_bf16_out():
    B, N, n_max = 2, 5000, 5056
    ck, cv, q, uk, uv, muk, muv, pk, pv = _case(SMALL, 192, 320, B, N, n_max, 0, 2, False, torch.bfloat16)
    lens, qp = [5000, 2345], [4999, 100000]
    ctx = torch.tensor(lens, dtype=torch.int32, device=DEV)
    qpos = torch.tensor(qp, dtype=torch.int32, device=DEV)
    ref = _oracle(q, ck, cv, uk, uv, None, None, ctx_len=lens, q_pos=qp)
    ws = lla.new_workspace(B, SMALL.H, 320, N)
    for out_dtype in (torch.float32, torch.bfloat16):
        out = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, ctx_len=ctx, q_pos=qpos, workspace=ws,
                                       out_dtype=out_dtype)
        torch.cuda.synchronize()
        assert out.dtype == out_dtype
        assert_close(f64(out), ref, torch.bfloat16, f"out={out_dtype}", out_bf16=out_dtype == torch.bfloat16)
        if out_dtype == torch.float32:
            _tight(f64(out), ref, "fp32 out")


def test_bf16_peaked_scores():
    B, N = 2, 1024
    ck, cv, q, uk, uv, muk, muv, pk, pv = _case(SMALL, 96, 160, B, N, N, 0, 3, True, torch.bfloat16)
    q4 = (q.float() * 4).to(torch.bfloat16)
    out = lla.decode_attn_fullrope(q4, pk, pv, uk, uv, n_ctx=N, mu_k=muk, mu_v=muv,
                                   workspace=lla.new_workspace(B, SMALL.H, 160, N))
    torch.cuda.synchronize()
    ref = _oracle(q4, ck, cv, uk, uv, muk, muv)
    assert_close(f64(out), ref, torch.bfloat16, "peaked")
    _tight(f64(out), ref, "peaked")


def test_rotation_matters_and_mu_k_does_not_cancel():
    """The result differs from the absorbed NoPE decode and depends on mu_k."""
    B, N = 2, 400
    ck, cv, q, uk, uv, muk, muv, pk, pv = _case(SMALL, 96, 160, B, N, 448, 0, 0, True, torch.bfloat16)
    a = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, mu_k=muk, mu_v=muv)
    b = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, mu_k=None, mu_v=muv)
    c = lla.decode_attn(q, pk, pv, uk, uv, n_ctx=N, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    assert_close(f64(a), _oracle(q, ck, cv, uk, uv, muk, muv), torch.bfloat16, "with mu_k")
    assert_close(f64(b), _oracle(q, ck, cv, uk, uv, None, muv), torch.bfloat16, "without mu_k")
    assert float((a - b).abs().max()) > 1e-3
    assert float((a - c).abs().max()) > 1e-3


def test_out_of_range_lengths_give_nan():
    B, N = 3, 256
    ck, cv, q, uk, uv, muk, muv, pk, pv = _case(SMALL, 96, 160, B, N, 256, 0, 0, False, torch.bfloat16)
    ctx = torch.tensor([0, 100, 257], dtype=torch.int32, device=DEV)
    ws = lla.new_workspace(B, SMALL.H, 160, N)
    for w in (None, ws):
        out = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, ctx_len=ctx, workspace=w)
        torch.cuda.synchronize()
        o = f64(out)
        assert np.all(np.isnan(o[0])) and np.all(np.isnan(o[2]))
        assert_close(o[1:2], _oracle(q[1:2], ck[1:2], cv[1:2], uk, uv, None, None, ctx_len=[100]),
                     torch.bfloat16, "valid row")
    out = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, workspace=ws)  # counters back at zero
    torch.cuda.synchronize()
    assert_close(f64(out), _oracle(q, ck, cv, uk, uv, None, None), torch.bfloat16, "after NaN call")


def test_bf16_other_head_width_runs_the_plain_kernel():
    B, N = 2, 200
    ck, cv, q, uk, uv, muk, muv, pk, pv = _case(SMALL, 40, 24, B, N, 256, 0, 0, True, torch.bfloat16, d=64)
    out = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=N, mu_k=muk, mu_v=muv)
    torch.cuda.synchronize()
    assert_close(f64(out), _oracle(q, ck, cv, uk, uv, muk, muv), torch.bfloat16, "d=64")


# ---------------------------------------------------------------------------
# Full size: the Ouro-1.4B-shaped decode call the benchmark times (batch 32,
# context 4096, (192, 320), the library's split choice), sampled (b, h).
# ---------------------------------------------------------------------------

@pytest.mark.slow
def test_full_ouro14b_fullrope():
    wl = W.WORKLOADS["ouro14b_decode"]
    r_k, r_v = 192, 320
    n_max = wl.N + 64
    for layer, loop in ((0, 0), (23, 3)):
        log(f"fullrope ouro14b layer={layer} loop={loop}")
        pk = lla.to_paged(W.latents(wl, r_k, "k", layer, device=DEV), n_max)
        pv = lla.to_paged(W.latents(wl, r_v, "v", layer, device=DEV), n_max)
        q = W.queries(wl, layer, loop, device=DEV)
        uk, uv, _, _ = W.codec_loop(wl, r_k, r_v, layer, loop, DEV)
        ws = lla.new_workspace(wl.B, wl.H, r_v, wl.N)
        out = lla.decode_attn_fullrope(q, pk, pv, uk, uv, n_ctx=wl.N, workspace=ws)
        torch.cuda.synchronize()
        o = f64(out)
        for b, h in [(0, 0), (7, 5), (16, 15), (31, 8)]:
            ck = f64(lla.from_paged(pk[b:b + 1, h:h + 1], wl.N))[0, 0]
            cv = f64(lla.from_paged(pv[b:b + 1, h:h + 1], wl.N))[0, 0]
            ref = oracle.decode_attn_fullrope(f64(q[b, h]), ck, cv, f64(uk[h]), f64(uv[h]))
            assert_close(o[b, h], ref, torch.bfloat16, f"unit ({b},{h})")
            _tight(o[b, h], ref, f"unit ({b},{h})")
        del pk, pv
        torch.cuda.empty_cache()
