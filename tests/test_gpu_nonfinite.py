"""Non-finite data and the fp16 range of the prefills, on the GPU, through the
C ABI: each assertion here is a sentence of include/lla.h.

* A NaN in an attended latent makes the outputs of exactly the queries that
  attend it non-finite; decode ignores whatever the slots past N_b hold.
* In the prefills a masked (future) key of a 64-key page enters the value
  product with weight 0, and 0 * NaN = NaN: a NaN value latent at position n
  may also reach the queries at positions 64 floor(n/64) - 31 .. n - 1.
  Queries further back are untouched.  A NaN key latent reaches no query that
  does not attend it (masked scores are replaced by -inf).
* The per-head prefill converts latent pages to fp16: the largest bf16 value
  below fp16's maximum (65280) still gives the oracle's result; the next bf16
  value (65536) overflows, and the queries that attend it get non-finite
  outputs.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_15456_amd import lla, workloads as W
from tests.helpers import BF16_REL_L2, assert_close, f64, log

pytestmark = pytest.mark.gpu

DEV = "cuda"
WL = W.Workload("nonfinite", 1, 2, 128, 4, 1, 0, ((18, 30),), torch.bfloat16)


def _per_head_case(M, r_k=18, r_v=30):
    B, H = 1, WL.H
    ck = W.latents(WL, r_k, "k", 0, B=B, N=M, device=DEV)
    cv = W.latents(WL, r_v, "v", 0, B=B, N=M, device=DEV)
    q = W.queries(WL, 0, 1, B=B, M=M, device=DEV)
    uk, uv, _, _ = W.codec_loop(WL, r_k, r_v, 0, 1, DEV)
    return q, ck, cv, uk, uv


def _prefill_rows_ref(q, ck, cv, uk, uv, rows, b=0, h=0):
    q64, k64, v64, uk64, uv64 = f64(q), f64(ck), f64(cv), f64(uk), f64(uv)
    return np.stack([oracle.decode_attn_absorbed(q64[b, h, m], k64[b, h, :m + 1], v64[b, h, :m + 1], uk64[h], uv64[h])
                     for m in rows])


@pytest.mark.parametrize("axis", ["k", "v"])
def test_prefill_nan_latent(axis):
    M, n_bad, b, h = 320, 200, 0, 1
    q, ck, cv, uk, uv = _per_head_case(M)
    bad = ck if axis == "k" else cv
    bad[b, h, n_bad, 3] = float("nan")
    n_max = 384
    out = f64(lla.prefill_attn(q, lla.to_paged(ck, n_max), lla.to_paged(cv, n_max), uk, uv, p0=0))
    log(f"prefill NaN in c_{axis} at position {n_bad}")
    assert np.all(np.isnan(out[b, h, n_bad:])), "queries attending the NaN must be NaN"
    first_clean = 64 * (n_bad // 64) - 31 if axis == "v" else n_bad
    rows = list(range(0, first_clean))
    assert_close(out[b, h, rows], _prefill_rows_ref(q, ck, cv, uk, uv, rows, b, h), torch.bfloat16,
                 f"rows before {first_clean}")
    other = [m for m in range(M)]
    assert_close(out[b, 1 - h], _prefill_rows_ref(q, ck, cv, uk, uv, other, b, 1 - h), torch.bfloat16,
                 "the other head")


@pytest.mark.parametrize("axis", ["k", "v"])
def test_prefill_2d_nan_latent(axis):
    B, H, M, r_k, r_v, n_bad = 1, 2, 320, 32, 48, 200
    wl = W.Workload("nonfinite_2d", 1, H, 128, 4, B, 0, ((r_k, r_v),), torch.bfloat16)
    ck = W.latents_2d(wl, r_k, "k", 0, B=B, N=M, device=DEV)
    cv = W.latents_2d(wl, r_v, "v", 0, B=B, N=M, device=DEV)
    q = W.queries(wl, 0, 1, B=B, M=M, device=DEV)
    uk, uv = W.codec_loop_2d(wl, r_k, r_v, 0, 1, DEV)
    (ck if axis == "k" else cv)[0, n_bad, 5] = float("nan")
    n_max = 384
    kc = ck.new_zeros((B, n_max, r_k))
    kc[:, :M] = ck
    vfull = cv.new_zeros((B, n_max, r_v))
    vfull[:, :M] = cv
    vc = vfull.view(B, n_max // 64, 64, r_v).transpose(-1, -2).contiguous()
    out = f64(lla.prefill_attn_2d(q, kc, vc, uk, uv, p0=0))
    log(f"2D prefill NaN in c_{axis} at position {n_bad}")
    assert np.all(np.isnan(out[0, :, n_bad:]))
    first_clean = 64 * (n_bad // 64) - 31 if axis == "v" else n_bad
    ref = oracle.prefill_attn_2d(f64(q)[0][:, :first_clean], f64(ck)[0], f64(cv)[0], f64(uk), f64(uv))
    assert_close(out[0, :, :first_clean], ref, torch.bfloat16, f"rows before {first_clean}")


def test_decode_nan_inside_and_past_context():
    B, H, N, n_max, r_k, r_v = 2, 2, 300, 384, 36, 60
    ck = W.latents(WL, r_k, "k", 0, B=B, N=n_max, device=DEV)
    cv = W.latents(WL, r_v, "v", 0, B=B, N=n_max, device=DEV)
    q = W.queries(WL, 0, 0, B=B, device=DEV)
    uk, uv, _, _ = W.codec_loop(WL, r_k, r_v, 0, 0, DEV)
    ck[:, :, N:] = float("nan")   # slots past the context: never attended
    cv[:, :, N:] = float("nan")
    cv[1, 0, 17, 2] = float("nan")  # an attended value of sequence 1, head 0
    pk, pv = lla.to_paged(ck, n_max), lla.to_paged(cv, n_max)
    out = f64(lla.decode_attn(q, pk, pv, uk, uv, n_ctx=N))
    assert np.all(np.isnan(out[1, 0]))
    ref = oracle.decode_attn_batched(f64(q), f64(ck), f64(cv), f64(uk), f64(uv), ctx_len=N)
    assert_close(out[0], ref[0], torch.bfloat16, "sequence 0")
    assert_close(out[1, 1:], ref[1, 1:], torch.bfloat16, "sequence 1, other head")


@pytest.mark.parametrize("big,finite", [(65280.0, True), (65536.0, False)])
def test_prefill_fp16_range_of_value_latents(big, finite):
    """65280 is the largest bf16 value fp16 holds (its maximum is 65504); 65536
    is the next bf16 value and overflows fp16."""
    M, n_big, b, h = 256, 200, 0, 0
    q, ck, cv, uk, uv = _per_head_case(M)
    cv[b, h, n_big, :] = big
    cv[b, h, n_big, 1::2] = -big
    assert float(cv[b, h, n_big, 0]) == big  # bf16-exact
    out = f64(lla.prefill_attn(q, lla.to_paged(ck, 320), lla.to_paged(cv, 320), uk, uv, p0=0))
    log(f"value latents of magnitude {big}")
    ref = _prefill_rows_ref(q, ck, cv, uk, uv, list(range(M)), b, h)
    first_clean = 64 * (n_big // 64) - 31
    assert_close(out[b, h, :first_clean], ref[:first_clean], torch.bfloat16, "rows well before it")
    if finite:
        assert np.all(np.isfinite(out))
        err = out[b, h, n_big:] - ref[n_big:]
        rel = np.linalg.norm(err) / np.linalg.norm(ref[n_big:])
        log(f"  attending rows: rel_l2={rel:.3e}, largest |out| {np.abs(out[b, h, n_big:]).max():.1f}")
        assert rel <= BF16_REL_L2
    else:
        assert not np.isfinite(out[b, h, n_big:]).all(axis=-1).any(), "attending rows must be non-finite"
