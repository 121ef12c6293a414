"""GPU parity of the decoupled rotary branch (App. J "Absorbed attention": a
NoPE content path plus a small explicit rotary key per token, shared across
loops) against the float64 oracle, through the C ABI: the rotary writes and
query rotation, and decode and prefill with the branch."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_15456_amd import lla, workloads as W
from tests.helpers import assert_close, f64, f64_dev, log

pytestmark = pytest.mark.gpu

DEV = "cuda"
SENTINEL = 3.0
SMALL = W.Workload("rope_small", 1, 4, 128, 4, 3, 0, ((18, 30),), torch.bfloat16)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("dr,Hr,M,pos0,n_max", [(64, 1, 5, 0, 128), (32, 4, 70, 61, 192), (96, 2, 1, 4095, 4160),
                                               (8, 1, 3, 262140, 262144)])
def test_rope_write_matches_oracle(dtype, dr, Hr, M, pos0, n_max):
    log(f"rope_write dr={dr} Hr={Hr} M={M} pos0={pos0} {dtype}")
    B = 2
    k = W.rotary_keys(SMALL, dr, Hr, 0, B=B, N=M, device=DEV, dtype=dtype)
    rc = torch.full((B, Hr, n_max // 64, dr, 64), SENTINEL, dtype=dtype, device=DEV)
    lla.rope_write(k, rc, pos0=pos0, base=10000.0)
    torch.cuda.synchronize()
    got = f64(lla.from_paged(rc))                                  # [B, Hr, n_max, dr]
    ref = oracle.rope(f64(k), (pos0 + np.arange(M))[None, :, None], 10000.0)  # [B, M, Hr, dr]
    assert_close(got[:, :, pos0:pos0 + M], ref.transpose(0, 2, 1, 3), dtype, "rotated keys",
                 out_bf16=dtype == torch.bfloat16)
    rest = np.concatenate([got[:, :, :pos0].ravel(), got[:, :, pos0 + M:].ravel()])
    assert np.all(rest == SENTINEL), "slots outside [pos0, pos0 + M) changed"


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_rope_rotate_matches_oracle(dtype):
    B, G, M, dr = 3, 4, 9, 64
    x = W.normal((B, G, M, dr), ("rope_rotate", "x"), 1.0, dtype, DEV)
    pos = torch.tensor([0, 17, 100000], dtype=torch.int32, device=DEV)
    for p, p0 in ((None, 33), (pos, 0)):
        y = lla.rope_rotate(x, pos=p, pos0=p0, base=500000.0)
        torch.cuda.synchronize()
        base_pos = np.full(B, p0) if p is None else pos.cpu().numpy()
        P = base_pos[:, None, None] + np.arange(M)[None, None, :]
        ref = oracle.rope(f64(x), P, 500000.0)
        assert_close(f64(y), ref, dtype, f"rotate pos={'array' if p is not None else p0}",
                     out_bf16=dtype == torch.bfloat16)
    # [B, G, d_rope] rows are rotated at pos[b] (M = 1)
    y1 = lla.rope_rotate(x[:, :, 0].contiguous(), pos=pos)
    ref1 = oracle.rope(f64(x[:, :, 0]), pos.cpu().numpy()[:, None].astype(np.float64))
    assert_close(f64(y1), ref1, dtype, "rotate M=1", out_bf16=dtype == torch.bfloat16)


def _decode_case(wl, r_k, r_v, dr, Hr, B, N, n_max, dtype, means):
    ck = W.latents(wl, r_k, "k", 0, B=B, N=N, device=DEV, dtype=dtype)
    cv = W.latents(wl, r_v, "v", 0, B=B, N=N, device=DEV, dtype=dtype)
    kr = W.rotary_keys(wl, dr, Hr, 0, B=B, N=N, device=DEV, dtype=dtype)
    q = W.queries(wl, 0, 1, B=B, device=DEV, dtype=dtype)
    qr = W.rotary_queries(wl, dr, 0, 1, B=B, device=DEV, dtype=dtype)
    uk, uv, muk, muv = W.codec_loop(wl, r_k, r_v, 0, 1, DEV, dtype, means=means)
    rc = lla.alloc_cache(B, Hr, n_max, dr, dtype=dtype, device=DEV)
    lla.rope_write(kr, rc, pos0=0)
    return ck, cv, kr, q, qr, uk, uv, muk, muv, rc


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("r_k,r_v,dr,Hr", [(18, 30, 64, 1), (96, 160, 64, 4), (7, 9, 32, 1), (192, 320, 64, 1),
                                           (36, 60, 96, 4)])
@pytest.mark.parametrize("N", [1, 130, 700])
def test_decode_rope(dtype, r_k, r_v, dr, Hr, N):
    wl, B = SMALL, 3
    n_max = ((N + 63) // 64) * 64
    log(f"decode rope r=({r_k},{r_v}) dr={dr} Hr={Hr} N={N} {dtype}")
    ck, cv, kr, q, qr, uk, uv, muk, muv, rc = _decode_case(wl, r_k, r_v, dr, Hr, B, N, n_max, dtype, True)
    qr_rot = lla.rope_rotate(qr, pos0=N - 1)
    out = lla.decode_attn(q, lla.to_paged(ck, n_max), lla.to_paged(cv, n_max), uk, uv, n_ctx=N, mu_k=muk,
                          mu_v=muv, q_rope=qr_rot, r_cache=rc)
    torch.cuda.synchronize()
    ref = oracle.decode_attn_rope_batched(f64(q), f64(qr), f64(ck), f64(cv), f64(kr).transpose(0, 2, 1, 3),
                                          f64(uk), f64(uv), f64(muk), f64(muv))
    assert_close(f64(out), ref, dtype, "decode rope")


@pytest.mark.parametrize("r_k,r_v,dr,Hr", [(17, 30, 8, 1), (33, 160, 24, 4), (95, 9, 40, 1), (1, 1, 8, 4),
                                           (7, 300, 64, 1)])
@pytest.mark.parametrize("N,lens", [(1500, [1500, 700, 65]), (1000, [1000, 513, 1])])
def test_decode_rope_short_context(r_k, r_v, dr, Hr, N, lens):
    """Short bf16 contexts.  At 17 to 24 pages the K phase takes groups of 4
    pages, each wave-wide load covering two feature rows: an odd r_k, or a
    rotary width that is not a multiple of 16, leaves the last pair half past
    its range.  At up to 16 pages the wavefronts split the feature rows of
    each 8-page group (8-row blocks of content and rotary rows, 8-row value
    groups): ranks that are not multiples of 8 or 32 leave blocks and groups
    partly past their range.  The per-sequence lengths give partial groups,
    ragged last pages and a one-token context."""
    wl, B, n_max = SMALL, 3, 1536
    dtype = torch.bfloat16
    log(f"decode rope short context N={N} r=({r_k},{r_v}) dr={dr} Hr={Hr}")
    ck, cv, kr, q, qr, uk, uv, muk, muv, rc = _decode_case(wl, r_k, r_v, dr, Hr, B, N, n_max, dtype, True)
    lens = torch.tensor(lens, dtype=torch.int32, device=DEV)
    qr_rot = lla.rope_rotate(qr, pos=lens - 1)
    out = lla.decode_attn(q, lla.to_paged(ck, n_max), lla.to_paged(cv, n_max), uk, uv, n_ctx=N, ctx_len=lens,
                          mu_k=muk, mu_v=muv, q_rope=qr_rot, r_cache=rc)
    torch.cuda.synchronize()
    ref = np.stack([oracle.decode_attn_rope_batched(f64(q)[b:b + 1], f64(qr)[b:b + 1], f64(ck)[b:b + 1],
                                                    f64(cv)[b:b + 1], f64(kr).transpose(0, 2, 1, 3)[b:b + 1],
                                                    f64(uk), f64(uv), f64(muk), f64(muv), ctx_len=int(lens[b]))[0]
                    for b in range(B)])
    assert_close(f64(out), ref, dtype, "decode rope, short contexts")


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_decode_rope_ragged_lengths_and_split(dtype):
    """Per-sequence lengths (each query rotated at its own newest position) and
    the split-K workspace path."""
    wl, B, N, n_max = SMALL, 2, 3000, 3008
    r_k, r_v, dr, Hr = 96, 160, 64, 1
    ck, cv, kr, q, qr, uk, uv, muk, muv, rc = _decode_case(wl, r_k, r_v, dr, Hr, B, N, n_max, dtype, False)
    lens = torch.tensor([3000, 1234], dtype=torch.int32, device=DEV)
    qr_rot = lla.rope_rotate(qr, pos=lens - 1)
    ws = lla.new_workspace(B, wl.H, r_v, N)
    out = lla.decode_attn(q, lla.to_paged(ck, n_max), lla.to_paged(cv, n_max), uk, uv, n_ctx=N, ctx_len=lens,
                          q_rope=qr_rot, r_cache=rc, workspace=ws)
    torch.cuda.synchronize()
    ref = np.stack([oracle.decode_attn_rope_batched(f64(q)[b:b + 1], f64(qr)[b:b + 1], f64(ck)[b:b + 1],
                                                    f64(cv)[b:b + 1], f64(kr).transpose(0, 2, 1, 3)[b:b + 1],
                                                    f64(uk), f64(uv), ctx_len=int(lens[b]))[0]
                    for b in range(B)])
    assert_close(f64(out), ref, dtype, "decode rope ragged + split")


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("r_k,r_v,dr,Hr", [(18, 30, 64, 1), (7, 9, 32, 4), (31, 60, 32, 1), (24, 95, 64, 4)])
@pytest.mark.parametrize("M,p0", [(1, 0), (130, 0), (77, 100), (200, 5)])
def test_prefill_rope(dtype, r_k, r_v, dr, Hr, M, p0):
    wl, B = SMALL, 2
    N = p0 + M
    n_max = ((N + 63) // 64) * 64 + 64
    log(f"prefill rope r=({r_k},{r_v}) dr={dr} Hr={Hr} M={M} p0={p0} {dtype}")
    ck = W.latents(wl, r_k, "k", 0, B=B, N=N, device=DEV, dtype=dtype)
    cv = W.latents(wl, r_v, "v", 0, B=B, N=N, device=DEV, dtype=dtype)
    kr = W.rotary_keys(wl, dr, Hr, 0, B=B, N=N, device=DEV, dtype=dtype)
    q = W.queries(wl, 0, 2, B=B, M=M, device=DEV, dtype=dtype)
    qr = W.rotary_queries(wl, dr, 0, 2, B=B, M=M, device=DEV, dtype=dtype)
    uk, uv, muk, muv = W.codec_loop(wl, r_k, r_v, 0, 2, DEV, dtype, means=True)
    rc = torch.full((B, Hr, n_max // 64, dr, 64), float("nan"), dtype=dtype, device=DEV)  # unwritten: NaN
    lla.rope_write(kr, rc, pos0=0)
    pk = lla.to_paged(ck, n_max)
    pv = lla.to_paged(cv, n_max)
    qr_rot = lla.rope_rotate(qr, pos0=p0)
    out = lla.prefill_attn(q, pk, pv, uk, uv, p0=p0, mu_k=muk, mu_v=muv, q_rope=qr_rot, r_cache=rc)
    torch.cuda.synchronize()
    ref = oracle.prefill_attn_rope_batched(f64(q), f64(qr), f64(ck), f64(cv), f64(kr).transpose(0, 2, 1, 3),
                                           f64(uk), f64(uv), f64(muk), f64(muv), p0=p0)
    assert_close(f64(out), ref, dtype, "prefill rope")


@pytest.mark.parametrize("N,r_k,r_v,Hr", [(32768, 96, 160, 1), (32768, 192, 320, 16), (131072, 96, 160, 1),
                                           (16384, 96, 160, 1), (16384, 192, 320, 16)])
def test_decode_rope_split_k(N, r_k, r_v, Hr):
    """One sequence of 16 heads over a long context with the rotary branch,
    the shape of the absorbed-against-rebuilt latency comparison (App. J):
    the launch splits each (b, h) context over 16 workgroups of 8 wavefronts
    (4-page K groups at 32,768 tokens, 8-page groups at 131,072, the row-split
    kernel's 16-page slices at 16,384) and merges their partial states.  Full
    and ragged lengths, every head checked."""
    B, H, dr, dtype = 1, 16, 64, torch.bfloat16
    # (16,384 tokens: the row-split kernel over 16-page slices, 20 or more row blocks)
    assert lla.decode_splits(dtype, B, H, N, r_k, r_v, dr) == 16
    wl = W.Workload("rope_split", 1, H, 128, 4, B, N, ((r_k, r_v),), dtype)
    log(f"decode rope split-K N={N} r=({r_k},{r_v}) Hr={Hr}")
    ck, cv, kr, q, qr, uk, uv, muk, muv, rc = _decode_case(wl, r_k, r_v, dr, Hr, B, N, N, dtype, True)
    pk, pv = lla.to_paged(ck, N), lla.to_paged(cv, N)
    ws = lla.new_workspace(B, H, r_v, N)
    q64, qr64, ck64, cv64 = f64(q), f64(qr), f64_dev(ck), f64_dev(cv)
    kr64, uk64, uv64, muk64, muv64 = f64(kr).transpose(0, 2, 1, 3), f64(uk), f64(uv), f64(muk), f64(muv)
    del ck, cv
    for n in (N, N - 777):
        lens = torch.tensor([n], dtype=torch.int32, device=DEV)
        qr_rot = lla.rope_rotate(qr, pos=lens - 1)
        out = lla.decode_attn(q, pk, pv, uk, uv, n_ctx=N, ctx_len=lens, mu_k=muk, mu_v=muv,
                              q_rope=qr_rot, r_cache=rc, workspace=ws)
        torch.cuda.synchronize()
        ref = oracle.decode_attn_rope_batched(q64, qr64, ck64, cv64, kr64, uk64, uv64, muk64, muv64, ctx_len=n)
        assert_close(f64(out), ref, dtype, f"decode rope split-K n={n}")
    assert int(ws[:4 * B * H].view(torch.int32).abs().sum()) == 0
