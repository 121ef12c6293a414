"""Host-side checks of the C ABI (no GPU needed).

The library must load and export every entry point include/lla.h declares;
host-only entry points (rho, cache bytes, workspace size, status strings) are
checked against the paper's printed values; every invalid argument must be
rejected with its status code before anything is launched.  No call here
reaches a kernel: each device entry point is only called with arguments that
host validation refuses.
"""

import ctypes
import os
import re
from fractions import Fraction

import pytest

from paper_2607_15456_amd import lla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lla.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:const char\*|int|lla_status)\s+(lla_\w+)\(", src, re.M)))


def test_header_declares_the_boundary():
    names = _declared()
    assert names == sorted(["lla_status_string", "lla_abi_version", "lla_rho", "lla_cache_bytes",
                            "lla_encode", "lla_decode_workspace_bytes", "lla_decode_splits", "lla_decode_attn",
                            "lla_decode_attn_noalloc",
                            "lla_prefill_attn", "lla_prefill_workspace_bytes", "lla_rope_write",
                            "lla_rope_rotate",
                            "lla_decode_attn_rope", "lla_prefill_attn_rope", "lla_encode_ring",
                            "lla_rope_write_ring", "lla_encode_2d", "lla_encode_2d_workspace_bytes",
                            "lla_decode_2d_workspace_bytes", "lla_decode_attn_2d",
                            "lla_decode_attn_fullrope", "lla_prefill_2d_workspace_bytes",
                            "lla_prefill_attn_2d"])


def test_library_exports_every_declared_symbol():
    h = ctypes.CDLL(lla.LIB_PATH)
    for name in _declared():
        assert hasattr(h, name), name
    assert lla.abi_version() == 10


def test_decode_split_choice():
    """The split-K choice (the library's launch heuristic on a 256-CU MI355X): a
    batch that fills the machine with one workgroup per (b, h) is not split; one
    sequence of 16 heads over a long context is, in proportion to its pages."""
    import torch
    bf, f32 = torch.bfloat16, torch.float32
    r2 = (192, 320)  # the Ouro-1.4B ranks
    assert lla.decode_splits(bf, 32, 16, 4096, *r2) == 1          # the Ouro-1.4B decode step
    assert lla.decode_splits(bf, 16, 16, 32768, 36, 60) == 1      # the Ouro-2.6B long-context step
    assert lla.decode_splits(bf, 64, 16, 8192, 96, 160) == 1      # the rank sweep
    # one sequence: fp32 keeps a whole 8-page group per wavefront; bf16 takes the
    # row-split kernel over 8-page slices up to one workgroup per compute unit
    # (8192 tokens), beyond that one 4-page group per wavefront
    assert lla.decode_splits(f32, 1, 16, 8192, *r2) == 2
    assert lla.decode_splits(bf, 1, 16, 8192, *r2) == 16
    assert lla.decode_splits(f32, 1, 16, 32768, *r2) == 8
    assert lla.decode_splits(bf, 1, 16, 32768, *r2) == 16
    assert lla.decode_splits(bf, 1, 16, 1024, *r2) == 2
    assert lla.decode_splits(bf, 4, 16, 16384, *r2) == 4          # 64 units: 8-page groups, 4 splits
    for dt in (bf, f32):
        assert lla.decode_splits(dt, 2, 16, 32768, *r2) == 8
        assert lla.decode_splits(dt, 1, 16, 32768, *r2, with_workspace=False) == 1
        assert lla.decode_splits(dt, 1, 16, 512, *r2) == 1
    # more than 16 row blocks (8-row key blocks with the rotary rows, or value
    # groups): 16-page slices where 8-page ones would need two workgroups per
    # compute unit; smaller ranks keep the general kernel's shapes
    assert lla.decode_splits(bf, 1, 16, 16384, *r2) == 16
    assert lla.decode_splits(bf, 1, 16, 16384, 36, 60) == 8
    assert lla.decode_splits(bf, 2, 16, 8192, 288, 480) == 8
    assert lla.decode_splits(bf, 2, 16, 8192, 36, 60) == 4
    assert lla.decode_splits(bf, 2, 16, 8192, 64, 128) == 4       # 16 row blocks
    assert lla.decode_splits(bf, 2, 16, 8192, 64, 64, 72) == 8    # 8 + 9 key blocks
    assert lla.decode_splits(f32, 1, 16, 16384, *r2) == 4
    # 129-256 units over at most 128 pages at 16-60 row blocks (or at most 32
    # pages at any rank): one row-split workgroup per (b, h), not split;
    # smaller ranks over longer contexts keep the general kernel's 2
    assert lla.decode_splits(bf, 16, 16, 2048, 288, 480) == 1
    assert lla.decode_splits(bf, 16, 16, 2048, 36, 60) == 1
    assert lla.decode_splits(bf, 12, 16, 8192, 64, 128) == 1
    assert lla.decode_splits(bf, 12, 16, 8192, 36, 60) == 2
    with pytest.raises(lla.LLAError):
        lla.decode_splits(bf, 0, 16, 4096, *r2)
    with pytest.raises(lla.LLAError):
        lla.decode_splits(bf, 1, 16, 4096, 0, 320)
    with pytest.raises(lla.LLAError):
        lla.decode_splits(bf, 1, 16, 4096, 192, 320, -8)


def test_status_strings():
    for code, tag in [(0, "LLA_OK"), (1, "INVALID_ARG"), (2, "UNSUPPORTED"), (3, "WORKSPACE"), (4, "HIP"),
                      (5, "SCRATCH")]:
        assert tag in lla.status_string(code)
    assert "unknown" in lla.status_string(99)


def _golden(name):
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


def test_rho_matches_printed_tiers():
    for T, d, rk, rv, printed, dec, *_ in _golden("rho_tiers.txt"):
        r = lla.rho(int(T), int(d), int(rk), int(rv))
        assert r == Fraction(2 * int(T) * int(d), int(rk) + int(rv))
        assert f"{float(r):.{int(dec)}f}" == printed
    assert lla.rho(4, 128, 36, 60) == Fraction(32, 3)
    assert lla.rho(4, 128, 18, 30) == Fraction(64, 3)


def test_rho_rejects_bad_args():
    for bad in [(0, 128, 96, 160), (4, -1, 96, 160), (4, 128, 0, 160), (4, 128, 96, 0)]:
        with pytest.raises(lla.LLAError) as e:
            lla.rho(*bad)
        assert e.value.status == lla.LLA_ERR_INVALID_ARG


UNIT = {"KiB": 1024, "MiB": 1024 ** 2, "GiB": 1024 ** 3}


def test_cache_bytes_match_tab_memory():
    for layers, tokens, rk, rv, val, unit, *_ in _golden("cache_bytes.txt"):
        latent = int(rk) > 0
        got = lla.cache_bytes(int(layers), 16, 4, 128, int(rk) or 1, int(rv) or 1, int(tokens), 2, latent)
        assert got == int(val) * UNIT[unit]


def test_cache_bytes_overflow_and_bad_args():
    with pytest.raises(lla.LLAError):
        lla.cache_bytes(1 << 40, 1 << 20, 4, 128, 1, 1, 1 << 20, 2, True)
    with pytest.raises(lla.LLAError):
        lla.cache_bytes(24, 16, 4, 128, 96, 160, -1, 2, True)
    assert lla.cache_bytes(24, 16, 4, 128, 96, 160, 0, 2, True) == 0


def test_workspace_bytes():
    # counters (256-byte aligned) + B*H*S*(r_v+2) floats, S = min(64, pages)
    assert lla.decode_workspace_bytes(32, 16, 320, 4096) == 2048 + 512 * 64 * 322 * 4
    assert lla.decode_workspace_bytes(1, 16, 160, 512) == 256 + 16 * 8 * 162 * 4
    with pytest.raises(lla.LLAError):
        lla.decode_workspace_bytes(0, 16, 160, 512)
    with pytest.raises(lla.LLAError):
        lla.decode_workspace_bytes(1, 16, 513, 512)


# ---- device entry points: invalid arguments are refused on the host ----

P = 0x10000  # aligned fake device address: never dereferenced, validation fails first
MIS = 0x10008  # misaligned


def _decode(**kw):
    a = dict(dtype=1, out_dtype=0, B=2, H=16, d=128, rk=96, rv=160, n_max=512, n_ctx=512, ctx_len=None,
             q=P, ck=P, cv=P, uk=P, uv=P, muk=None, muv=None, scale=0.088, out=P, ws=None, ws_bytes=0,
             stream=None)
    a.update(kw)
    return lla.lib().lla_decode_attn(a["dtype"], a["out_dtype"], a["B"], a["H"], a["d"], a["rk"], a["rv"],
                                     a["n_max"], a["n_ctx"], a["ctx_len"], a["q"], a["ck"], a["cv"],
                                     a["uk"], a["uv"], a["muk"], a["muv"], a["scale"], a["out"], a["ws"],
                                     a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=2), 1), (dict(out_dtype=-1), 1), (dict(B=0), 1), (dict(H=0), 1),
    (dict(d=48), 1), (dict(d=512), 1), (dict(rk=0), 1), (dict(rv=513), 1),
    (dict(n_max=500), 1), (dict(n_ctx=0), 1), (dict(n_ctx=513), 1),
    (dict(scale=0.0), 1), (dict(scale=float("nan")), 1), (dict(scale=float("inf")), 1),
    (dict(q=None), 1), (dict(ck=MIS), 1), (dict(out=None), 1), (dict(muv=MIS), 1),
    (dict(ctx_len=P + 2), 1),
    (dict(ws=P, ws_bytes=0), 3), (dict(ws=None, ws_bytes=64), 3), (dict(ws=P, ws_bytes=64), 3),
    (dict(ws=MIS, ws_bytes=1 << 30), 3),
    # one (b, h) region of n_max * r elements must stay below 2 GiB (32-bit offsets)
    (dict(n_max=1 << 23), 2), (dict(dtype=0, n_max=1 << 22), 2),
])
def test_decode_rejects(kw, code):
    assert _decode(**kw) == code


def _decode_noalloc(**kw):
    a = dict(dtype=1, out_dtype=0, B=2, H=16, d=128, rk=96, rv=160, n_max=512, n_ctx=512, ctx_len=None,
             q=P, ck=P, cv=P, uk=P, uv=P, muk=None, muv=None, scale=0.088, out=P, stream=None)
    a.update(kw)
    return lla.lib().lla_decode_attn_noalloc(a["dtype"], a["out_dtype"], a["B"], a["H"], a["d"], a["rk"],
                                             a["rv"], a["n_max"], a["n_ctx"], a["ctx_len"], a["q"], a["ck"],
                                             a["cv"], a["uk"], a["uv"], a["muk"], a["muv"], a["scale"], a["out"],
                                             a["stream"])


@pytest.mark.parametrize("kw", [
    dict(dtype=2), dict(B=0), dict(d=48), dict(rk=0), dict(rv=513), dict(n_max=500), dict(n_ctx=0),
    dict(n_ctx=513), dict(scale=float("nan")), dict(q=None), dict(ck=MIS), dict(out=None), dict(ctx_len=P + 2),
])
def test_decode_noalloc_rejects(kw):
    assert _decode_noalloc(**kw) == lla.LLA_ERR_INVALID_ARG


def _encode(**kw):
    a = dict(dtype=1, B=2, M=8, H=16, T=4, d=128, rk=18, rv=30, xk=P, xv=P, muk=None, muv=None, wk=P, wv=P,
             ck=P, cv=P, n_max=512, pos0=0, stream=None)
    a.update(kw)
    return lla.lib().lla_encode(a["dtype"], a["B"], a["M"], a["H"], a["T"], a["d"], a["rk"], a["rv"],
                                a["xk"], a["xv"], a["muk"], a["muv"], a["wk"], a["wv"], a["ck"], a["cv"],
                                a["n_max"], a["pos0"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(dtype=3), dict(B=0), dict(M=0), dict(H=0), dict(T=0), dict(d=100), dict(rk=0), dict(rv=600),
    dict(n_max=100), dict(pos0=-1), dict(pos0=505), dict(xk=None), dict(wv=MIS), dict(cv=None),
    dict(muk=MIS),
])
def test_encode_rejects(kw):
    assert _encode(**kw) == lla.LLA_ERR_INVALID_ARG


def _prefill(**kw):
    a = dict(dtype=1, out_dtype=0, B=1, H=16, M=64, d=128, rk=18, rv=30, n_max=512, p0=0, q=P, ck=P, cv=P,
             uk=P, uv=P, muk=None, muv=None, scale=0.088, out=P, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return lla.lib().lla_prefill_attn(a["dtype"], a["out_dtype"], a["B"], a["H"], a["M"], a["d"], a["rk"],
                                      a["rv"], a["n_max"], a["p0"], a["q"], a["ck"], a["cv"], a["uk"],
                                      a["uv"], a["muk"], a["muv"], a["scale"], a["out"], a["ws"],
                                      a["ws_bytes"], a["stream"])


REBUILD = dict(rk=96, rv=160)  # the 4x tier: bf16 takes the rebuild path, which needs a workspace
REBUILD_WS = 4 * 1 * 16 * 128 * 64  # B * H * d_head * (p0 + M rounded up to 64) * 2 tensors * 2 bytes


@pytest.mark.parametrize("kw,code", [
    (dict(M=0), 1), (dict(p0=-1), 1), (dict(p0=449), 1), (dict(d=40), 1), (dict(q=MIS), 1),
    (dict(scale=-1.0), 1), (dict(rk=96), 2), (dict(rv=96), 2), (dict(d=256), 2),
    (dict(REBUILD), 3), (dict(REBUILD, ws=P, ws_bytes=REBUILD_WS - 16), 3), (dict(REBUILD, ws=MIS, ws_bytes=1 << 30), 3),
    (dict(REBUILD, ws=P, ws_bytes=0), 3), (dict(rk=100, rv=160, ws=P, ws_bytes=1 << 30), 2),
    (dict(REBUILD, d=64, ws=P, ws_bytes=1 << 30), 2), (dict(ws=None, ws_bytes=16), 3),
    (dict(n_max=1 << 26), 2),
])
def test_prefill_rejects(kw, code):
    assert _prefill(**kw) == code


def test_prefill_workspace_bytes():
    assert lla.prefill_workspace_bytes(torch_bf16(), 1, 16, 64, 128, 96, 160, 0) == REBUILD_WS
    assert lla.prefill_workspace_bytes(torch_bf16(), 4, 16, 8192, 128, 288, 480, 0) == 4 * 4 * 16 * 128 * 8192
    assert lla.prefill_workspace_bytes(torch_bf16(), 2, 3, 100, 128, 96, 160, 5) == 4 * 2 * 3 * 128 * 128
    assert lla.prefill_workspace_bytes(torch_bf16(), 4, 16, 8192, 128, 18, 30, 0) == 0   # absorbed kernel
    import torch
    assert lla.prefill_workspace_bytes(torch.float32, 1, 16, 64, 128, 96, 160, 0) == 0   # fp32 scan
    with pytest.raises(lla.LLAError):
        lla.prefill_workspace_bytes(torch_bf16(), 1, 16, 0, 128, 96, 160, 0)


def torch_bf16():
    import torch
    return torch.bfloat16


# ---- the decoupled rotary branch ----

def _decode_rope(**kw):
    a = dict(dtype=1, out_dtype=0, B=2, H=16, d=128, rk=96, rv=160, dr=64, Hr=1, n_max=512, n_ctx=512,
             ctx_len=None, q=P, qr=P, ck=P, cv=P, rc=P, uk=P, uv=P, muk=None, muv=None, scale=0.088, out=P,
             ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return lla.lib().lla_decode_attn_rope(a["dtype"], a["out_dtype"], a["B"], a["H"], a["d"], a["rk"],
                                          a["rv"], a["dr"], a["Hr"], a["n_max"], a["n_ctx"], a["ctx_len"],
                                          a["q"], a["qr"], a["ck"], a["cv"], a["rc"], a["uk"], a["uv"],
                                          a["muk"], a["muv"], a["scale"], a["out"], a["ws"], a["ws_bytes"],
                                          a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(dr=0), 1), (dict(dr=12), 1), (dict(dr=264), 1), (dict(Hr=2), 1), (dict(Hr=0), 1),
    (dict(qr=None), 1), (dict(rc=None), 1), (dict(qr=MIS), 1), (dict(rk=500, dr=16), 1),
    (dict(B=0), 1), (dict(ws=P, ws_bytes=0), 3), (dict(rk=8, rv=8, dr=256, n_max=1 << 22), 2),
])
def test_decode_rope_rejects(kw, code):
    assert _decode_rope(**kw) == code


def _prefill_rope(**kw):
    a = dict(dtype=1, out_dtype=0, B=1, H=16, M=64, d=128, rk=18, rv=30, dr=64, Hr=16, n_max=512, p0=0,
             q=P, qr=P, ck=P, cv=P, rc=P, uk=P, uv=P, muk=None, muv=None, scale=0.088, out=P, stream=None)
    a.update(kw)
    return lla.lib().lla_prefill_attn_rope(a["dtype"], a["out_dtype"], a["B"], a["H"], a["M"], a["d"],
                                           a["rk"], a["rv"], a["dr"], a["Hr"], a["n_max"], a["p0"], a["q"],
                                           a["qr"], a["ck"], a["cv"], a["rc"], a["uk"], a["uv"], a["muk"],
                                           a["muv"], a["scale"], a["out"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(dr=0), 1), (dict(dr=20), 1), (dict(Hr=3), 1), (dict(qr=None), 1), (dict(rc=MIS), 1),
    (dict(M=0), 1), (dict(rk=32, dr=64), 2), (dict(rv=96), 2),
])
def test_prefill_rope_rejects(kw, code):
    assert _prefill_rope(**kw) == code


def _rope_write(**kw):
    a = dict(dtype=1, B=2, M=8, Hr=1, dr=64, x=P, base=10000.0, rc=P, n_max=512, pos0=0, stream=None)
    a.update(kw)
    return lla.lib().lla_rope_write(a["dtype"], a["B"], a["M"], a["Hr"], a["dr"], a["x"], a["base"], a["rc"],
                                    a["n_max"], a["pos0"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(dtype=2), dict(B=0), dict(M=0), dict(Hr=0), dict(dr=6), dict(dr=0), dict(x=None), dict(rc=MIS),
    dict(n_max=100), dict(pos0=-1), dict(pos0=505), dict(base=1.0), dict(base=float("nan")),
    dict(Hr=65536, M=1, B=1),
])
def test_rope_write_rejects(kw):
    assert _rope_write(**kw) == lla.LLA_ERR_INVALID_ARG


def _rope_rotate(**kw):
    a = dict(dtype=1, B=2, G=16, M=1, dr=64, x=P, pos=None, pos0=0, base=10000.0, y=P, stream=None)
    a.update(kw)
    return lla.lib().lla_rope_rotate(a["dtype"], a["B"], a["G"], a["M"], a["dr"], a["x"], a["pos"], a["pos0"],
                                     a["base"], a["y"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(dtype=5), dict(B=0), dict(G=0), dict(M=0), dict(dr=10), dict(x=None), dict(y=MIS),
    dict(pos=P + 2), dict(pos0=-3), dict(base=0.5), dict(G=65536),
])
def test_rope_rotate_rejects(kw):
    assert _rope_rotate(**kw) == lla.LLA_ERR_INVALID_ARG


# ---- eviction (ring slots) ----

def _encode_ring(**kw):
    a = dict(dtype=1, B=2, M=8, H=16, T=4, d=128, rk=18, rv=30, xk=P, xv=P, muk=None, muv=None, wk=P, wv=P,
             ck=P, cv=P, n_max=320, pos0=1000, sink=4, window=256, stream=None)
    a.update(kw)
    return lla.lib().lla_encode_ring(a["dtype"], a["B"], a["M"], a["H"], a["T"], a["d"], a["rk"], a["rv"],
                                     a["xk"], a["xv"], a["muk"], a["muv"], a["wk"], a["wv"], a["ck"], a["cv"],
                                     a["n_max"], a["pos0"], a["sink"], a["window"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(window=0), dict(window=-1), dict(sink=-1), dict(sink=100, window=256), dict(M=257),
    dict(pos0=-1), dict(n_max=256), dict(xk=None), dict(dtype=7),
    dict(pos0=0, M=261),  # 257 of the 261 positions would share 256 ring slots
])
def test_encode_ring_rejects(kw):
    assert _encode_ring(**kw) == lla.LLA_ERR_INVALID_ARG


def _rope_write_ring(**kw):
    a = dict(dtype=1, B=2, M=8, Hr=1, dr=64, x=P, base=10000.0, rc=P, n_max=320, pos0=1 << 20, sink=4,
             window=256, stream=None)
    a.update(kw)
    return lla.lib().lla_rope_write_ring(a["dtype"], a["B"], a["M"], a["Hr"], a["dr"], a["x"], a["base"],
                                         a["rc"], a["n_max"], a["pos0"], a["sink"], a["window"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(window=0), dict(sink=65, window=256), dict(M=300), dict(dr=12), dict(rc=None), dict(base=-2.0),
])
def test_rope_write_ring_rejects(kw):
    assert _rope_write_ring(**kw) == lla.LLA_ERR_INVALID_ARG


# ---- LLA-2D ----

def _decode_2d(**kw):
    a = dict(dtype=1, out_dtype=0, B=2, H=16, d=128, rk=288, rv=480, n_max=512, n_ctx=512, ctx_len=None,
             q=P, ck=P, cv=P, uk=P, uv=P, muk=None, muv=None, scale=0.088, out=P, ws=P, ws_bytes=1 << 30,
             stream=None)
    a.update(kw)
    return lla.lib().lla_decode_attn_2d(a["dtype"], a["out_dtype"], a["B"], a["H"], a["d"], a["rk"], a["rv"],
                                        a["n_max"], a["n_ctx"], a["ctx_len"], a["q"], a["ck"], a["cv"],
                                        a["uk"], a["uv"], a["muk"], a["muv"], a["scale"], a["out"], a["ws"],
                                        a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), 1), (dict(d=40), 1), (dict(n_ctx=0), 1), (dict(n_ctx=600), 1), (dict(q=None), 1),
    (dict(ck=MIS), 1), (dict(scale=0.0), 1), (dict(dtype=0), 2), (dict(H=8), 2), (dict(rk=300), 2),
    (dict(rv=490), 2), (dict(rk=1056), 2), (dict(ws=None, ws_bytes=0), 3), (dict(ws_bytes=64), 3),
    (dict(ws=MIS), 3), (dict(n_max=1 << 22), 2),
])
def test_decode_2d_rejects(kw, code):
    assert _decode_2d(**kw) == code


def test_decode_2d_workspace_grows_with_ranks():
    a = lla.decode_2d_workspace_bytes(32, 16, 288, 480, 4096)
    b = lla.decode_2d_workspace_bytes(32, 16, 576, 960, 4096)
    assert 0 < a < b


def _encode_2d(**kw):
    a = dict(dtype=1, B=2, M=8, H=16, T=4, d=128, rk=288, rv=480, xk=P, xv=P, muk=None, muv=None, wk=P,
             wv=P, ck=P, cv=P, n_max=512, pos0=0, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return lla.lib().lla_encode_2d(a["dtype"], a["B"], a["M"], a["H"], a["T"], a["d"], a["rk"], a["rv"],
                                   a["xk"], a["xv"], a["muk"], a["muv"], a["wk"], a["wv"], a["ck"], a["cv"],
                                   a["n_max"], a["pos0"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), 1), (dict(pos0=510), 1), (dict(xk=MIS), 1), (dict(n_max=500), 1), (dict(dtype=0), 2),
    (dict(rk=100), 2),
    (dict(B=32, M=1, ws=P, ws_bytes=16), 3), (dict(B=32, M=1, ws=MIS, ws_bytes=1 << 30), 3),
])
def test_encode_2d_rejects(kw, code):
    assert _encode_2d(**kw) == code


def test_encode_2d_workspace_only_for_split_writes():
    # a decode step's write (32 tokens, a 8192-value stack) is split; a prefill-sized one is not
    assert lla.encode_2d_workspace_bytes(32, 1, 16, 4, 128, 288, 480) > 0
    assert lla.encode_2d_workspace_bytes(4, 1024, 16, 4, 128, 288, 480) == 0
    assert lla.encode_2d_workspace_bytes(32, 1, 4, 1, 64, 288, 480) == 0  # stack of 256


# ---- full-RoPE reconstruct-then-attend decode ----

def _decode_fullrope(**kw):
    a = dict(dtype=1, out_dtype=0, B=2, H=16, d=128, rk=192, rv=320, n_max=512, n_ctx=512, ctx_len=None,
             q_pos=None, q=P, ck=P, cv=P, uk=P, uv=P, muk=None, muv=None, base=10000.0, scale=0.088, out=P,
             ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return lla.lib().lla_decode_attn_fullrope(a["dtype"], a["out_dtype"], a["B"], a["H"], a["d"], a["rk"],
                                              a["rv"], a["n_max"], a["n_ctx"], a["ctx_len"], a["q_pos"], a["q"],
                                              a["ck"], a["cv"], a["uk"], a["uv"], a["muk"], a["muv"], a["base"],
                                              a["scale"], a["out"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=2), 1), (dict(B=0), 1), (dict(d=48), 1), (dict(rk=0), 1), (dict(rv=513), 1),
    (dict(n_max=100), 1), (dict(n_ctx=0), 1), (dict(n_ctx=513), 1), (dict(scale=0.0), 1),
    (dict(base=1.0), 1), (dict(base=float("inf")), 1), (dict(q=None), 1), (dict(ck=MIS), 1),
    (dict(muk=MIS), 1), (dict(q_pos=P + 2), 1), (dict(ctx_len=P + 1), 1),
    (dict(ws=P, ws_bytes=0), 3), (dict(ws=P, ws_bytes=64), 3), (dict(ws=MIS, ws_bytes=1 << 30), 3),
    (dict(n_max=1 << 22), 2),
])
def test_decode_fullrope_rejects(kw, code):
    assert _decode_fullrope(**kw) == code


# ---- LLA-2D causal prefill ----

def test_prefill_2d_workspace_bytes():
    # rebuilt keys and values of every head, bf16: 4 * B * H * d * (n_keys rounded up to 64)
    assert lla.prefill_2d_workspace_bytes(4, 16, 128, 8192) == 4 * 4 * 16 * 128 * 8192
    assert lla.prefill_2d_workspace_bytes(1, 1, 128, 1) == 4 * 128 * 64
    assert lla.prefill_2d_workspace_bytes(2, 3, 128, 65) == 4 * 2 * 3 * 128 * 128


def _prefill_2d(**kw):
    a = dict(dtype=1, out_dtype=0, B=2, H=16, M=100, d=128, rk=288, rv=480, n_max=512, p0=0, q=P, ck=P, cv=P,
             uk=P, uv=P, muk=None, muv=None, scale=0.088, out=P, ws=P, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return lla.lib().lla_prefill_attn_2d(a["dtype"], a["out_dtype"], a["B"], a["H"], a["M"], a["d"], a["rk"],
                                         a["rv"], a["n_max"], a["p0"], a["q"], a["ck"], a["cv"], a["uk"], a["uv"],
                                         a["muk"], a["muv"], a["scale"], a["out"], a["ws"], a["ws_bytes"],
                                         a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=2), 1), (dict(B=0), 1), (dict(M=0), 1), (dict(d=48), 1), (dict(rk=0), 1),
    (dict(n_max=100), 1), (dict(p0=-1), 1), (dict(p0=413), 1), (dict(scale=float("nan")), 1),
    (dict(q=None), 1), (dict(cv=MIS), 1), (dict(muv=MIS), 1), (dict(B=65536, H=1, M=1), 1),
    (dict(dtype=0), 2), (dict(d=64), 2), (dict(rk=40), 2), (dict(rv=520), 2),
    (dict(ws=None), 3), (dict(ws_bytes=4 * 2 * 16 * 128 * 128 - 1), 3), (dict(ws=MIS), 3),
    (dict(n_max=1 << 22), 2),
])
def test_prefill_2d_rejects(kw, code):
    assert _prefill_2d(**kw) == code


def test_noalloc_scratch_bound_over_shapes():
    """The non-allocating decode needs (4 bytes per (b, h) rounded up to 256)
    plus 4 (r_v + 2) bytes per unit and split when the launch splits.  On a
    256-CU MI355X the shape heuristic splits only below 512 units, and takes
    at most 768 unit-slices (the bf16 4-page shapes below 256 units), so that
    stays below 1.6 MiB at r_v = 512, inside LLA_NOALLOC_SCRATCH_BYTES (4 MiB).
    Checked for every unit count that can split and page counts up to 4096."""
    import ctypes
    f, out = lla.lib().lla_decode_splits, ctypes.c_int()
    pages_set = list(range(1, 65)) + list(range(72, 4097, 8))
    worst, worst_slices = 0, 0
    for dt in (lla.LLA_BF16, lla.LLA_F32):
        for r_k, r_v in ((18, 30), (192, 320), (512, 512)):
            for units in range(1, 520):
                for p in pages_set:
                    assert f(dt, units, 1, p * 64, r_k, r_v, 0, 1, ctypes.byref(out)) == 0
                    s = out.value
                    if s > 1:
                        assert units < 512
                        worst_slices = max(worst_slices, units * s)
                        worst = max(worst, (units * 4 + 255) // 256 * 256 + units * s * (r_v + 2) * 4)
    assert worst_slices <= 768, worst_slices
    assert worst <= int(1.6 * 2**20) and worst <= 4 << 20, worst
