"""The C ABI library: it loads, exports every declared symbol, and its host-side
validation returns the documented status codes before touching the GPU."""
import ctypes
import math
import os
import re

import pytest

from paper_2607_08186_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hd.h")

FAKE = 0x10000  # aligned fake device addresses: validation fails before any use
INVALID, UNSUPPORTED = binding.HD_ERR_INVALID_ARG, binding.HD_ERR_UNSUPPORTED


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hd_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return binding.lib()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(binding.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code, name in [(0, "HD_OK"), (1, "HD_ERR_INVALID_ARG"), (2, "HD_ERR_UNSUPPORTED"),
                       (3, "HD_ERR_HIP")]:
        assert lib.hd_status_str(code).decode() == name


def fwd(lib, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=FAKE, B=1, L=8, n=2, Hq=4, Hkv=2, D=64,
             mode=0, scale=0.125, dtype=0)
    a.update(kw)
    return lib.hd_sfa_fwd(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["L"], a["n"],
                          a["Hq"], a["Hkv"], a["D"], a["mode"], a["scale"], a["dtype"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), INVALID), (dict(lse=None), INVALID), (dict(B=0), INVALID),
    (dict(L=-1), INVALID), (dict(n=0), INVALID), (dict(Hkv=3), INVALID),
    (dict(Hq=0), INVALID), (dict(scale=float("nan")), INVALID),
    (dict(scale=float("inf")), INVALID), (dict(scale=-0.1), INVALID), (dict(scale=0.0), INVALID),
    (dict(mode=2), INVALID), (dict(dtype=7), INVALID), (dict(D=96), UNSUPPORTED),
    (dict(D=256), UNSUPPORTED), (dict(q=FAKE + 8), INVALID), (dict(lse=FAKE + 4), INVALID),
    (dict(L=1 << 20, n=64, Hq=64), INVALID),  # per-batch slice beyond 2^31 bytes
])
def test_fwd_validation(lib, kw, code):
    assert fwd(lib, **kw) == code
    assert lib.hd_last_error().decode() != ""


def fwd_local(lib, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=FAKE, B=1, L=8, n=2, Hq=4, Hkv=2, D=64,
             window=5, scale=0.125, dtype=0)
    a.update(kw)
    return lib.hd_sfa_fwd_local(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["L"],
                                a["n"], a["Hq"], a["Hkv"], a["D"], a["window"], a["scale"],
                                a["dtype"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(window=0), INVALID), (dict(window=-3), INVALID), (dict(q=None), INVALID),
    (dict(Hkv=3), INVALID), (dict(scale=0.0), INVALID), (dict(D=96), UNSUPPORTED),
    (dict(o=FAKE + 8), INVALID), (dict(dtype=4), INVALID),
])
def test_fwd_local_validation(lib, kw, code):
    assert fwd_local(lib, **kw) == code
    assert lib.hd_last_error().decode() != ""


def test_local_mode_needs_local_entry_points(lib):
    """A local layer without a window is an error, not a silent full causal layer."""
    assert fwd(lib, mode=binding.HD_SFA_LOCAL) == INVALID
    assert "hd_sfa_fwd_local" in lib.hd_last_error().decode()
    st, _ = bwd(lib, mode=binding.HD_SFA_LOCAL)
    assert st == INVALID
    assert "hd_sfa_bwd_local" in lib.hd_last_error().decode()


def bwd(lib, ws_bytes=None, ws=FAKE * 16, **kw):
    a = dict(B=1, L=8, n=2, Hq=4, Hkv=2, D=64, mode=1, scale=0.125, dtype=0)
    a.update(kw)
    need = lib.hd_sfa_bwd_workspace_bytes(a["B"], a["L"], a["n"], a["Hq"], a["Hkv"], a["D"],
                                          a["mode"], a["dtype"])
    ptrs = [FAKE] * 9
    for i, name in enumerate(["q", "k", "v", "o", "lse", "dO", "dq", "dk", "dv"]):
        if name in kw:
            ptrs[i] = kw[name]
    return lib.hd_sfa_bwd(*ptrs, a["B"], a["L"], a["n"], a["Hq"], a["Hkv"], a["D"], a["mode"],
                          a["scale"], a["dtype"], ws, need if ws_bytes is None else ws_bytes,
                          None), need


def _ds_tiles(len_, window=None):
    """dS tiles (64 query rows x 128 keys, 16 KB) stored per causal problem: those that
    hold a visible pair, counted by brute force over the tiles' pairs."""
    nqt, nkt = -(-len_ // 64), -(-len_ // 128)
    w = window if window is not None else len_
    count = 0
    for qt in range(nqt):
        rows = range(qt * 64, min(len_, qt * 64 + 64))
        per_row = 0
        for kt in range(nkt):
            k_lo, k_hi = kt * 128, min(len_, kt * 128 + 128) - 1
            if any(k_lo <= r and r - k_hi < w for r in rows):
                per_row += 1
        count += per_row
    return count


def test_workspace_size_formula(lib):
    a256 = lambda x: math.ceil(x / 256) * 256
    B, L, n, Hq, Hkv, D = 2, 100, 3, 4, 2, 64
    rows = B * Hq * n * L
    stats = 2 * a256(rows * 4)  # delta and lse2, fp32 per query row
    # fp32: statistics only
    assert lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, 0, 1) == stats
    # bf16 adds the dS tiles of every problem: exactly the tiles holding a visible pair
    # for causal layers (intra: one problem per stream)
    for mode, len_, streams in ((0, L, n), (1, n * L, 1)):
        ds = B * Hq * streams * _ds_tiles(len_) * 16384
        assert lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, mode, 0) == stats + ds
    for dtype in (0, 1):  # without a window a local layer gets the full causal size
        assert (lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, 2, dtype)
                == lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, 1, dtype))
    assert lib.hd_sfa_bwd_workspace_bytes(1, 8, 2, 4, 2, 64, 3, 0) == 0  # mode
    assert lib.hd_sfa_bwd_workspace_bytes(1, 8, 2, 4, 3, 64, 0, 0) == 0  # Hq % Hkv
    assert lib.hd_sfa_bwd_workspace_bytes(1, 8, 2, 4, 2, 48, 0, 0) == 0  # D


def _sweep(len_, kt):
    """64-row query tiles [first, end) of a causal problem (no window) with a row that
    sees a key of 128-key tile kt."""
    return kt * 128 // 64, -(-len_ // 64)


def test_split_sweep_workspace(lib):
    """Small dK/dV grids (under 512 workgroups) with at least four key tiles split the
    sweeps longer than half the longest one; the one-pass workspace then also holds
    their two halves' fp32 partials: 4 x key problems x split keys x D floats."""
    a256 = lambda x: math.ceil(x / 256) * 256
    for B, L, n, Hq, Hkv, D, mode in ((2, 2048, 1, 32, 8, 128, 0), (1, 1000, 1, 2, 2, 64, 1),
                                      (1, 2000, 2, 8, 1, 64, 0), (1, 4096, 4, 32, 8, 128, 0)):
        len_, streams = (L, n) if mode == 0 else (n * L, 1)
        nkt = -(-len_ // 128)
        kprobs = B * Hkv * streams
        lens = [e - f for f, e in (_sweep(len_, kt) for kt in range(nkt))]
        ns = 0
        if nkt >= 4 and nkt * kprobs < 512:
            while ns < nkt and 2 * lens[ns] > max(lens) and lens[ns] >= 2:
                ns += 1
        stats = 2 * a256(B * Hq * n * L * 4)
        ds = B * Hq * streams * _ds_tiles(len_) * 16384
        want = stats + ds + 4 * kprobs * ns * 128 * D * 4
        assert lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, mode, 0) == want, (B, L, n, mode, ns)
        if (B, L, n) == (2, 2048, 1):
            assert ns == 8  # the n=1 sweep shape: key tiles 0..7 of 16


def _ds_tiles_of_query_tiles(len_, qts):
    """dS tiles holding a visible pair of a causal problem (no window), for the listed
    64-row query tiles, by brute force over the tiles' pairs."""
    nkt = -(-len_ // 128)
    count = 0
    for qt in qts:
        rows = range(qt * 64, min(len_, qt * 64 + 64))
        count += sum(1 for kt in range(nkt) if any(kt * 128 <= r for r in rows))
    return count


@pytest.mark.parametrize("B,L,n,Hq,Hkv,D", [(2, 100, 3, 4, 2, 64), (1, 4096, 4, 32, 8, 128),
                                            (1, 700, 1, 2, 1, 32)])
def test_min_workspace_size_formula(lib, B, L, n, Hq, Hkv, D):
    """The smallest bf16 workspace: the row statistics, fp32 dK/dV partials and the dS
    tiles of the largest 256-row band unit (four 64-row query tiles)."""
    a256 = lambda x: math.ceil(x / 256) * 256
    N = n * L
    stats = 2 * a256(B * Hq * N * 4)
    parts = 2 * a256(B * N * Hkv * D * 4)
    for mode, len_, streams in ((0, L, n), (1, N, 1)):
        nqt = -(-len_ // 64)
        unit = max(_ds_tiles_of_query_tiles(len_, range(qa, min(nqt, qa + 4)))
                   for qa in range(0, nqt, 4))
        full = lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, mode, 0)
        want = min(full, stats + parts + B * Hq * streams * unit * 16384)
        assert lib.hd_sfa_bwd_min_workspace_bytes(B, L, n, Hq, Hkv, D, mode, 0) == want
        # fp32 keeps no dS tiles: one size
        assert (lib.hd_sfa_bwd_min_workspace_bytes(B, L, n, Hq, Hkv, D, mode, 1)
                == lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, mode, 1))
    # local layers: never above the one-pass size; at least statistics and partials
    for w in (1, 300, 10 ** 6):
        full = lib.hd_sfa_bwd_local_workspace_bytes(B, L, n, Hq, Hkv, D, w, 0)
        got = lib.hd_sfa_bwd_local_min_workspace_bytes(B, L, n, Hq, Hkv, D, w, 0)
        assert got <= full and (got == full or got > stats + parts)
    assert lib.hd_sfa_bwd_min_workspace_bytes(1, 8, 2, 4, 3, 64, 0, 0) == 0  # Hq % Hkv
    assert lib.hd_sfa_bwd_local_min_workspace_bytes(B, L, n, Hq, Hkv, D, 0, 0) == 0
    assert lib.hd_sfa_bwd_final_min_workspace_bytes(B, L, n, Hq, Hkv, D, -1, 0) == 0


def test_min_workspace_at_the_long_forward_limit(lib):
    """At B=1, N=131008, Hq=64, Hkv=8, D=128 the one-pass dS tiles take about a
    terabyte; the banded backward runs from a few gigabytes up."""
    for mode, (L, n) in ((0, (32752, 4)), (1, (32752, 4))):
        full = lib.hd_sfa_bwd_workspace_bytes(1, L, n, 64, 8, 128, mode, 0)
        low = lib.hd_sfa_bwd_min_workspace_bytes(1, L, n, 64, 8, 128, mode, 0)
        assert full > 2 * 10 ** 11 and 0 < low < 8 * 2 ** 30, (mode, full, low)


def test_short_workspace_is_rejected_below_the_minimum(lib):
    a = dict(B=1, L=300, n=4, Hq=4, Hkv=2, D=64, mode=1, dtype=0)
    low = lib.hd_sfa_bwd_min_workspace_bytes(a["B"], a["L"], a["n"], a["Hq"], a["Hkv"], a["D"],
                                             a["mode"], a["dtype"])
    full = lib.hd_sfa_bwd_workspace_bytes(a["B"], a["L"], a["n"], a["Hq"], a["Hkv"], a["D"],
                                          a["mode"], a["dtype"])
    assert 0 < low < full
    st, _ = bwd(lib, ws_bytes=low - 1, **a)
    assert st == INVALID
    assert "short" in lib.hd_last_error().decode()


@pytest.mark.parametrize("L,n,window", [(100, 3, 1), (100, 3, 64), (100, 3, 129), (100, 3, 299),
                                        (100, 3, 300), (100, 3, 10 ** 6), (700, 4, 200),
                                        (700, 4, 1000), (2048, 2, 4096)])
def test_local_workspace_size(lib, L, n, window):
    B, Hq, Hkv, D = 1, 2, 1, 32
    full = lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, 1, 0)
    got = lib.hd_sfa_bwd_local_workspace_bytes(B, L, n, Hq, Hkv, D, window, 0)
    # never more than the window-free size, and never less than the tiles holding a
    # visible pair of this window
    stats = lib.hd_sfa_bwd_workspace_bytes(B, L, n, Hq, Hkv, D, 1, 1)
    assert stats + B * Hq * _ds_tiles(n * L, window) * 16384 <= got <= full
    if window >= n * L:
        assert got == full
    assert lib.hd_sfa_bwd_local_workspace_bytes(B, L, n, Hq, Hkv, D, 0, 0) == 0
    assert (lib.hd_sfa_bwd_local_workspace_bytes(B, L, n, Hq, Hkv, D, window, 1)
            == stats)


@pytest.mark.parametrize("kw,code", [
    (dict(dq=None), INVALID), (dict(dO=None), INVALID), (dict(ws=None), INVALID),
    (dict(ws=FAKE * 16 + 16), INVALID), (dict(ws_bytes=16), INVALID), (dict(D=48), UNSUPPORTED),
    (dict(dk=FAKE + 2), INVALID), (dict(Hkv=0), INVALID),
])
def test_bwd_validation(lib, kw, code):
    st, _ = bwd(lib, **kw)
    assert st == code


@pytest.mark.parametrize("kw,code", [
    (dict(window=0), INVALID), (dict(dv=None), INVALID), (dict(ws=None), INVALID),
    (dict(ws_bytes=16), INVALID), (dict(D=48), UNSUPPORTED), (dict(dq=FAKE + 2), INVALID),
])
def test_bwd_local_validation(lib, kw, code):
    a = dict(B=1, L=8, n=2, Hq=4, Hkv=2, D=64, window=5, scale=0.125, dtype=0, ws=FAKE * 16)
    a.update(kw)
    need = lib.hd_sfa_bwd_workspace_bytes(a["B"], a["L"], a["n"], a["Hq"], a["Hkv"], a["D"],
                                          binding.HD_SFA_LOCAL, a["dtype"])
    ptrs = [kw.get(name, FAKE) for name in ["q", "k", "v", "o", "lse", "dO", "dq", "dk", "dv"]]
    st = lib.hd_sfa_bwd_local(*ptrs, a["B"], a["L"], a["n"], a["Hq"], a["Hkv"], a["D"],
                              a["window"], a["scale"], a["dtype"], a["ws"],
                              kw.get("ws_bytes", need), None)
    assert st == code
    assert lib.hd_last_error().decode() != ""


@pytest.mark.parametrize("args,code", [
    (dict(ids=None), INVALID), (dict(B=0), INVALID), (dict(V=0), INVALID),
    (dict(V=1 << 40), INVALID), (dict(Dm=0), INVALID), (dict(dtype=5), INVALID),
    (dict(out=FAKE + 8), INVALID), (dict(bad=FAKE + 2), INVALID),
    (dict(n=1 << 16, Dm=1 << 15), INVALID),  # a token's rows would exceed 2^31 bytes
])
def test_expand_validation(lib, args, code):
    a = dict(ids=FAKE, tables=FAKE, out=FAKE, B=1, L=4, n=2, V=10, Dm=8, dtype=0, bad=None)
    a.update(args)
    st = lib.hd_expand_embed(a["ids"], a["tables"], a["out"], a["B"], a["L"], a["n"], a["V"],
                             a["Dm"], a["dtype"], a["bad"], None)
    assert st == code


@pytest.mark.parametrize("args,code", [
    (dict(ids=None), INVALID), (dict(drows=None), INVALID), (dict(num=None), INVALID),
    (dict(B=0), INVALID), (dict(n=0), INVALID), (dict(V=0), INVALID), (dict(V=1 << 40), INVALID),
    (dict(Dm=0), INVALID), (dict(dtype=7), INVALID), (dict(L=4194305), INVALID),
    (dict(dout=FAKE + 8), INVALID), (dict(drows=FAKE + 4), INVALID), (dict(uniq=FAKE + 2), INVALID),
    (dict(ws=None), INVALID), (dict(ws=FAKE + 128), INVALID), (dict(ws_bytes=100), INVALID),
])
def test_expand_bwd_validation(lib, args, code):
    a = dict(ids=FAKE, dout=FAKE, B=1, L=4, n=2, V=10, Dm=8, dtype=0, uniq=FAKE, drows=FAKE,
             num=FAKE, ws=FAKE)
    a.update(args)
    need = lib.hd_expand_embed_bwd_workspace_bytes(1, 4)
    st = lib.hd_expand_embed_bwd(a["ids"], a["dout"], a["B"], a["L"], a["n"], a["V"], a["Dm"],
                                 a["dtype"], a["uniq"], a["drows"], a["num"], a["ws"],
                                 a.get("ws_bytes", need), None)
    assert st == code
    assert lib.hd_last_error().decode() != ""


def test_expand_bwd_workspace_size(lib):
    """Sort buffers (4 x 4 bytes per token), histograms, scan sums, segment indices and
    starts; 0 for sizes the entry point rejects."""
    assert lib.hd_expand_embed_bwd_workspace_bytes(0, 5) == 0
    assert lib.hd_expand_embed_bwd_workspace_bytes(1, 4194305) == 0
    for B, L in [(1, 1), (1, 4096), (2, 2049), (1, 4194304)]:
        M = B * L
        got = lib.hd_expand_embed_bwd_workspace_bytes(B, L)
        assert got >= 6 * 4 * M + 4 and got < 6 * 4 * M + 256 * 4 * (M // 2048 + 1) + 16384
        assert got % 256 == 0


@pytest.mark.parametrize("args,code", [
    (dict(uniq=None), INVALID), (dict(dtables=None), INVALID), (dict(rows=0), INVALID),
    (dict(n=0), INVALID), (dict(V=0), INVALID), (dict(Dm=-1), INVALID), (dict(drows=FAKE + 2), INVALID),
])
def test_grad_scatter_add_validation(lib, args, code):
    a = dict(uniq=FAKE, drows=FAKE, num=FAKE, rows=4, n=2, V=10, Dm=8, dtables=FAKE)
    a.update(args)
    st = lib.hd_embed_grad_scatter_add(a["uniq"], a["drows"], a["num"], a["rows"], a["n"],
                                       a["V"], a["Dm"], a["dtables"], None)
    assert st == code


@pytest.mark.parametrize("args,code", [
    (dict(src=None), INVALID), (dict(n=0), INVALID), (dict(m=3), INVALID), (dict(m=1), INVALID),
    (dict(V=0), INVALID), (dict(dtype=9), INVALID), (dict(dst=FAKE + 8), INVALID),
    (dict(dst=FAKE + 8192), INVALID),  # one 8 KB table past src: overlaps without aliasing
])
def test_cyclic_replicate_validation(lib, args, code):
    a = dict(src=FAKE, dst=FAKE + (1 << 30), n=2, m=4, V=64, Dm=64, dtype=0)
    a.update(args)
    st = lib.hd_cyclic_replicate(a["src"], a["dst"], a["n"], a["m"], a["V"], a["Dm"], a["dtype"],
                                 None)
    assert st == code


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), INVALID), (dict(window=-1), INVALID), (dict(dtype=1), UNSUPPORTED),
    (dict(n=64), UNSUPPORTED), (dict(D=48), UNSUPPORTED), (dict(Hkv=3), INVALID),
])
def test_final_validation(lib, kw, code):
    a = dict(q=FAKE, B=1, L=8, n=2, Hq=4, Hkv=2, D=64, window=0, scale=0.125, dtype=0)
    a.update(kw)
    st = lib.hd_sfa_fwd_final(a["q"], FAKE, FAKE, FAKE, FAKE, a["B"], a["L"], a["n"], a["Hq"],
                              a["Hkv"], a["D"], a["window"], a["scale"], a["dtype"], None)
    assert st == code
    need = lib.hd_sfa_bwd_final_workspace_bytes(a["B"], a["L"], a["n"], a["Hq"], a["Hkv"], a["D"],
                                                a["window"], a["dtype"])
    if a["q"] is not None:  # size and dtype errors make the workspace query return 0
        assert (need == 0) == (code != 0)
    st = lib.hd_sfa_bwd_final(a["q"], FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, a["B"],
                              a["L"], a["n"], a["Hq"], a["Hkv"], a["D"], a["window"], a["scale"],
                              a["dtype"], FAKE, max(need, 1 << 30), None)
    assert st == code


def test_final_workspace_sizes(lib):
    """Row statistics per final-stream query row, plus bf16 dS tiles of 16 KB per 64
    query rows x 128 keys: every key tile without a window, a band of
    (w + 63 n - 1)/128 + 1 key tiles with one."""
    B, L, n, Hq, Hkv, D = 1, 4096, 4, 32, 8, 128
    stats = 2 * ((B * Hq * L * 4 + 255) // 256 * 256)
    nqt, nkt = L // 64, n * L // 128
    full = lib.hd_sfa_bwd_final_workspace_bytes(B, L, n, Hq, Hkv, D, 0, 0)
    assert full == stats + B * Hq * nqt * nkt * 16384
    w = 4096
    band = (w + 63 * n - 1 + 127) // 128 + 1
    local = lib.hd_sfa_bwd_final_workspace_bytes(B, L, n, Hq, Hkv, D, w, 0)
    assert local == stats + B * Hq * nqt * band * 16384


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), INVALID), (dict(ctx=None), INVALID), (dict(B=0), INVALID),
    (dict(Hkv=3), INVALID), (dict(mode=7), INVALID), (dict(mode=2, window=0), INVALID),
    (dict(max_ctx=16), INVALID), (dict(max_ctx=-1), INVALID), (dict(scale=0.0), INVALID),
    (dict(dtype=1), UNSUPPORTED), (dict(D=96), UNSUPPORTED), (dict(o=FAKE + 8), INVALID),
    (dict(ctx=FAKE + 2), INVALID), (dict(ws=None), INVALID), (dict(ws=FAKE + 64), INVALID),
    (dict(ws_bytes=10), INVALID),
])
def test_decode_validation(lib, kw, code):
    a = dict(q=FAKE, ctx=FAKE, o=FAKE, B=2, Lcap=16, n=4, Hq=8, Hkv=2, D=64, mode=1, window=0,
             max_ctx=10, scale=0.125, dtype=0, ws=FAKE)
    a.update(kw)
    need = lib.hd_sfa_decode_workspace_bytes(2, 16, 4, 8, 2, 64, 1, 0, 10)
    st = lib.hd_sfa_decode(a["q"], FAKE, FAKE, a["ctx"], a["max_ctx"], a["o"], FAKE, a["B"],
                           a["Lcap"], a["n"], a["Hq"], a["Hkv"], a["D"], a["mode"], a["window"],
                           a["scale"], a["dtype"], a["ws"], a.get("ws_bytes", need), None)
    assert st == code
    assert lib.hd_last_error().decode() != ""


def test_decode_workspace_size(lib):
    """fp32 partials (D sums, max and sum per query slot of the problem) per 256 cached
    rows of every problem: (b, kv head, head chunk[, stream]); a problem's slots are its
    heads (intra-stream) or its heads times the n streams, at most 32."""
    B, Lcap, n, Hq, Hkv, D = 2, 5000, 4, 32, 8, 128
    rows = 4096 * n  # max_ctx + 1 = 4096 tokens
    mix = lib.hd_sfa_decode_workspace_bytes(B, Lcap, n, Hq, Hkv, D, 1, 0, 4095)
    # G*n = 16 slots: one head chunk
    assert mix == B * Hkv * 1 * (rows // 256) * 16 * (D + 2) * 4
    intra = lib.hd_sfa_decode_workspace_bytes(B, Lcap, n, Hq, Hkv, D, 0, 0, 4095)
    assert intra == B * Hkv * n * (4096 // 256) * 4 * (D + 2) * 4  # G = 4 slots per stream
    wide = lib.hd_sfa_decode_workspace_bytes(1, 100, 8, 64, 4, 64, 1, 0, 99)  # G*n = 128 slots
    assert wide == 1 * 4 * 4 * ((100 * 8 + 255) // 256) * 32 * 66 * 4
    assert lib.hd_sfa_decode_workspace_bytes(B, Lcap, n, Hq, Hkv, D, 1, 0, Lcap) == 0


def _decode_noalloc(lib, **kw):
    a = dict(q=FAKE, ctx=FAKE, o=FAKE, B=2, Lcap=16, n=4, Hq=8, Hkv=2, D=64, mode=1, window=0,
             max_ctx=10, scale=0.125, dtype=0)
    a.update(kw)
    return lib.hd_sfa_decode_noalloc(a["q"], FAKE, FAKE, a["ctx"], a["max_ctx"], a["o"], FAKE,
                                     a["B"], a["Lcap"], a["n"], a["Hq"], a["Hkv"], a["D"],
                                     a["mode"], a["window"], a["scale"], a["dtype"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), INVALID), (dict(ctx=None), INVALID), (dict(B=0), INVALID),
    (dict(Hkv=3), INVALID), (dict(mode=7), INVALID), (dict(mode=2, window=0), INVALID),
    (dict(max_ctx=16), INVALID), (dict(scale=0.0), INVALID), (dict(dtype=1), UNSUPPORTED),
    (dict(D=96), UNSUPPORTED), (dict(o=FAKE + 8), INVALID), (dict(ctx=FAKE + 2), INVALID),
    # 32 sequences x 4096 tokens, n=4, 32/8 heads of width 128: 136 MB of partials
    (dict(B=32, Lcap=4096, n=4, Hq=32, Hkv=8, D=128, max_ctx=4095), INVALID),
])
def test_decode_noalloc_validation(lib, kw, code):
    """The allocation-free decode validates like hd_sfa_decode and rejects sizes whose
    partials exceed its scratch, all before touching the GPU."""
    assert _decode_noalloc(lib, **kw) == code
    assert lib.hd_last_error().decode() != ""


def test_decode_noalloc_limit(lib):
    """128 MiB of scratch: the 16-sequence, 4096-token serving shape of every mode fits
    (65 MiB of partials for a full cross-stream layer), twice that does not."""
    limit = binding.hd_sfa_decode_noalloc_max_bytes()
    assert limit == 128 << 20
    for mode, window in ((0, 0), (1, 0), (2, 4096)):
        need = lib.hd_sfa_decode_workspace_bytes(16, 4096, 4, 32, 8, 128, mode, window, 4095)
        assert 0 < need <= limit
    assert lib.hd_sfa_decode_workspace_bytes(32, 4096, 4, 32, 8, 128, 1, 0, 4095) > limit


def test_missing_library_raises(monkeypatch, tmp_path):
    """No silent fallback: a missing libhd.so is an ImportError on first use."""
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "libhd.so"))
    with pytest.raises(ImportError):
        binding.lib()


def test_timing_collect_empty(lib):
    assert binding.hd_timing_collect() == []


def test_timing_filter_set_and_reset(lib):
    assert lib.hd_timing_filter(b"sfa_dkdv") == 0
    assert lib.hd_timing_filter(None) == 0
    binding.hd_timing_filter("sfa_fwd")
    binding.hd_timing_filter(None)
    assert binding.hd_timing_collect() == []


# h at FAKE is [B][n*L][Dm] = 2*3*5*8 bf16 = 480 bytes; out [B][L][Dm] = 160 bytes
@pytest.mark.parametrize("args,code", [
    (dict(src=None), INVALID), (dict(dst=None), INVALID), (dict(B=0), INVALID),
    (dict(L=-1), INVALID), (dict(n=0), INVALID), (dict(Dm=0), INVALID), (dict(dtype=7), INVALID),
    (dict(src=FAKE + 4), INVALID), (dict(dst=FAKE + (1 << 20) + 8), INVALID),
    (dict(dst=FAKE + 464), INVALID),      # overlaps the end of the larger buffer
    (dict(dst=FAKE - 144), INVALID),      # the smaller buffer ends inside the larger one
    (dict(B=1 << 16, L=1 << 16), INVALID),  # B*n*L beyond int32
])
@pytest.mark.parametrize("backward", [False, True])
def test_final_stream_gather_validation(lib, args, code, backward):
    a = dict(src=FAKE, dst=FAKE + (1 << 20), B=2, L=5, n=3, Dm=8, dtype=0)
    a.update(args)
    if backward:  # src is dout (small), dst is dh (large): mirror the overlap cases
        if "dst" in args and args["dst"] is not None and args["dst"] != FAKE + (1 << 20) + 8:
            a["src"], a["dst"] = a["dst"], FAKE
        st = lib.hd_final_stream_gather_bwd(a["src"], a["dst"], a["B"], a["L"], a["n"], a["Dm"],
                                            a["dtype"], None)
    else:
        st = lib.hd_final_stream_gather(a["src"], a["dst"], a["B"], a["L"], a["n"], a["Dm"],
                                        a["dtype"], None)
    assert st == code


def test_binding_rejects_host_and_strided_tensors(lib):
    """Host tensors would hand the kernels host addresses, strided views a layout they do
    not read: both are refused in the binding before any call."""
    import torch

    q = torch.zeros((1, 8, 2, 32), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU"):
        binding.hd_sfa_fwd(q, q, q, q, q, 1, 4, 2, 2, 2, 32, 0, 0.125)
    with pytest.raises(ValueError, match="GPU"):
        binding.final_stream_gather(torch.zeros((1, 8, 16)), 2)
    with pytest.raises(ValueError, match="GPU"):
        binding.expand_embed(torch.zeros((1, 4), dtype=torch.int32), torch.zeros((2, 5, 8)))
