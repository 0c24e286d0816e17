"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

None of these re-types the oracle's formulas.  Each check uses an independent
statement of the result: torch's fp64 scaled_dot_product_attention (a library routine)
on de-interleaved or expanded sequences, closed forms, invariants, hand-written
golden fixtures and central finite differences.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from paper_2607_08186_amd import synth

INTRA, MIX, LOCAL = 0, 1, 2
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(seed, B, L, n, Hq, Hkv, D, std=1.0):
    N = n * L
    r = np.random.default_rng(seed)
    q = r.standard_normal((B, N, Hq, D)) * std
    k = r.standard_normal((B, N, Hkv, D)) * std
    v = r.standard_normal((B, N, Hkv, D))
    do = r.standard_normal((B, N, Hq, D))
    return q, k, v, do


def _torch_causal(q, k, v, do, scale):
    """Library causal attention on [B][S][H][D] fp64 arrays with GQA by head repeat.

    Returns o [B][S][Hq][D], lse [B][Hq][S], dq, dk, dv (dk/dv summed over groups).
    """
    Hq, Hkv = q.shape[2], k.shape[2]
    G = Hq // Hkv
    tq = torch.tensor(q).permute(0, 2, 1, 3).contiguous().requires_grad_(True)
    tk = torch.tensor(k).permute(0, 2, 1, 3).contiguous().requires_grad_(True)
    tv = torch.tensor(v).permute(0, 2, 1, 3).contiguous().requires_grad_(True)
    kk = tk.repeat_interleave(G, dim=1)
    vv = tv.repeat_interleave(G, dim=1)
    o = F.scaled_dot_product_attention(tq, kk, vv, is_causal=True, scale=scale)
    o.backward(torch.tensor(do).permute(0, 2, 1, 3))
    S = q.shape[1]
    logits = scale * torch.matmul(tq.detach(), kk.detach().transpose(-1, -2))
    keep = torch.ones(S, S, dtype=torch.bool).tril()
    lse = torch.logsumexp(logits.masked_fill(~keep, float("-inf")), dim=-1)
    back = lambda t: t.permute(0, 2, 1, 3).detach().numpy()
    return back(o), lse.numpy(), back(tq.grad), back(tk.grad), back(tv.grad)


def _deinterleave(x, n, s):
    B, N, H, D = x.shape
    return x.reshape(B, N // n, n, H, D)[:, :, s]


SHAPES = [  # B, L, n, Hq, Hkv, D
    (1, 7, 3, 2, 1, 4),
    (2, 5, 2, 4, 2, 8),
    (1, 6, 4, 3, 3, 5),
    (1, 9, 1, 2, 2, 6),
]


@pytest.mark.parametrize("shape", SHAPES)
def test_intra_equals_causal_per_stream(oracle_mod, shape):
    """INTRA(n) == ordinary causal attention on each de-interleaved stream (fwd + bwd)."""
    B, L, n, Hq, Hkv, D = shape
    q, k, v, do = _rand(1, *shape)
    scale = 1.0 / math.sqrt(D)
    o, lse = oracle_mod.sfa_fwd(q, k, v, L=L, n=n, mode=INTRA, scale=scale)
    dq, dk, dv = oracle_mod.sfa_bwd(q, k, v, do, L=L, n=n, mode=INTRA, scale=scale)
    for s in range(n):
        ro, rlse, rdq, rdk, rdv = _torch_causal(*(_deinterleave(x, n, s) for x in (q, k, v, do)),
                                                scale)
        np.testing.assert_allclose(_deinterleave(o, n, s), ro, atol=1e-12, rtol=0)
        np.testing.assert_allclose(lse[:, :, s::n], rlse, atol=1e-12, rtol=0)
        np.testing.assert_allclose(_deinterleave(dq, n, s), rdq, atol=1e-11, rtol=0)
        np.testing.assert_allclose(_deinterleave(dk, n, s), rdk, atol=1e-11, rtol=0)
        np.testing.assert_allclose(_deinterleave(dv, n, s), rdv, atol=1e-11, rtol=0)


@pytest.mark.parametrize("shape", SHAPES)
def test_mix_equals_causal_over_expanded(oracle_mod, shape):
    """MIX(n) == ordinary causal attention over all n*L expanded rows, for every n."""
    B, L, n, Hq, Hkv, D = shape
    q, k, v, do = _rand(2, *shape)
    scale = 1.0 / math.sqrt(D)
    o, lse = oracle_mod.sfa_fwd(q, k, v, L=L, n=n, mode=MIX, scale=scale)
    dq, dk, dv = oracle_mod.sfa_bwd(q, k, v, do, L=L, n=n, mode=MIX, scale=scale)
    ro, rlse, rdq, rdk, rdv = _torch_causal(q, k, v, do, scale)
    np.testing.assert_allclose(o, ro, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, rlse, atol=1e-12, rtol=0)
    np.testing.assert_allclose(dq, rdq, atol=1e-11, rtol=0)
    np.testing.assert_allclose(dk, rdk, atol=1e-11, rtol=0)
    np.testing.assert_allclose(dv, rdv, atol=1e-11, rtol=0)


def test_n1_modes_coincide(oracle_mod):
    """With one stream the two masks are the same causal mask."""
    q, k, v, do = _rand(3, 1, 11, 1, 2, 1, 8)
    a = oracle_mod.sfa_fwd(q, k, v, L=11, n=1, mode=INTRA, scale=0.3)
    b = oracle_mod.sfa_fwd(q, k, v, L=11, n=1, mode=MIX, scale=0.3)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_masks_match_hand_written_golden(oracle_mod):
    lines = [ln.strip() for ln in open(os.path.join(GOLDEN, "masks_n2_L3.txt"))
             if ln.strip() and not ln.startswith("#")]
    want = {}
    cur = None
    for ln in lines:
        if ln in ("intra", "mix", "local3"):
            cur = ln
            want[cur] = []
        else:
            want[cur].append([int(c) for c in ln])
    np.testing.assert_array_equal(oracle_mod.sfa_mask(3, 2, INTRA), np.array(want["intra"]))
    np.testing.assert_array_equal(oracle_mod.sfa_mask(3, 2, MIX), np.array(want["mix"]))
    np.testing.assert_array_equal(oracle_mod.sfa_mask(3, 2, LOCAL, 3), np.array(want["local3"]))


@pytest.mark.parametrize("L,n", [(5, 3), (16, 4), (7, 1), (4, 8)])
def test_mask_is_progression_or_prefix(oracle_mod, L, n):
    """INTRA row p sees exactly range(p % n, p + 1, n); MIX row p sees range(0, p + 1)."""
    N = n * L
    mi = oracle_mod.sfa_mask(L, n, INTRA)
    mm = oracle_mod.sfa_mask(L, n, MIX)
    for p in range(N):
        want_i = np.zeros(N, np.uint8)
        want_i[list(range(p % n, p + 1, n))] = 1
        want_m = np.zeros(N, np.uint8)
        want_m[: p + 1] = 1
        np.testing.assert_array_equal(mi[p], want_i)
        np.testing.assert_array_equal(mm[p], want_m)


def test_rows_sum_to_one_via_constant_values(oracle_mod):
    """With every V entry equal to 1, O is exactly the row sum of P, which must be 1."""
    q, k, v, _ = _rand(4, 2, 6, 3, 4, 2, 5)
    v = np.ones_like(v)
    for mode in (INTRA, MIX):
        o, _ = oracle_mod.sfa_fwd(q, k, v, L=6, n=3, mode=mode, scale=0.7)
        np.testing.assert_allclose(o, 1.0, atol=1e-12, rtol=0)


@pytest.mark.parametrize("mode", [INTRA, MIX])
def test_first_token_rows_closed_form(oracle_mod, mode):
    """A row that sees only itself copies its own v, lse = scale q.k, and dQ = 0."""
    B, L, n, Hq, Hkv, D = 1, 6, 4, 4, 2, 8
    q, k, v, do = _rand(5, B, L, n, Hq, Hkv, D)
    scale = 0.37
    o, lse = oracle_mod.sfa_fwd(q, k, v, L=L, n=n, mode=mode, scale=scale)
    dq, _, _ = oracle_mod.sfa_bwd(q, k, v, do, L=L, n=n, mode=mode, scale=scale)
    rows = range(n) if mode == INTRA else range(1)
    for p in rows:
        for h in range(Hq):
            hk = h // (Hq // Hkv)
            np.testing.assert_allclose(o[0, p, h], v[0, p, hk], atol=1e-14, rtol=0)
            assert abs(lse[0, h, p] - scale * float(q[0, p, h] @ k[0, p, hk])) < 1e-13
            np.testing.assert_allclose(dq[0, p, h], 0.0, atol=1e-15)


@pytest.mark.parametrize("mode", [INTRA, MIX])
def test_uniform_logit_probe(oracle_mod, mode):
    """Q = 0 makes every visible logit 0: lse = ln |vis(p)| and, with one-hot
    V_j = e_(j mod D), O_p[d] = #{j in vis(p): j = d mod D} / |vis(p)|."""
    L, n, D = 8, 4, 16
    N = n * L
    q = np.zeros((1, N, 1, D))
    k = np.random.default_rng(6).standard_normal((1, N, 1, D))
    v = np.zeros((1, N, 1, D))
    for j in range(N):
        v[0, j, 0, j % D] = 1.0
    o, lse = oracle_mod.sfa_fwd(q, k, v, L=L, n=n, mode=mode, scale=1.0)
    for p in range(N):
        vis = list(range(p % n, p + 1, n)) if mode == INTRA else list(range(p + 1))
        assert abs(lse[0, 0, p] - math.log(len(vis))) < 1e-13
        want = np.bincount(np.array(vis) % D, minlength=D) / len(vis)
        np.testing.assert_allclose(o[0, p, 0], want, atol=1e-14, rtol=0)
        if mode == INTRA:  # n | D: columns of other residues are exactly zero
            assert np.all(o[0, p, 0][np.arange(D) % n != p % n] == 0.0)


def test_stream_replicated_inputs(oracle_mod):
    """Identical q/k/v across the n streams of a token (what eq. (cyclic_init) yields at
    the input).  INTRA: each stream is causal attention over the L tokens.  MIX: row
    (t, s) weights earlier tokens by n and its own token by s + 1; at s = n - 1 the
    output is the causal-L output and lse gains ln n."""
    B, L, n, H, D = 1, 7, 3, 2, 6
    r = np.random.default_rng(7)
    base = [r.standard_normal((B, L, H, D)) for _ in range(3)]
    rep = [np.repeat(x, n, axis=1) for x in base]  # row t*n+s = token t
    scale = 0.45
    do = np.zeros((B, L, H, D))
    ro, rlse, *_ = _torch_causal(*base, do, scale)
    oi, lsei = oracle_mod.sfa_fwd(*rep, L=L, n=n, mode=INTRA, scale=scale)
    om, lsem = oracle_mod.sfa_fwd(*rep, L=L, n=n, mode=MIX, scale=scale)
    for s in range(n):
        np.testing.assert_allclose(oi[:, s::n], ro, atol=1e-12, rtol=0)
        np.testing.assert_allclose(lsei[:, :, s::n], rlse, atol=1e-12, rtol=0)
    np.testing.assert_allclose(om[:, n - 1::n], ro, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lsem[:, :, n - 1::n], rlse + math.log(n), atol=1e-12, rtol=0)
    # intermediate streams: explicit weighted softmax over tokens
    q, k, v = base
    for t in range(L):
        for s in range(n):
            for h in range(H):
                x = scale * (k[0, : t + 1, h] @ q[0, t, h])
                w = np.full(t + 1, float(n))
                w[t] = s + 1
                a = w * np.exp(x - x.max())
                np.testing.assert_allclose(om[0, t * n + s, h], a @ v[0, : t + 1, h] / a.sum(),
                                           atol=1e-12, rtol=0)
                assert abs(lsem[0, h, t * n + s] - (x.max() + math.log(a.sum()))) < 1e-12


@pytest.mark.parametrize("mode", [INTRA, MIX])
def test_gradient_sums(oracle_mod, mode):
    """Sum over keys of dV equals the group's summed dO; sum over keys of dK is 0 --
    per (b, kv-head), and per stream for INTRA."""
    B, L, n, Hq, Hkv, D = 2, 6, 3, 4, 2, 5
    q, k, v, do = _rand(8, B, L, n, Hq, Hkv, D)
    dq, dk, dv = oracle_mod.sfa_bwd(q, k, v, do, L=L, n=n, mode=mode, scale=0.6)
    G = Hq // Hkv
    for b in range(B):
        for hk in range(Hkv):
            group_do = do[b, :, hk * G:(hk + 1) * G]
            np.testing.assert_allclose(dv[b, :, hk].sum(0), group_do.sum((0, 1)), atol=1e-12)
            np.testing.assert_allclose(dk[b, :, hk].sum(0), 0.0, atol=1e-12)
            if mode == INTRA:
                for s in range(n):
                    np.testing.assert_allclose(dv[b, s::n, hk].sum(0),
                                               group_do[s::n].sum((0, 1)), atol=1e-12)
                    np.testing.assert_allclose(dk[b, s::n, hk].sum(0), 0.0, atol=1e-12)


def test_gqa_equals_repeated_heads(oracle_mod):
    """Grouped heads == one key/value head per query head with K/V repeated;
    dK/dV are the group sums of the repeated-head gradients."""
    B, L, n, Hq, Hkv, D = 1, 5, 2, 6, 2, 4
    G = Hq // Hkv
    q, k, v, do = _rand(9, B, L, n, Hq, Hkv, D)
    kr, vr = np.repeat(k, G, axis=2), np.repeat(v, G, axis=2)
    for mode in (INTRA, MIX):
        o, lse = oracle_mod.sfa_fwd(q, k, v, L=L, n=n, mode=mode, scale=0.5)
        o2, lse2 = oracle_mod.sfa_fwd(q, kr, vr, L=L, n=n, mode=mode, scale=0.5)
        np.testing.assert_allclose(o, o2, atol=1e-14)
        np.testing.assert_allclose(lse, lse2, atol=1e-14)
        dq, dk, dv = oracle_mod.sfa_bwd(q, k, v, do, L=L, n=n, mode=mode, scale=0.5)
        dq2, dk2, dv2 = oracle_mod.sfa_bwd(q, kr, vr, do, L=L, n=n, mode=mode, scale=0.5)
        np.testing.assert_allclose(dq, dq2, atol=1e-13)
        np.testing.assert_allclose(dk, dk2.reshape(B, n * L, Hkv, G, D).sum(3), atol=1e-13)
        np.testing.assert_allclose(dv, dv2.reshape(B, n * L, Hkv, G, D).sum(3), atol=1e-13)


def _fd_check(oracle_mod, shape, mode, seed, max_entries=None):
    B, L, n, Hq, Hkv, D = shape
    q, k, v, do = _rand(seed, *shape)
    scale = 1.0 / math.sqrt(D)
    grads = oracle_mod.sfa_bwd(q, k, v, do, L=L, n=n, mode=mode, scale=scale)
    h = 1e-6

    def f(qq, kk, vv):
        o, _ = oracle_mod.sfa_fwd(qq, kk, vv, L=L, n=n, mode=mode, scale=scale, nthreads=1)
        return float((do * o).sum())

    r = np.random.default_rng(seed + 100)
    for idx, (name, g) in enumerate(zip("qkv", grads)):
        x = [q, k, v][idx]
        entries = np.arange(x.size)
        if max_entries is not None and x.size > max_entries:
            entries = r.choice(x.size, size=max_entries, replace=False)
        gmax = np.abs(g).max()
        for e in entries:
            args = [q.copy(), k.copy(), v.copy()]
            args[idx].flat[e] += h
            fp = f(*args)
            args[idx].flat[e] -= 2 * h
            fm = f(*args)
            fd = (fp - fm) / (2 * h)
            assert abs(fd - g.flat[e]) <= 1e-6 * max(gmax, 1.0), (name, e, fd, g.flat[e])


@pytest.mark.parametrize("mode", [INTRA, MIX])
def test_finite_differences_every_entry_small(oracle_mod, mode):
    _fd_check(oracle_mod, (1, 4, 3, 2, 1, 4), mode, seed=10)


@pytest.mark.parametrize("mode", [INTRA, MIX])
def test_finite_differences_tiny_config_sampled(oracle_mod, mode):
    """Seeded subset of entries at the tiny fp32 workload shape (B=1 L=64 n=2 Hq=2 Hkv=1 D=32)."""
    _fd_check(oracle_mod, (1, 64, 2, 2, 1, 32), mode, seed=11, max_entries=24)


def test_bf16_inputs_upcast_exactly(oracle_mod):
    """bf16 bit patterns are read as their exact values (same result as fp64 input)."""
    B, L, n, Hq, Hkv, D = 1, 5, 2, 2, 1, 8
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=12, dtype="bf16")
    as64 = {kk: synth.bf16_bits_to_f32(vv).astype(np.float64) for kk, vv in ins.items()}
    for mode in (INTRA, MIX):
        a = oracle_mod.sfa_fwd(ins["q"], ins["k"], ins["v"], L=L, n=n, mode=mode, scale=0.3)
        b = oracle_mod.sfa_fwd(as64["q"], as64["k"], as64["v"], L=L, n=n, mode=mode, scale=0.3)
        np.testing.assert_array_equal(a[0], b[0])
        ga = oracle_mod.sfa_bwd(ins["q"], ins["k"], ins["v"], ins["dout"], L=L, n=n, mode=mode,
                                scale=0.3)
        gb = oracle_mod.sfa_bwd(as64["q"], as64["k"], as64["v"], as64["dout"], L=L, n=n,
                                mode=mode, scale=0.3)
        for x, y in zip(ga, gb):
            np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("mode", [INTRA, MIX])
def test_row_sampled_entry_points_match_full(oracle_mod, mode):
    B, L, n, Hq, Hkv, D = 2, 6, 3, 4, 2, 8
    q, k, v, do = _rand(13, B, L, n, Hq, Hkv, D)
    kw = dict(L=L, n=n, mode=mode, scale=0.4)
    o, lse = oracle_mod.sfa_fwd(q, k, v, **kw)
    dq, dk, dv = oracle_mod.sfa_bwd(q, k, v, do, **kw)
    rows = np.array([[0, 0, 0], [1, 3, 17], [0, 2, 9], [1, 1, 5]])
    ro, rl = oracle_mod.sfa_fwd_rows(q, k, v, rows, **kw)
    rdq = oracle_mod.sfa_bwd_dq_rows(q, k, v, do, rows, **kw)
    for i, (b, h, p) in enumerate(rows):
        np.testing.assert_array_equal(ro[i], o[b, p, h])
        assert rl[i] == lse[b, h, p]
        np.testing.assert_array_equal(rdq[i], dq[b, p, h])
    krows = np.array([[0, 0, 0], [1, 1, 17], [0, 1, 10]])
    rdk, rdv = oracle_mod.sfa_bwd_dkdv_rows(q, k, v, do, krows, **kw)
    for i, (b, h, j) in enumerate(krows):
        np.testing.assert_allclose(rdk[i], dk[b, j, h], atol=1e-13)
        np.testing.assert_allclose(rdv[i], dv[b, j, h], atol=1e-13)


def test_expand_matches_paper_two_stream_example(oracle_mod):
    g = json.load(open(os.path.join(GOLDEN, "expand_n2.json")))
    tables = np.array([g["tables_E1"], g["tables_E2"]], dtype=np.uint16)
    ids = np.array([g["ids"]], dtype=np.int32)
    out, bad = oracle_mod.expand_embed(ids, tables)
    assert bad == 0
    np.testing.assert_array_equal(out[0], np.array(g["expected_rows"], dtype=np.uint16))
    cyc = np.concatenate([tables, tables])  # eq. (cyclic_init): (E1, E2, E1, E2)
    out4, _ = oracle_mod.expand_embed(ids, cyc)
    np.testing.assert_array_equal(out4[0], np.array(g["cyclic_expected_rows_n4"], np.uint16))


def test_expand_bad_ids_zero_and_counted(oracle_mod):
    tables = np.arange(2 * 4 * 3, dtype=np.uint16).reshape(2, 4, 3) + 1
    ids = np.array([[0, -1, 4, 3], [7, 2, 2, 0]], dtype=np.int32)
    out, bad = oracle_mod.expand_embed(ids, tables)
    assert bad == 3
    assert np.all(out[0, 2:4] == 0) and np.all(out[0, 4:6] == 0) and np.all(out[1, 0:2] == 0)
    np.testing.assert_array_equal(out[0, 6], tables[0, 3])
    np.testing.assert_array_equal(out[0, 7], tables[1, 3])
    np.testing.assert_array_equal(out[1, 3], tables[1, 2])


# ------------------------------------------------------------------ local layers


def _torch_masked(q, k, v, do, scale, keep):
    """Library attention with an explicit boolean keep-mask [S][S] (True = visible)."""
    Hq, Hkv = q.shape[2], k.shape[2]
    G = Hq // Hkv
    tq = torch.tensor(q).permute(0, 2, 1, 3).contiguous().requires_grad_(True)
    tk = torch.tensor(k).permute(0, 2, 1, 3).contiguous().requires_grad_(True)
    tv = torch.tensor(v).permute(0, 2, 1, 3).contiguous().requires_grad_(True)
    kk = tk.repeat_interleave(G, dim=1)
    vv = tv.repeat_interleave(G, dim=1)
    keep_t = torch.tensor(keep)
    o = F.scaled_dot_product_attention(tq, kk, vv, attn_mask=keep_t, scale=scale)
    o.backward(torch.tensor(do).permute(0, 2, 1, 3))
    logits = scale * torch.matmul(tq.detach(), kk.detach().transpose(-1, -2))
    lse = torch.logsumexp(logits.masked_fill(~keep_t, float("-inf")), dim=-1)
    back = lambda t: t.permute(0, 2, 1, 3).detach().numpy()
    return back(o), lse.numpy(), back(tq.grad), back(tk.grad), back(tv.grad)


def _band(S, w):
    i = np.arange(S)
    return (i[None, :] <= i[:, None]) & (i[:, None] - i[None, :] < w)


@pytest.mark.parametrize("L,n,w", [(5, 3, 1), (16, 4, 7), (7, 1, 3), (4, 8, 13), (6, 2, 100)])
def test_local_mask_is_window_of_prefix(oracle_mod, L, n, w):
    """LOCAL row p sees exactly range(max(0, p - w + 1), p + 1)."""
    N = n * L
    m = oracle_mod.sfa_mask(L, n, LOCAL, w)
    for p in range(N):
        want = np.zeros(N, np.uint8)
        want[max(0, p - w + 1): p + 1] = 1
        np.testing.assert_array_equal(m[p], want)


@pytest.mark.parametrize("shape,w", [((1, 9, 1, 2, 2, 6), 4), ((2, 5, 3, 4, 2, 8), 6),
                                     ((1, 6, 4, 3, 3, 5), 9), ((1, 8, 2, 2, 1, 4), 1)])
def test_local_equals_sliding_window_attention(oracle_mod, shape, w):
    """LOCAL(w) == library attention under a sliding-window band over the expanded rows."""
    B, L, n, Hq, Hkv, D = shape
    q, k, v, do = _rand(21, *shape)
    scale = 1.0 / math.sqrt(D)
    kw = dict(L=L, n=n, mode=LOCAL, scale=scale, window=w)
    o, lse = oracle_mod.sfa_fwd(q, k, v, **kw)
    dq, dk, dv = oracle_mod.sfa_bwd(q, k, v, do, **kw)
    ro, rlse, rdq, rdk, rdv = _torch_masked(q, k, v, do, scale, _band(n * L, w))
    for got, ref in ((o, ro), (lse, rlse), (dq, rdq), (dk, rdk), (dv, rdv)):
        np.testing.assert_allclose(got, ref, atol=1e-12, rtol=0)


def test_local_wide_window_equals_mix(oracle_mod):
    B, L, n, Hq, Hkv, D = 1, 6, 3, 2, 1, 4
    q, k, v, do = _rand(22, B, L, n, Hq, Hkv, D)
    a = oracle_mod.sfa_fwd(q, k, v, L=L, n=n, mode=LOCAL, scale=0.4, window=n * L)
    b = oracle_mod.sfa_fwd(q, k, v, L=L, n=n, mode=MIX, scale=0.4)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    ga = oracle_mod.sfa_bwd(q, k, v, do, L=L, n=n, mode=LOCAL, scale=0.4, window=10 * n * L)
    gb = oracle_mod.sfa_bwd(q, k, v, do, L=L, n=n, mode=MIX, scale=0.4)
    for x, y in zip(ga, gb):
        np.testing.assert_array_equal(x, y)


def test_local_window_one_closed_form(oracle_mod):
    """w = 1: every row sees only itself, so O = v of its own row, lse = scale q.k, dV
    collects the group's dO, and dQ = dK = 0 (P = 1 makes dS = 0)."""
    B, L, n, Hq, Hkv, D = 1, 5, 2, 4, 2, 3
    q, k, v, do = _rand(23, B, L, n, Hq, Hkv, D)
    G = Hq // Hkv
    kw = dict(L=L, n=n, mode=LOCAL, scale=0.7, window=1)
    o, lse = oracle_mod.sfa_fwd(q, k, v, **kw)
    dq, dk, dv = oracle_mod.sfa_bwd(q, k, v, do, **kw)
    kr = np.repeat(k, G, axis=2)
    vr = np.repeat(v, G, axis=2)
    np.testing.assert_allclose(o, vr, atol=1e-14)
    np.testing.assert_allclose(lse, 0.7 * np.einsum("bphd,bphd->bhp", q, kr), atol=1e-13)
    np.testing.assert_allclose(dv, do.reshape(B, n * L, Hkv, G, D).sum(3), atol=1e-13)
    np.testing.assert_allclose(dq, 0, atol=1e-13)
    np.testing.assert_allclose(dk, 0, atol=1e-13)


def test_local_finite_differences_every_entry_small(oracle_mod):
    B, L, n, Hq, Hkv, D = 1, 4, 3, 2, 1, 4
    q, k, v, do = _rand(24, B, L, n, Hq, Hkv, D)
    scale = 1.0 / math.sqrt(D)
    kw = dict(L=L, n=n, mode=LOCAL, scale=scale, window=5)
    grads = oracle_mod.sfa_bwd(q, k, v, do, **kw)
    h = 1e-6

    def f(qq, kk, vv):
        o, _ = oracle_mod.sfa_fwd(qq, kk, vv, nthreads=1, **kw)
        return float((do * o).sum())

    for idx, g in enumerate(grads):
        x = [q, k, v][idx]
        for e in range(x.size):
            args = [q.copy(), k.copy(), v.copy()]
            args[idx].flat[e] += h
            fp = f(*args)
            args[idx].flat[e] -= 2 * h
            fd = (fp - f(*args)) / (2 * h)
            assert abs(fd - g.flat[e]) <= 1e-6 * max(np.abs(g).max(), 1.0)


def test_local_row_sampled_entry_points_match_full(oracle_mod):
    B, L, n, Hq, Hkv, D = 2, 6, 3, 4, 2, 5
    q, k, v, do = _rand(25, B, L, n, Hq, Hkv, D)
    kw = dict(L=L, n=n, mode=LOCAL, scale=0.5, window=7)
    o, lse = oracle_mod.sfa_fwd(q, k, v, **kw)
    dq, dk, dv = oracle_mod.sfa_bwd(q, k, v, do, **kw)
    rows = np.array([[0, 1, 0], [1, 3, 17], [0, 2, 9], [1, 0, 11]])
    ro, rl = oracle_mod.sfa_fwd_rows(q, k, v, rows, **kw)
    rdq = oracle_mod.sfa_bwd_dq_rows(q, k, v, do, rows, **kw)
    for i, (b, h, p) in enumerate(rows):
        np.testing.assert_allclose(ro[i], o[b, p, h], atol=1e-14)
        np.testing.assert_allclose(rl[i], lse[b, h, p], atol=1e-14)
        np.testing.assert_allclose(rdq[i], dq[b, p, h], atol=1e-14)
    krows = np.array([[0, 1, 0], [1, 0, 17], [0, 1, 9]])
    rdk, rdv = oracle_mod.sfa_bwd_dkdv_rows(q, k, v, do, krows, **kw)
    for i, (b, h, j) in enumerate(krows):
        np.testing.assert_allclose(rdk[i], dk[b, j, h], atol=1e-14)
        np.testing.assert_allclose(rdv[i], dv[b, j, h], atol=1e-14)


# ------------------------------------------------- expansion backward, cyclic init


def _interleave_embedding(ids, tables):
    """Library form of eq. (expansion): torch embedding lookups of the n tables,
    stacked on a new stream axis and flattened token-major ([B][L][n] -> [B][n*L])."""
    rows = torch.stack([F.embedding(ids, tables[s]) for s in range(tables.shape[0])], dim=2)
    B, L, n, Dm = rows.shape
    return rows.reshape(B, L * n, Dm)


def test_expand_bwd_matches_hand_worked_golden(oracle_mod):
    g = json.load(open(os.path.join(GOLDEN, "expand_bwd_n2.json")))
    ids = np.array([g["ids"]], dtype=np.int32)
    dout = np.array([g["dout"]], dtype=np.float64)
    d = oracle_mod.expand_embed_bwd(ids, dout, g["V"])
    np.testing.assert_array_equal(d[0], np.array(g["expected_dE1"], dtype=np.float64))
    np.testing.assert_array_equal(d[1], np.array(g["expected_dE2"], dtype=np.float64))


@pytest.mark.parametrize("B,L,n,V,Dm", [(1, 40, 2, 7, 5), (3, 17, 4, 50, 8), (2, 9, 1, 3, 4)])
def test_expand_bwd_equals_library_autograd(oracle_mod, B, L, n, V, Dm):
    """The gradient through torch's embedding lookups (autograd, fp64) of the interleaved
    expansion equals the oracle's scatter-add, duplicates included."""
    r = np.random.default_rng(B * 100 + L)
    ids = r.integers(0, V, size=(B, L)).astype(np.int32)  # V small: many repeats
    tables = torch.tensor(r.standard_normal((n, V, Dm)), requires_grad=True)
    dout = r.standard_normal((B, n * L, Dm))
    out = _interleave_embedding(torch.tensor(ids, dtype=torch.int64), tables)
    out.backward(torch.tensor(dout))
    np.testing.assert_allclose(oracle_mod.expand_embed_bwd(ids, dout, V), tables.grad.numpy(),
                               rtol=1e-13, atol=1e-13)


def test_expand_bwd_is_adjoint_of_forward(oracle_mod):
    """<expand(E), G> == <E, expand_bwd(G)> for random E, G, with repeated and
    out-of-range ids (the oracle's forward copies bytes, so fp64 tables go through it
    exactly)."""
    r = np.random.default_rng(7)
    B, L, n, V, Dm = 2, 33, 3, 11, 6
    ids = r.integers(-2, V + 2, size=(B, L)).astype(np.int32)
    E = r.standard_normal((n, V, Dm))
    G = r.standard_normal((B, n * L, Dm))
    fwd, bad = oracle_mod.expand_embed(ids, E)
    assert bad == int(np.sum((ids < 0) | (ids >= V)))
    lhs = float(np.sum(fwd * G))
    rhs = float(np.sum(E * oracle_mod.expand_embed_bwd(ids, G, V)))
    assert abs(lhs - rhs) <= 1e-12 * np.sum(np.abs(fwd * G))


def test_expand_bwd_distinct_ids_is_a_permutation(oracle_mod):
    """All ids distinct: each upstream row lands, unchanged, in one table row."""
    r = np.random.default_rng(8)
    L, n, V, Dm = 20, 4, 64, 8
    ids = r.permutation(V)[:L].astype(np.int32).reshape(1, L)
    dout = synth.to_bf16_bits(r.standard_normal((1, n * L, Dm)))
    d = oracle_mod.expand_embed_bwd(ids, dout, V)
    rows = synth.bf16_bits_to_f32(dout).astype(np.float64)
    for t in range(L):
        for s in range(n):
            np.testing.assert_array_equal(d[s, ids[0, t]], rows[0, t * n + s])
    untouched = np.setdiff1d(np.arange(V), ids[0])
    assert np.all(d[:, untouched] == 0)


def test_expand_bwd_one_repeated_id_sums_each_stream(oracle_mod):
    """Every token has the same id x: table s at x holds the sum of the stream-s rows."""
    r = np.random.default_rng(9)
    B, L, n, V, Dm = 2, 30, 3, 5, 4
    ids = np.full((B, L), 3, dtype=np.int32)
    dout = r.standard_normal((B, n * L, Dm))
    d = oracle_mod.expand_embed_bwd(ids, dout, V)
    for s in range(n):
        np.testing.assert_allclose(d[s, 3], dout[:, s::n].sum(axis=(0, 1)), rtol=1e-13)
    assert np.all(d[:, [0, 1, 2, 4]] == 0)


def test_expand_bwd_rows_equal_dense(oracle_mod):
    r = np.random.default_rng(10)
    B, L, n, V, Dm = 2, 25, 2, 9, 3
    ids = r.integers(-1, V + 1, size=(B, L)).astype(np.int32)
    dout = r.standard_normal((B, n * L, Dm))
    dense = oracle_mod.expand_embed_bwd(ids, dout, V)
    req = np.array([0, 8, 4, -1, V, 4], dtype=np.int32)
    rows = oracle_mod.expand_embed_bwd_rows(ids, dout, V, req)
    for i, x in enumerate(req):
        want = dense[:, x] if 0 <= x < V else np.zeros((n, Dm))
        np.testing.assert_array_equal(rows[i], want)


def test_cyclic_replicate_matches_paper_examples(oracle_mod):
    g = json.load(open(os.path.join(GOLDEN, "expand_bwd_n2.json")))
    V, Dm = 3, 2
    for n, m, want in ((2, 4, g["cyclic_n2_to_4"]), (4, 8, g["cyclic_n4_to_8"])):
        tables = np.stack([np.full((V, Dm), s + 1, dtype=np.uint16) for s in range(n)])
        out = oracle_mod.cyclic_replicate(tables, m)
        assert [int(out[s, 0, 0]) for s in range(m)] == want
        np.testing.assert_array_equal(out[:n], tables)


def test_cyclic_replicate_reproduces_the_smaller_model_rows(oracle_mod):
    """After E_{n+k} <- E_k the expanded rows of stream s and s + n coincide, and the
    first n streams of every token are the n-stream expansion (the expanded model
    starts from the smaller one's inputs)."""
    r = np.random.default_rng(11)
    n, V, Dm, L = 2, 10, 4, 6
    tables = synth.to_bf16_bits(r.standard_normal((n, V, Dm)))
    ids = r.integers(0, V, size=(1, L)).astype(np.int32)
    big = oracle_mod.cyclic_replicate(tables, 2 * n)
    out2, _ = oracle_mod.expand_embed(ids, tables)
    out4, _ = oracle_mod.expand_embed(ids, big)
    for t in range(L):
        for s in range(n):
            np.testing.assert_array_equal(out4[0, t * 2 * n + s], out4[0, t * 2 * n + s + n])
            np.testing.assert_array_equal(out4[0, t * 2 * n + s], out2[0, t * n + s])


# ------------------------------------------------- final-stream query layers


def _embed_final(xf, n, fill):
    """[B][L][H][D] final-stream rows placed at expanded positions t*n + n - 1 of a
    [B][n*L][H][D] array whose other rows are `fill`."""
    B, L, H, D = xf.shape
    full = np.array(fill, dtype=np.float64, copy=True).reshape(B, n * L, H, D)
    full[:, n - 1::n] = xf
    return full


FINAL_SHAPES = [(1, 7, 3, 2, 1, 4), (2, 5, 2, 4, 2, 8), (1, 6, 4, 3, 3, 5), (1, 9, 1, 2, 2, 6)]


@pytest.mark.parametrize("mode,w", [(MIX, 0), (LOCAL, 5), (LOCAL, 1), (LOCAL, 100)])
@pytest.mark.parametrize("shape", FINAL_SHAPES, ids=[str(s) for s in FINAL_SHAPES])
def test_final_stream_layer_equals_library_rows(oracle_mod, shape, mode, w):
    """Final-stream queries over all n streams' keys == library attention over the whole
    expanded sequence (other query rows arbitrary, their upstream gradient zero), read at
    the rows t*n + n - 1: outputs, lse, dq of those rows, and dk/dv of every key."""
    B, L, n, Hq, Hkv, D = shape
    N = n * L
    r = np.random.default_rng(31 + L)
    qf = r.standard_normal((B, L, Hq, D))
    k = r.standard_normal((B, N, Hkv, D))
    v = r.standard_normal((B, N, Hkv, D))
    dof = r.standard_normal((B, L, Hq, D))
    qfull = _embed_final(qf, n, r.standard_normal((B, N, Hq, D)))
    dofull = _embed_final(dof, n, np.zeros((B, N, Hq, D)))
    scale = 0.7
    keep = _band(N, w) if mode == LOCAL else _band(N, N)
    to, tl, tdq, tdk, tdv = _torch_masked(qfull, k, v, dofull, scale, keep)
    kw = dict(L=L, n=n, mode=mode, scale=scale, window=w, final=True)
    o, lse = oracle_mod.sfa_fwd(qf, k, v, **kw)
    dq, dk, dv = oracle_mod.sfa_bwd(qf, k, v, dof, **kw)
    np.testing.assert_allclose(o, to[:, n - 1::n], atol=1e-12)
    np.testing.assert_allclose(lse, tl[:, :, n - 1::n], atol=1e-12)
    np.testing.assert_allclose(dq, tdq[:, n - 1::n], atol=1e-12)
    np.testing.assert_allclose(dk, tdk, atol=1e-12)
    np.testing.assert_allclose(dv, tdv, atol=1e-12)


def test_final_stream_with_one_stream_is_the_mixing_layer(oracle_mod):
    q, k, v, do = _rand(33, 2, 11, 1, 4, 2, 8)
    kw = dict(L=11, n=1, mode=MIX, scale=0.4)
    for a, b in zip(oracle_mod.sfa_fwd(q, k, v, **kw) + oracle_mod.sfa_bwd(q, k, v, do, **kw),
                    oracle_mod.sfa_fwd(q, k, v, final=True, **kw)
                    + oracle_mod.sfa_bwd(q, k, v, do, final=True, **kw)):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("mode,w", [(MIX, 0), (LOCAL, 6)])
def test_final_stream_uniform_logits(oracle_mod, mode, w):
    """q = 0: token t's final-stream query sees (t+1)n keys (min with w for LOCAL), so
    lse = ln|vis| and O is the mean of the visible values."""
    L, n, D = 9, 3, 4
    N = n * L
    r = np.random.default_rng(34)
    qf = np.zeros((1, L, 1, D))
    k = r.standard_normal((1, N, 1, D))
    v = r.standard_normal((1, N, 1, D))
    o, lse = oracle_mod.sfa_fwd(qf, k, v, L=L, n=n, mode=mode, scale=1.0, window=w, final=True)
    for t in range(L):
        p = t * n + n - 1
        lo = max(0, p - w + 1) if mode == LOCAL else 0
        assert abs(lse[0, 0, t] - math.log(p + 1 - lo)) < 1e-12
        np.testing.assert_allclose(o[0, t, 0], v[0, lo:p + 1, 0].mean(axis=0), atol=1e-12)


def test_final_stream_replicated_streams_reduce_to_token_causal(oracle_mod):
    """Keys/values identical across the n streams of every token (eq. (cyclic_init) at
    the input): the final stream of token t sees n copies of each token <= t, i.e.
    causal attention over the L tokens with lse raised by ln n."""
    B, L, n, Hq, Hkv, D = 1, 10, 4, 2, 1, 6
    r = np.random.default_rng(35)
    qf = r.standard_normal((B, L, Hq, D))
    kt = r.standard_normal((B, L, Hkv, D))
    vt = r.standard_normal((B, L, Hkv, D))
    k, v = np.repeat(kt, n, axis=1), np.repeat(vt, n, axis=1)
    o, lse = oracle_mod.sfa_fwd(qf, k, v, L=L, n=n, mode=MIX, scale=0.5, final=True)
    to, tl, _, _, _ = _torch_causal(qf, kt, vt, np.zeros_like(qf), 0.5)
    np.testing.assert_allclose(o, to, atol=1e-12)
    np.testing.assert_allclose(lse, tl + math.log(n), atol=1e-12)


@pytest.mark.parametrize("mode,w", [(MIX, 0), (LOCAL, 4)])
def test_final_stream_finite_differences(oracle_mod, mode, w):
    B, L, n, Hq, Hkv, D = 1, 4, 3, 2, 1, 4
    r = np.random.default_rng(36)
    qf = r.standard_normal((B, L, Hq, D))
    k = r.standard_normal((B, n * L, Hkv, D))
    v = r.standard_normal((B, n * L, Hkv, D))
    dof = r.standard_normal((B, L, Hq, D))
    kw = dict(L=L, n=n, mode=mode, scale=0.5, window=w, final=True)
    grads = oracle_mod.sfa_bwd(qf, k, v, dof, **kw)

    def f(qq, kk, vv):
        return float((dof * oracle_mod.sfa_fwd(qq, kk, vv, nthreads=1, **kw)[0]).sum())

    h = 1e-6
    for idx, g in enumerate(grads):
        x = [qf, k, v][idx]
        gmax = max(np.abs(g).max(), 1.0)
        for e in range(x.size):
            args = [qf.copy(), k.copy(), v.copy()]
            args[idx].flat[e] += h
            fp = f(*args)
            args[idx].flat[e] -= 2 * h
            fd = (fp - f(*args)) / (2 * h)
            assert abs(fd - g.flat[e]) <= 1e-6 * gmax, ("qkv"[idx], e)


def test_final_stream_rows_equal_full(oracle_mod):
    B, L, n, Hq, Hkv, D = 2, 6, 3, 4, 2, 5
    r = np.random.default_rng(37)
    qf = r.standard_normal((B, L, Hq, D))
    k = r.standard_normal((B, n * L, Hkv, D))
    v = r.standard_normal((B, n * L, Hkv, D))
    dof = r.standard_normal((B, L, Hq, D))
    kw = dict(L=L, n=n, mode=LOCAL, scale=0.6, window=7, final=True)
    o, lse = oracle_mod.sfa_fwd(qf, k, v, **kw)
    dq, dk, dv = oracle_mod.sfa_bwd(qf, k, v, dof, **kw)
    rows = np.array([[0, 0, 0], [1, 3, 5], [0, 2, 3]])
    ro, rl = oracle_mod.sfa_fwd_rows(qf, k, v, rows, **kw)
    rdq = oracle_mod.sfa_bwd_dq_rows(qf, k, v, dof, rows, **kw)
    for i, (b, h, t) in enumerate(rows):
        np.testing.assert_allclose(ro[i], o[b, t, h], atol=1e-13)
        assert abs(rl[i] - lse[b, h, t]) < 1e-13
        np.testing.assert_allclose(rdq[i], dq[b, t, h], atol=1e-13)
    krows = np.array([[0, 0, 0], [1, 1, 17], [0, 1, 10]])
    rdk, rdv = oracle_mod.sfa_bwd_dkdv_rows(qf, k, v, dof, krows, **kw)
    for i, (b, h, j) in enumerate(krows):
        np.testing.assert_allclose(rdk[i], dk[b, j, h], atol=1e-13)
        np.testing.assert_allclose(rdv[i], dv[b, j, h], atol=1e-13)


# ------------------------------------------------------- parallel-stream decode


@pytest.mark.parametrize("mode,w", [(MIX, 0), (INTRA, 0), (LOCAL, 6)])
def test_decode_equals_library_last_rows(oracle_mod, mode, w):
    """Decode of the new token's n streams == library attention over each sequence's
    cached prefix (its own context length) read at the last n rows; intra-stream layers
    compare with causal attention over the de-interleaved stream."""
    B, Lcap, n, Hq, Hkv, D = 3, 9, 3, 4, 2, 5
    r = np.random.default_rng(41 + mode)
    ctx = np.array([0, 8, 4])
    q = r.standard_normal((B, n, Hq, D))
    kc = r.standard_normal((B, n * Lcap, Hkv, D))
    vc = r.standard_normal((B, n * Lcap, Hkv, D))
    o, lse = oracle_mod.sfa_decode(q, kc, vc, ctx, n=n, mode=mode, scale=0.6, window=w)
    for b in range(B):
        c = int(ctx[b])
        S = n * (c + 1)
        if mode == INTRA:
            for s in range(n):
                ks, vs = kc[b:b + 1, s:S:n], vc[b:b + 1, s:S:n]
                qs = np.zeros((1, c + 1, Hq, D))
                qs[0, c] = q[b, s]
                to, tl, _, _, _ = _torch_causal(qs, ks, vs, np.zeros_like(qs), 0.6)
                np.testing.assert_allclose(o[b, s], to[0, c], atol=1e-12)
                np.testing.assert_allclose(lse[b, :, s], tl[0, :, c], atol=1e-12)
            continue
        qf = np.zeros((1, S, Hq, D))
        qf[0, c * n:] = q[b]
        keep = _band(S, w) if mode == LOCAL else _band(S, S)
        to, tl, _, _, _ = _torch_masked(qf, kc[b:b + 1, :S], vc[b:b + 1, :S],
                                        np.zeros_like(qf), 0.6, keep)
        np.testing.assert_allclose(o[b], to[0, c * n:], atol=1e-12)
        np.testing.assert_allclose(lse[b], tl[0, :, c * n:], atol=1e-12)


def test_decode_ignores_cache_past_the_new_token_and_other_streams(oracle_mod):
    """Rows past ctx*n + n - 1 are never read; intra-stream decode reads only its
    stream's rows (poisoning the rest changes nothing)."""
    B, Lcap, n, Hq, Hkv, D = 2, 7, 2, 2, 1, 4
    r = np.random.default_rng(42)
    ctx = np.array([3, 5])
    q = r.standard_normal((B, n, Hq, D))
    kc = r.standard_normal((B, n * Lcap, Hkv, D))
    vc = r.standard_normal((B, n * Lcap, Hkv, D))
    for mode in (MIX, INTRA):
        o, lse = oracle_mod.sfa_decode(q, kc, vc, ctx, n=n, mode=mode, scale=0.5)
        kp, vp = kc.copy(), vc.copy()
        for b in range(B):
            kp[b, (ctx[b] + 1) * n:] = 1e6
            vp[b, (ctx[b] + 1) * n:] = np.nan
        o2, lse2 = oracle_mod.sfa_decode(q, kp, vp, ctx, n=n, mode=mode, scale=0.5)
        np.testing.assert_array_equal(o, o2)
        np.testing.assert_array_equal(lse, lse2)
    kp, vp = kc.copy(), vc.copy()
    kp[:, 1::n], vp[:, 1::n] = 1e6, np.nan  # stream 1 poisoned: stream 0 unchanged
    o, lse = oracle_mod.sfa_decode(q, kc, vc, ctx, n=n, mode=INTRA, scale=0.5)
    o2, lse2 = oracle_mod.sfa_decode(q, kp, vp, ctx, n=n, mode=INTRA, scale=0.5)
    np.testing.assert_array_equal(o[:, 0], o2[:, 0])
    np.testing.assert_array_equal(lse[:, :, 0], lse2[:, :, 0])


def test_final_gather_reads_the_supervised_stream(oracle_mod):
    """eq. (hd_loss) supervises the final stream E_n(x_i) of each token: gathered from the
    layer-0 expanded sequence it is the paper's n=2 example's E2 rows, and in general the
    final table's rows of the ids (numpy indexing)."""
    g = json.load(open(os.path.join(GOLDEN, "expand_n2.json")))
    tables = np.array([g["tables_E1"], g["tables_E2"]], dtype=np.uint16)
    ids = np.array([g["ids"]], dtype=np.int32)
    out, _ = oracle_mod.expand_embed(ids, tables)
    fin = oracle_mod.final_gather(out, 2)
    np.testing.assert_array_equal(fin[0], np.array(g["expected_rows"], dtype=np.uint16)[1::2])
    r = np.random.default_rng(21)
    for n in (1, 3, 5):
        B, L, V, Dm = 2, 13, 9, 4
        ids = r.integers(0, V, size=(B, L)).astype(np.int32)
        tab = r.standard_normal((n, V, Dm))
        out, _ = oracle_mod.expand_embed(ids, tab)
        np.testing.assert_array_equal(oracle_mod.final_gather(out, n), tab[n - 1][ids])
        if n == 1:  # one stream: the gather is the identity
            np.testing.assert_array_equal(oracle_mod.final_gather(out, 1), out)


def test_final_gather_bwd_equals_library_autograd_and_is_adjoint(oracle_mod):
    """The gradient of torch's index_select of rows i*n + n-1 (autograd, fp64) equals the
    oracle's backward, which is zero at the other n-1 rows of each token, and
    <gather(h), y> == <h, gather_bwd(y)>."""
    r = np.random.default_rng(22)
    for B, L, n, Dm in ((1, 7, 4, 3), (3, 10, 2, 5), (2, 6, 1, 4)):
        h = torch.tensor(r.standard_normal((B, n * L, Dm)), requires_grad=True)
        y = r.standard_normal((B, L, Dm))
        torch.index_select(h, 1, torch.arange(L) * n + n - 1).backward(torch.tensor(y))
        dh = oracle_mod.final_gather_bwd(y, n)
        np.testing.assert_array_equal(dh, h.grad.numpy())
        hv = h.detach().numpy()
        lhs = float(np.sum(oracle_mod.final_gather(hv, n) * y))
        assert abs(lhs - float(np.sum(hv * dh))) <= 1e-12 * np.sum(np.abs(hv[:, n - 1::n] * y))
