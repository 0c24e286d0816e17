"""GPU parity over a seeded random draw of small shapes, beyond the hand-picked cases:
batch, length, stream count, grouped-query ratio, head dim, layer type (intra-stream,
full and local cross-stream, final-stream full and local) and window, each forward and
backward against the fp64 oracle at the bf16 tolerances (max |O - O_ref| and
max |lse - lse_ref| <= 2e-2; max |g - g_ref| / max |g_ref| <= 5e-2 for dQ, dK, dV).
Decode steps are drawn the same way (batch, cache capacity, ragged per-sequence contexts,
mask, window, heads), and fp32-path shapes (max error <= 1e-4 on every output).  The lists are drawn once from fixed seeds, so every run checks the
same cases."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth
from tests import gpu_helpers as G

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

INTRA, MIX, LOCAL = 0, 1, 2


def _draw(count=32, seed=20261202):
    r = np.random.default_rng(seed)
    cases = []
    for _ in range(count):
        kind = ["intra", "mix", "local", "final", "final-local"][int(r.integers(5))]
        n = int(r.integers(1, 9))
        L = int(r.integers(1, 1200 // n + 1)) if kind in ("mix", "local") else int(r.integers(1, 400))
        B = int(r.integers(1, 3))
        Hkv = int(r.integers(1, 3))
        Hq = Hkv * int(r.choice([1, 2, 4, 8]))
        D = int(r.choice([32, 64, 128]))
        window = int(r.integers(1, 2 * n * L + 2)) if "local" in kind else 0
        cases.append((kind, B, L, n, Hq, Hkv, D, window))
    return cases


CASES = _draw()


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-B{c[1]}-L{c[2]}-n{c[3]}-Hq{c[4]}-Hkv{c[5]}-D{c[6]}-w{c[7]}"
                                               for c in CASES])
def test_random_shape_parity(case):
    kind, B, L, n, Hq, Hkv, D, window = case
    seed = synth.seed_for("random_shapes", case)
    print(f"random shape {case} seed={seed}", flush=True)
    scale = 1.0 / math.sqrt(D)
    final = kind.startswith("final")
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=seed, dtype="bf16", qkv_std=2 ** -0.5)
    if final:  # queries and upstream gradients at the final stream of each token only
        ins["q"] = np.ascontiguousarray(ins["q"][:, n - 1::n])
        ins["dout"] = np.ascontiguousarray(ins["dout"][:, n - 1::n])
        q, k, v, do = (G.to_dev(ins[x]) for x in ("q", "k", "v", "dout"))
        o, lse = hd.sfa_final_forward(q, k, v, n=n, window=window, scale=scale)
        dq, dk, dv = hd.sfa_final_backward(q, k, v, o, lse, do, n=n, window=window, scale=scale)
        mode = LOCAL if window else MIX
    else:
        mode = {"intra": INTRA, "mix": MIX, "local": LOCAL}[kind]
        q, k, v, do = (G.to_dev(ins[x]) for x in ("q", "k", "v", "dout"))
        o, lse = hd.sfa_forward(q, k, v, n=n, mode=mode, scale=scale,
                                window=window if mode == LOCAL else None)
        dq, dk, dv = hd.sfa_backward(q, k, v, o, lse, do, n=n, mode=mode, scale=scale,
                                     window=window if mode == LOCAL else None)
    torch.cuda.synchronize()
    kw = dict(L=L, n=n, mode=mode, scale=scale, window=window, final=final)
    ro, rl = oracle.sfa_fwd(ins["q"], ins["k"], ins["v"], **kw)
    rdq, rdk, rdv = oracle.sfa_bwd(ins["q"], ins["k"], ins["v"], ins["dout"], **kw)
    G.assert_close_fwd(G.to_host64(o), G.to_host64(lse), ro, rl, "bf16", str(case))
    for name, got, ref in (("dq", dq, rdq), ("dk", dk, rdk), ("dv", dv, rdv)):
        G.assert_close_grad(G.to_host64(got), ref, "bf16", name, str(case))


def _draw_decode(count=16, seed=20261203):
    r = np.random.default_rng(seed)
    cases = []
    for _ in range(count):
        mode = int(r.integers(3))
        n = int(r.integers(1, 9))
        B = int(r.integers(1, 5))
        Lcap = int(r.integers(1, 1500))
        Hkv = int(r.integers(1, 3))
        Hq = Hkv * int(r.choice([1, 2, 4, 8]))
        D = int(r.choice([32, 64, 128]))
        window = int(r.integers(1, 2 * n * Lcap + 2)) if mode == LOCAL else 0
        ctx = [int(c) for c in r.integers(0, Lcap, size=B)]
        cases.append((mode, B, Lcap, n, Hq, Hkv, D, window, ctx))
    return cases


DECODE_CASES = _draw_decode()


@pytest.mark.parametrize("case", DECODE_CASES,
                         ids=[f"m{c[0]}-B{c[1]}-Lcap{c[2]}-n{c[3]}-Hq{c[4]}-Hkv{c[5]}-D{c[6]}-w{c[7]}"
                              for c in DECODE_CASES])
def test_random_decode_parity(case):
    mode, B, Lcap, n, Hq, Hkv, D, window, ctx = case
    seed = synth.seed_for("random_decode", str(case))
    print(f"random decode {case} seed={seed}", flush=True)
    to = synth.to_bf16_bits
    q = to(synth.normal(seed, (B, n, Hq, D), 2 ** -0.5))
    k = to(synth.normal(seed + 1, (B, n * Lcap, Hkv, D), 2 ** -0.5))
    v = to(synth.normal(seed + 2, (B, n * Lcap, Hkv, D), 2 ** -0.5))
    tctx = torch.from_numpy(np.asarray(ctx, dtype=np.int32)).to(G.dev())
    o, lse = hd.sfa_decode(G.to_dev(q), G.to_dev(k), G.to_dev(v), tctx, max_ctx=max(ctx),
                           mode=mode, window=window, scale=D ** -0.5)
    torch.cuda.synchronize()
    ro, rl = oracle.sfa_decode(q, k, v, ctx, n=n, mode=mode, scale=D ** -0.5, window=window)
    G.assert_close_fwd(G.to_host64(o), G.to_host64(lse), ro, rl, "bf16", str(case))


def _draw_f32(count=8, seed=20261204):
    r = np.random.default_rng(seed)
    cases = []
    for _ in range(count):
        mode = int(r.integers(3))
        n = int(r.integers(1, 6))
        L = int(r.integers(1, 300 // n + 1))
        B = int(r.integers(1, 3))
        Hkv = int(r.integers(1, 3))
        Hq = Hkv * int(r.choice([1, 2, 4]))
        D = int(r.choice([32, 64, 128]))
        window = int(r.integers(1, 2 * n * L + 2)) if mode == LOCAL else 0
        cases.append((mode, B, L, n, Hq, Hkv, D, window))
    return cases


F32_CASES = _draw_f32()


@pytest.mark.parametrize("case", F32_CASES,
                         ids=[f"m{c[0]}-B{c[1]}-L{c[2]}-n{c[3]}-Hq{c[4]}-Hkv{c[5]}-D{c[6]}-w{c[7]}"
                              for c in F32_CASES])
def test_random_f32_parity(case):
    """The fp32 path at its 1e-4 bar (same forms as the bf16 one)."""
    mode, B, L, n, Hq, Hkv, D, window = case
    seed = synth.seed_for("random_f32", str(case))
    print(f"random f32 {case} seed={seed}", flush=True)
    scale = 1.0 / math.sqrt(D)
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=seed, dtype="f32")
    got = G.run_sfa(ins, n, mode, scale, window=window if mode == LOCAL else None)
    kw = dict(L=L, n=n, mode=mode, scale=scale, window=window)
    ro, rl = oracle.sfa_fwd(ins["q"], ins["k"], ins["v"], **kw)
    rdq, rdk, rdv = oracle.sfa_bwd(ins["q"], ins["k"], ins["v"], ins["dout"], **kw)
    G.assert_close_fwd(G.to_host64(got["o"]), G.to_host64(got["lse"]), ro, rl, "f32", str(case))
    for name, ref in (("dq", rdq), ("dk", rdk), ("dv", rdv)):
        G.assert_close_grad(G.to_host64(got[name]), ref, "f32", name, str(case))
