"""The two LDS rings of the bf16 dQ pass at head widths 64 and 32.

The dQ launch streams the stored dS tiles and the key rows through one of two rings:
32 keys x 2 stages with several workgroups per CU when the grid is larger than what the
CUs hold at once with that ring, else 64 keys x 3 stages with one workgroup per CU.  At
D=64 and D=32 the first holds 4 workgroups per CU (1024 on MI355X's 256 CUs).  Here a
B=1, L=4096, n=4, Hq=32, Hkv=8 layer (2048 dQ workgroups: the co-resident ring) and its
first 1536 tokens (768 workgroups: the other ring) run on the same inputs:
  * sampled dQ rows of both against the oracle, at the 5e-2 bar;
  * every dQ row of the short layer bitwise equal to the same row of the long one.
Causal attention makes the first tokens' rows independent of later tokens, so the
short layer's dS tiles are the long layer's, and both rings add the keys of a row in
the same ascending order.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth
from tests import gpu_helpers as G

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

INTRA, MIX = 0, 1
B, L, n, Hq, Hkv = 1, 4096, 4, 32, 8
L_SHORT = 1536


def _grid(Lq, mode):
    """dQ workgroups: 256 query rows each, per (b, hq[, stream])."""
    rows = Lq if mode == INTRA else n * Lq
    return (rows + 255) // 256 * B * Hq * (n if mode == INTRA else 1)


@pytest.mark.parametrize("D", [64, 32])
@pytest.mark.parametrize("mode", [INTRA, MIX], ids=["intra", "mix"])
def test_dq_rings_agree(mode, D):
    assert _grid(L, mode) > 4 * 256 >= _grid(L_SHORT, mode)
    seed = synth.seed_for("dq_rings", mode, D)
    print(f"dq rings mode={mode} D={D} seed={seed}", flush=True)
    ins = synth.sfa_inputs(B, L, n, Hq, Hkv, D, seed=seed, dtype="bf16", qkv_std=2 ** -0.5)
    scale = D ** -0.5
    long_ = G.run_sfa(ins, n, mode, scale)
    Ns = n * L_SHORT
    short_ins = {k: np.ascontiguousarray(v[:, :Ns]) for k, v in ins.items()}
    short = G.run_sfa(short_ins, n, mode, scale)
    # the short layer is the long one's prefix, row for row and bit for bit
    for name in ("o", "dq"):
        a = G.bits(long_[name][:, :Ns])
        b = G.bits(short[name])
        assert np.array_equal(a, b), f"{name}: {np.count_nonzero(a != b)} elements differ"
    rng = np.random.default_rng(seed & 0xFFFFFFFF)
    for what, got, L_, inputs in (("long", long_, L, ins), ("short", short, L_SHORT, short_ins)):
        N = n * L_
        rows = {(0, 0, 0), (0, Hq - 1, N - 1), (0, 5, N // 2)}
        while len(rows) < 24:
            rows.add((0, int(rng.integers(Hq)), int(rng.integers(N))))
        rows = np.array(sorted(rows), dtype=np.int64)
        kw = dict(L=L_, n=n, mode=mode, scale=scale)
        rdq = oracle.sfa_bwd_dq_rows(inputs["q"], inputs["k"], inputs["v"], inputs["dout"], rows,
                                     **kw)
        b, h, p = rows.T
        G.assert_close_grad(G.to_host64(got["dq"])[b, p, h], rdq, "bf16", "dq", f"{what} D={D}")
    torch.cuda.synchronize()
