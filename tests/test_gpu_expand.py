"""GPU parity of the multi-stream token expansion, eq. (expansion) (Sec. "Multi-Stream
Token Expansion"): out[b][t*n + s] = tables[s][ids[b][t]], against the oracle's literal
triple loop.  The expansion is a copy, so the bar is bit-exact: every expanded row, and
the count of out-of-range ids (whose n rows are zeros).

Row sizes pick the kernel's copy word: rows whose byte size is a multiple of 16 move as
16-byte words, other multiples of 4 as 4-byte words, the rest as 2-byte words.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth, workloads
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu


def _tables(seed, n, V, Dm, dtype):
    x = synth.normal(seed, (n, V, Dm), 0.02)
    return synth.to_bf16_bits(x) if dtype == "bf16" else x.astype(np.float32)


def _host(t, dtype):
    a = t.cpu()
    return a.view(torch.int16).numpy().view(np.uint16) if dtype == "bf16" else a.numpy()


def _expand(ids, tables, dtype, count_bad=True):
    tids = torch.from_numpy(np.ascontiguousarray(ids)).to(G.dev())
    bad = torch.zeros(1, dtype=torch.int32, device=G.dev()) if count_bad else None
    out = hd.expand_embed(tids, G.to_dev(tables), bad_id_count=bad)
    torch.cuda.synchronize()
    return _host(out, dtype), (int(bad.cpu()[0]) if count_bad else None)


# (B, L, n, V, Dm, dtype): Dm sets the copy word (bf16 rows of 2*Dm bytes, fp32 4*Dm)
CASES = [
    (1, 37, 1, 100, 64, "bf16"),    # n = 1: the plain embedding lookup; 16-byte words
    (3, 50, 2, 1000, 64, "bf16"),   # the paper's n = 2 interleave
    (1, 29, 3, 77, 136, "bf16"),    # odd n; 272-byte rows, 16-byte words
    (3, 64, 4, 500, 10, "bf16"),    # 20-byte rows: 4-byte words
    (1, 33, 8, 300, 7, "bf16"),     # 14-byte rows: 2-byte words
    (2, 45, 8, 64, 4096, "bf16"),   # n = 8, a full model width
    (1, 40, 4, 200, 32, "f32"),     # fp32 tables, 128-byte rows
    (3, 21, 2, 150, 5, "f32"),      # fp32, 20-byte rows: 4-byte words
    (1, 1, 3, 5, 2, "bf16"),        # one token, 4-byte rows
    (2, 3, 2, 1, 1, "bf16"),        # V = 1, 2-byte rows
]


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_expand_bit_exact(case):
    B, L, n, V, Dm, dtype = case
    seed = synth.seed_for("expand", case)
    print(f"expand case={case} seed={seed}", flush=True)
    ids = synth.token_ids(seed, B, L, V)
    tables = _tables(seed + 1, n, V, Dm, dtype)
    got, bad = _expand(ids, tables, dtype)
    ref, ref_bad = oracle.expand_embed(ids, tables)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref), f"{case}: {np.count_nonzero(got != ref)} elements differ"
    assert bad == ref_bad == 0


@pytest.mark.parametrize("dtype,Dm", [("bf16", 64), ("bf16", 10), ("bf16", 7), ("f32", 5)])
def test_expand_out_of_range_ids(dtype, Dm):
    """Ids outside [0, V) give n zero rows and are counted once per token, after the
    count the caller zeroed; the in-range tokens around them are unaffected."""
    B, L, n, V = 3, 41, 3, 120
    seed = synth.seed_for("expand_bad", dtype, Dm)
    print(f"expand bad ids dtype={dtype} Dm={Dm} seed={seed}", flush=True)
    ids = synth.token_ids(seed, B, L, V)
    bad_at = [(0, 0, -1), (0, 40, V), (1, 7, -2 ** 31), (2, 13, 2 ** 31 - 1), (2, 14, V + 5),
              (1, 40, -7)]
    for b, t, x in bad_at:
        ids[b, t] = x
    tables = _tables(seed + 1, n, V, Dm, dtype)
    got, bad = _expand(ids, tables, dtype)
    ref, ref_bad = oracle.expand_embed(ids, tables)
    assert ref_bad == len(bad_at)
    assert bad == ref_bad
    assert np.array_equal(got, ref)
    for b, t, _ in bad_at:
        assert not got[b, t * n:(t + 1) * n].any(), "an out-of-range id must give zero rows"
    # a second call adds to the count: the library increments, the caller zeroes
    tids = torch.from_numpy(ids).to(G.dev())
    cnt = torch.full((1,), 5, dtype=torch.int32, device=G.dev())
    hd.expand_embed(tids, G.to_dev(tables), bad_id_count=cnt)
    torch.cuda.synchronize()
    assert int(cnt.cpu()[0]) == 5 + len(bad_at)


def test_expand_without_a_count():
    """bad_id_count may be null: out-of-range ids still give zero rows."""
    B, L, n, V, Dm = 2, 30, 4, 90, 64
    seed = synth.seed_for("expand_nocount")
    ids = synth.token_ids(seed, B, L, V)
    ids[0, 3] = V
    ids[1, 29] = -1
    tables = _tables(seed + 1, n, V, Dm, "bf16")
    got, _ = _expand(ids, tables, "bf16", count_bad=False)
    ref, ref_bad = oracle.expand_embed(ids, tables)
    assert ref_bad == 2
    assert np.array_equal(got, ref)


@pytest.mark.slow
def test_expand_stack_shape():
    """The 36-layer workload's expansion: 4096 ids uniform in [0, 151936) through n=4
    bf16 tables of 151936 x 4096 (N(0, 0.02^2), drawn by torch's seeded device
    generator: a host draw of 2.5e9 normals takes minutes), every one of the 16384
    expanded rows compared with the oracle on host copies of the same tables.  A few
    ids are set to the first and last rows of the tables and two out of range."""
    B, L, n = 1, workloads.QWEN8B.shape.L, workloads.QWEN8B.shape.n
    V, Dm = workloads.STACK_VOCAB, workloads.STACK_DMODEL
    seed = synth.seed_for("expand_stack")
    print(f"expand stack shape L={L} n={n} V={V} Dm={Dm} seed={seed}", flush=True)
    ids = synth.token_ids(seed, B, L, V)
    ids[0, :4] = [0, V - 1, 0, V - 1]
    ids[0, 100] = V
    ids[0, L - 1] = -3
    tables = synth.device_normal((n, V, Dm), workloads.STACK_EMBED_STD, seed + 1, G.dev(),
                                 torch.bfloat16)
    bad = torch.zeros(1, dtype=torch.int32, device=G.dev())
    out = hd.expand_embed(torch.from_numpy(ids).to(G.dev()), tables, bad_id_count=bad)
    torch.cuda.synchronize()
    got = G.bits(out)
    host_tables = G.bits(tables)
    del tables
    ref, ref_bad = oracle.expand_embed(ids, host_tables)
    assert ref_bad == 2 and int(bad.cpu()[0]) == 2
    assert np.array_equal(got, ref), f"{np.count_nonzero(got != ref)} elements differ"
