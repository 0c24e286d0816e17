"""GPU parity of the expansion backward (sparse table gradient), its dense
scatter-add and the cyclic replication of the tables, against the fp64 oracle.

Integer outputs (the distinct ids and their count) must be bit-exact.  The gradient
rows are fp32 sums, in ascending token order, of k upstream values (bf16 or fp32
inputs, exact in fp32): each partial sum is rounded once, so
|gpu - exact| <= (k - 1) * 2^-24 * sum_i |x_i| per element; the tests use that bound with
k the largest run length of the batch and sum_i |x_i| from the oracle applied to |dout|.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_08186_amd as hd
from paper_2607_08186_amd import synth, workloads
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


def _dout(seed, B, N, Dm, dtype):
    x = synth.normal(seed, (B, N, Dm), 1.0)
    return synth.to_bf16_bits(x) if dtype == "bf16" else x.astype(np.float32)


def _as_f64(a):
    return synth.bf16_bits_to_f32(a).astype(np.float64) if a.dtype == np.uint16 else a.astype(
        np.float64)


def _run(ids, dout, V):
    tids = torch.from_numpy(ids).to(G.dev())
    tdout = G.to_dev(dout)
    uniq, drows, num = hd.expand_embed_backward(tids, tdout, V)
    torch.cuda.synchronize()
    k = int(num.cpu()[0])
    return uniq.cpu().numpy()[:k], drows.cpu().numpy()[:, :k], k


def _check(ids, dout, V):
    print(f"expand_bwd ids={ids.shape} dout={dout.shape} V={V} dtype={dout.dtype}", flush=True)
    uniq, drows, k = _run(ids, dout, V)
    valid = ids[(ids >= 0) & (ids < V)]
    want_ids, counts = np.unique(valid, return_counts=True)
    assert k == len(want_ids)
    np.testing.assert_array_equal(uniq, want_ids.astype(np.int32))
    if k == 0:
        return
    ref = oracle.expand_embed_bwd_rows(ids, dout, V, want_ids)            # [k][n][Dm]
    mag = oracle.expand_embed_bwd_rows(ids, np.abs(_as_f64(dout)), V, want_ids)
    got = np.transpose(drows, (1, 0, 2)).astype(np.float64)               # [k][n][Dm]
    kmax = int(counts.max())
    tol = max(kmax - 1, 0) * U32 * mag + 1e-30
    err = np.abs(got - ref)
    assert np.all(err <= tol), f"max err {err.max():.3e}, run length up to {kmax}"
    if kmax == 1:  # single-token runs are copies: exact
        np.testing.assert_array_equal(got, ref)


CASES = [
    # B, L, n, V, Dm, dtype
    (1, 64, 2, 50, 64, "bf16"),          # many repeats, one sort pass
    (2, 300, 4, 1000, 96, "bf16"),       # B=2, two passes
    (1, 2049, 3, 7, 40, "f32"),          # one chunk + 1 token, heavy repeats
    (3, 1000, 2, 151936, 16, "bf16"),    # the 151936-token vocabulary: three passes
    (1, 100, 1, 100000, 12, "f32"),      # Dm not a multiple of 8 (scalar path), n = 1
    (1, 5000, 2, 1 << 20, 8, "bf16"),
    (1, 300, 2, 2 ** 31 - 1, 8, "bf16"),  # ids over the whole int32 range: four passes
    (1, 1, 3, 10, 32, "bf16"),           # a single token
    (1, 16384, 2, 151936, 16, "bf16"),   # the largest batch of the one-pass counting sort
    (1, 16385, 2, 151936, 16, "bf16"),   # the smallest one of the radix sort
    (2, 8500, 1, 1000, 2056, "f32"),     # radix sort with heavy repeats; rows of 1+ chunks
]


@pytest.mark.parametrize("B,L,n,V,Dm,dtype", CASES, ids=[str(c) for c in CASES])
def test_expand_bwd_parity(B, L, n, V, Dm, dtype):
    seed = synth.seed_for("expand_bwd", B, L, n, V, Dm, dtype)
    ids = synth.token_ids(seed, B, L, V)
    _check(ids, _dout(seed + 1, B, n * L, Dm, dtype), V)


def test_expand_bwd_out_of_range_ids_are_dropped():
    B, L, n, V, Dm = 2, 700, 3, 64, 24
    seed = synth.seed_for("expand_bwd_bad")
    ids = synth.token_ids(seed, B, L, V + 40) - 20  # about 1/3 outside [0, V)
    assert np.any(ids < 0) and np.any(ids >= V)
    _check(ids, _dout(seed + 1, B, n * L, Dm, "bf16"), V)


@pytest.mark.parametrize("V", [(1 << 18) - 1, 1 << 18])
def test_expand_bwd_sort_key_packing_boundary(V):
    """The counting sort packs (id, token) into one 32-bit word while every key fits 18
    bits (V < 2^18, the out-of-range marker V included) and compares the two parts
    otherwise: ids near the top of [0, V), repeats and out-of-range ids on both sides of
    that boundary."""
    B, L, n, Dm = 2, 1500, 2, 16
    seed = synth.seed_for("expand_bwd_pack", V)
    ids = synth.token_ids(seed, B, L, 64) + (V - 48)  # 48 in range at the top, 16 at or past V
    ids[0, :7] = -1
    assert np.any(ids >= V) and np.any(ids == V - 1) and np.any(ids < 0)
    _check(ids, _dout(seed + 1, B, n * L, Dm, "bf16"), V)


def test_expand_bwd_all_ids_equal_and_all_bad():
    B, L, n, Dm = 1, 3000, 2, 32
    seed = synth.seed_for("expand_bwd_same")
    _check(np.full((B, L), 5, dtype=np.int32), _dout(seed, B, n * L, Dm, "f32"), 9)
    _check(np.full((B, L), -3, dtype=np.int32), _dout(seed, B, n * L, Dm, "f32"), 9)


def test_expand_bwd_distinct_ids_copy_rows():
    B, L, n, V, Dm = 1, 4096, 4, 151936, 64
    seed = synth.seed_for("expand_bwd_perm")
    ids = np.random.default_rng(seed).permutation(V)[:L].astype(np.int32).reshape(B, L)
    _check(ids, _dout(seed, B, n * L, Dm, "bf16"), V)


def test_expand_bwd_deterministic():
    B, L, n, V, Dm = 2, 2500, 4, 300, 128
    seed = synth.seed_for("expand_bwd_det")
    ids = torch.from_numpy(synth.token_ids(seed, B, L, V)).to(G.dev())
    dout = G.to_dev(_dout(seed, B, n * L, Dm, "bf16"))
    a = hd.expand_embed_backward(ids, dout, V)
    b = hd.expand_embed_backward(ids, dout, V)
    torch.cuda.synchronize()
    k = int(a[2].cpu()[0])
    assert k == int(b[2].cpu()[0])
    assert torch.equal(a[0][:k], b[0][:k]) and torch.equal(a[1][:, :k], b[1][:, :k])


def test_grad_scatter_add_into_dense_tables():
    B, L, n, V, Dm = 1, 900, 2, 120, 40
    seed = synth.seed_for("scatter_add")
    ids = synth.token_ids(seed, B, L, V + 10) - 5
    dout = _dout(seed + 1, B, n * L, Dm, "bf16")
    init = synth.normal(seed + 2, (n, V, Dm), 1.0).astype(np.float32)
    tids = torch.from_numpy(ids).to(G.dev())
    uniq, drows, num = hd.expand_embed_backward(tids, G.to_dev(dout), V)
    dtab = torch.from_numpy(init.copy()).to(G.dev())
    hd.hd_embed_grad_scatter_add(uniq, drows, num, B * L, n, V, Dm, dtab)
    torch.cuda.synchronize()
    ref = oracle.expand_embed_bwd(ids, dout, V)
    mag = oracle.expand_embed_bwd(ids, np.abs(_as_f64(dout)), V)
    kmax = int(np.unique(ids[(ids >= 0) & (ids < V)], return_counts=True)[1].max())
    got = dtab.cpu().numpy().astype(np.float64)
    want = init.astype(np.float64) + ref
    # one rounding of the run sum (bounded above) plus one of the final addition
    tol = max(kmax - 1, 0) * U32 * mag + U32 * (np.abs(init) + mag) * 2 + 1e-30
    assert np.all(np.abs(got - want) <= tol)
    untouched = np.setdiff1d(np.arange(V), ids)
    np.testing.assert_array_equal(got[:, untouched], init[:, untouched].astype(np.float64))


@pytest.mark.parametrize("n,m,V,Dm,dtype", [(2, 4, 37, 64, "bf16"), (4, 8, 100, 48, "f32"),
                                             (1, 3, 3, 5, "bf16"), (3, 3, 10, 8, "f32")])
def test_cyclic_replicate_bitexact(n, m, V, Dm, dtype):
    seed = synth.seed_for("cyclic", n, m, V, Dm, dtype)
    x = synth.normal(seed, (n, V, Dm), 0.02)
    tables = synth.to_bf16_bits(x) if dtype == "bf16" else x.astype(np.float32)
    out = hd.cyclic_replicate(G.to_dev(tables), m)
    torch.cuda.synchronize()
    want = oracle.cyclic_replicate(tables, m)
    got = G.bits(out) if dtype == "bf16" else out.cpu().numpy()
    np.testing.assert_array_equal(got, want)


def test_cyclic_replicate_in_place_growth():
    """One buffer with room for m tables: the first n are kept, the rest filled."""
    n, m, V, Dm = 2, 8, 50, 32
    x = synth.to_bf16_bits(synth.normal(synth.seed_for("cyclic_inplace"), (n, V, Dm), 0.02))
    buf = torch.zeros((m, V, Dm), dtype=torch.bfloat16, device=G.dev())
    buf[:n] = G.to_dev(x)
    hd.hd_cyclic_replicate(buf, buf, n, m, V, Dm)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(G.bits(buf), oracle.cyclic_replicate(x, m))


@pytest.mark.slow
def test_expand_bwd_fullsize_stack_shape():
    """The 36-layer stack's expansion: B=1, L=4096 ids over 151936 tokens, n=4 streams
    of width 4096 (bf16).  Sampled distinct ids against the oracle; every row against
    the column sums of its stream (the sum over distinct ids of the gradient rows is the
    sum of that stream's upstream rows)."""
    s = workloads.QWEN8B.shape
    V, Dm = workloads.STACK_VOCAB, workloads.STACK_DMODEL
    seed = synth.seed_for("expand_bwd_full")
    ids = synth.token_ids(seed, 1, s.L, V)
    dout = _dout(seed + 1, 1, s.N, Dm, "bf16")
    print(f"expand_bwd fullsize L={s.L} n={s.n} V={V} Dm={Dm}", flush=True)
    uniq, drows, k = _run(ids, dout, V)
    want_ids, counts = np.unique(ids, return_counts=True)
    assert k == len(want_ids)
    np.testing.assert_array_equal(uniq, want_ids.astype(np.int32))
    rng = np.random.default_rng(seed)
    pick = np.unique(np.concatenate([rng.choice(k, 40, replace=False),
                                     np.flatnonzero(counts > 1)[:20], [0, k - 1]]))
    ref = oracle.expand_embed_bwd_rows(ids, dout, V, want_ids[pick])
    mag = oracle.expand_embed_bwd_rows(ids, np.abs(_as_f64(dout)), V, want_ids[pick])
    got = np.transpose(drows[:, pick], (1, 0, 2)).astype(np.float64)
    tol = max(int(counts.max()) - 1, 0) * U32 * mag + 1e-30
    assert np.all(np.abs(got - ref) <= tol)
    x = _as_f64(dout)[0]
    for st in range(s.n):
        col = x[st::s.n].sum(axis=0)
        tot = drows[st].astype(np.float64).sum(axis=0)
        assert np.allclose(tot, col, rtol=0, atol=1e-3 * np.abs(x[st::s.n]).sum(axis=0).max())
