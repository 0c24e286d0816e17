"""The seeded input generator: determinism and bf16 rounding (checked against torch)."""
import numpy as np
import torch

from paper_2607_08186_amd import synth


def test_bf16_rounding_matches_torch():
    x = synth.normal(1, (4096,), 3.0).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8]  # ties to even both ways
    ours = synth.to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = synth.bf16_bits_to_f32(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_inputs_deterministic_and_shaped():
    a = synth.sfa_inputs(1, 8, 2, 4, 2, 16, seed=5)
    b = synth.sfa_inputs(1, 8, 2, 4, 2, 16, seed=5)
    assert a["q"].shape == (1, 16, 4, 16) and a["k"].shape == (1, 16, 2, 16)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
    c = synth.sfa_inputs(1, 8, 2, 4, 2, 16, seed=6)
    assert not np.array_equal(a["q"], c["q"])


def test_k_spike_rows_exact():
    base = synth.sfa_inputs(1, 100, 4, 2, 8, 16, seed=9)
    spk = synth.sfa_inputs(1, 100, 4, 2, 8, 16, seed=9, k_spike=(0.01, 8.0))
    a = synth.bf16_bits_to_f32(base["k"]).reshape(-1, 16)
    b = synth.bf16_bits_to_f32(spk["k"]).reshape(-1, 16)
    changed = np.where(np.any(a != b, axis=1))[0]
    assert len(changed) == int(0.01 * a.shape[0])  # 32 of 3200 rows
    np.testing.assert_array_equal(b[changed], a[changed] * 8)
