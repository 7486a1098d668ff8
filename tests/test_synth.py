"""Pins for the seeded input generator (CPU only)."""
import numpy as np
import pytest
import torch

import synth

M64 = 2**64 - 1


def _splitmix64_reference(seed, k):
    # SplitMix64 from its published definition, written independently of synth.c.
    z = (seed + (k + 1) * 0x9E3779B97F4A7C15) & M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def test_splitmix64_published_values():
    # First two outputs of the reference SplitMix64 generator started at state 0.
    assert synth.splitmix64(0, 0) == 0xE220A8397B1DCDAF
    assert synth.splitmix64(0, 1) == 0x6E789E6AA1B965F4


@pytest.mark.parametrize("seed", [1, 3003, 2**63 + 12345])
def test_splitmix64_matches_definition(seed):
    for k in [0, 1, 2, 17, 1000, 2**40]:
        assert synth.splitmix64(seed, k) == _splitmix64_reference(seed, k)


def test_normal_box_muller_definition():
    seed = 77
    got = synth.normal(seed, (6,), 1.0, "f64")
    for i in range(6):
        p = i // 2
        u1 = (_splitmix64_reference(seed, 2 * p) >> 11) * 2.0**-53
        u2 = (_splitmix64_reference(seed, 2 * p + 1) >> 11) * 2.0**-53
        r = np.sqrt(-2.0 * np.log(1.0 - u1))
        th = 2.0 * np.pi * u2
        want = r * (np.sin(th) if i % 2 else np.cos(th))
        assert abs(got[i] - want) <= 1e-15 * max(1.0, abs(want))


def test_normal_moments_and_sigma():
    x = synth.normal(5, (1 << 20,), 3.0, "f64")
    assert abs(x.mean()) < 0.02
    assert abs(x.std() - 3.0) < 0.02
    # fourth standardised moment of a normal is 3
    assert abs(((x / x.std()) ** 4).mean() - 3.0) < 0.05


def test_storage_roundings():
    n = 1 << 16
    x64 = synth.normal(9, (n,), 1.0, "f64")
    x32 = synth.normal(9, (n,), 1.0, "f32")
    xbf = synth.normal(9, (n,), 1.0, "bf16")
    assert np.array_equal(x32, x64.astype(np.float32))
    # bf16 is round-to-nearest-even of the fp32 value; torch's conversion is RNE too.
    want = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(xbf, want)
    assert np.array_equal(synth.f32_to_bf16_bits(x32), want)
    back = synth.bf16_bits_to_f32(xbf)
    assert np.array_equal(back, torch.from_numpy(x32).to(torch.bfloat16).float().numpy())


def test_deterministic_and_seed_dependent():
    a = synth.normal(11, (4, 5), 1.0, "bf16")
    b = synth.normal(11, (4, 5), 1.0, "bf16")
    c = synth.normal(12, (4, 5), 1.0, "bf16")
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c)


def test_workloads_shapes():
    w = synth.WORKLOADS["single_head_f32_n128_d64"]
    q, k, v = synth.make_inputs(w)
    assert q.shape == (1, 1, 128, 64) and q.dtype == np.float32
    assert k.shape == (1, 1, 128, 64) and v.shape == (1, 1, 128, 64)
    assert len(set(w.seeds())) == 3
    names = [x.name for x in synth.WORKLOADS.values()]
    assert len(names) == 5
    d = synth.WORKLOADS["decode_b64h32_nk8192_d128_bf16"]
    assert (d.Nq, d.Nk, d.dk, d.causal) == (1, 8192, 128, False)
    assert synth.WORKLOADS["causal_long_b1h32_n16384_d128_bf16_qk_sigma3"].sigma_qk == 3.0
