"""The seeded input generators: reproducibility, distributions and bf16 rounding (CPU only)."""
import numpy as np
import torch

from paper_2311_10770_amd import synth
from paper_2311_10770_amd.configs import HEADLINE, WORKLOADS


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, -3.0e38, 1e-40, np.inf, -np.inf],
                                 dtype=np.float32)])
    # halfway cases: low 16 bits exactly 0x8000, both parities of bit 16
    halves = (np.arange(1000, dtype=np.uint32) << 16 | 0x8000).view(np.float32)
    a = np.concatenate([a, halves])
    ours = synth.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = synth.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(a).to(torch.bfloat16).float().numpy())


def test_generators_are_seeded_and_shaped():
    a = synth.make_layer(3, 64, 768, 4, 2, "bf16", "bf16")
    b = synth.make_layer(3, 64, 768, 4, 2, "bf16", "bf16")
    for k in a:
        assert np.array_equal(a[k], b[k])
    assert a["x"].shape == (64, 768) and a["x"].dtype == np.uint16
    assert a["w_in"].shape == (2, 31, 768)
    c = synth.make_layer(3, 64, 768, 4, 2, "f32", "f32", layer=1)
    assert not np.array_equal(synth.f32_to_bf16_bits(c["x"]), a["x"])


def test_weight_variance_is_one_over_h():
    w_in, w_out = synth.make_weights(2, 768, 8, 1, "f32")
    assert abs(w_in.var() * 768 - 1.0) < 0.01
    assert abs(w_out.var() * 768 - 1.0) < 0.01
    x = synth.make_x(2, 4096, 768, "f32")
    assert abs(x.var() - 1.0) < 0.01


def test_prefix_property_of_x():
    big = synth.make_x(5, 64, 128, "bf16")
    small = synth.make_x(5, 8, 128, "bf16")
    # standard_normal fills row-major, so a smaller draw is NOT a prefix; callers slice the big draw.
    assert big[:8].shape == small.shape


def test_workload_table():
    w = WORKLOADS[HEADLINE]
    assert (w.n_tokens, w.hidden, w.depth, w.n_trees) == (65536, 768, 11, 1)
    assert w.nodes == 4095
    assert w.gathered_bytes_per_token() == 12 * 2 * 768 * 2
    assert WORKLOADS["d15_h4096_bf16"].nodes == 65535


def test_kxd_family_is_table1():
    """The swept shapes are exactly Table 1's UltraFastBERT-KxD models, with its N_T."""
    from paper_2311_10770_amd.configs import KXD_FAMILY, kxd_workload
    from tests.conftest import read_table

    table = {(int(r[1]), int(r[2])): int(r[3]) for r in read_table("table1_neuron_counts.txt")}
    assert set(KXD_FAMILY) == set(table)
    for k, d in KXD_FAMILY:
        w = kxd_workload(k, d)
        assert w.n_trees * w.nodes == table[(k, d)]
        assert w.n_trees == k and w.depth == d and w.n_tokens == 16384 and w.hidden == 768
        assert w.gathered_bytes_per_token() == k * (d + 1) * 2 * 768 * 2
