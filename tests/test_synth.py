"""Seeded input generator: known answers, determinism, distributions."""
import numpy as np

import synth


def test_philox_known_answers():
    # Known-answer vectors of Philox4x32-10 published with the generator
    # (Salmon et al., SC'11, Random123 distribution).
    kat = [
        ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
        ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
        ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
         [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
    ]
    for ctr, key, want in kat:
        assert synth.philox4x32(ctr, key).tolist() == want


def test_normal_is_index_pure_and_seeded():
    a = synth.normal(7, 3, (1001,))
    b = synth.normal(7, 3, (990,), start=11)
    assert np.array_equal(a[11:], b)
    assert not np.array_equal(a, synth.normal(8, 3, (1001,)))
    assert not np.array_equal(a, synth.normal(7, 4, (1001,)))
    bf = synth.normal(7, 3, (1001,), dtype="bf16")
    # bf16 values are the RNE rounding of the float32 values
    f = synth.bf16_bits_to_f32(bf)
    assert np.all(np.abs(f - a) <= np.abs(a) * 2.0 ** -8 + 1e-30)


def test_normal_moments():
    x = synth.normal(0, 13, (2_000_000,), std=0.02).astype(np.float64)
    assert abs(x.mean()) < 0.02 * 4 / np.sqrt(x.size)
    assert abs(x.std() / 0.02 - 1) < 3e-3
    # fourth moment of a normal is 3 sigma^4
    assert abs(np.mean((x / 0.02) ** 4) - 3.0) < 0.05


def test_uniform_int_range_and_balance():
    t = synth.uniform_int(11, 61, 400_000, 0, 4096)
    assert t.min() >= 0 and t.max() < 4096
    counts = np.bincount(t, minlength=4096)
    assert counts.min() > 40 and counts.max() < 170
    lens = synth.context_lengths(10_000, 1024, 2048, 2)
    assert lens.min() == 1024 and lens.max() == 2048


def test_zipf_bias_is_a_ranked_log():
    b = synth.zipf_router_bias(synth.FULL, 1.1)
    assert b.shape == (12, 64)
    for l in range(12):
        ranks = np.rint(np.exp(-b[l].astype(np.float64) / 1.1)).astype(int)
        assert sorted(ranks.tolist()) == list(range(1, 65))
    assert not np.array_equal(b[0], b[1])


def test_weight_shapes_and_init():
    cfg = synth.TINY
    w = synth.make_weights(cfg, 0, 1)
    for name, shp in synth.weight_shapes(cfg).items():
        assert w[name].shape == shp
    assert "lm_head" not in w                      # tied
    assert np.all(w["final_norm"] == 1.0)
    assert abs(w["wqkv"].std() - 0.02) < 1e-3
    # the draft block draws from its own seed
    w2 = synth.make_weights(cfg, 0, 2)
    assert np.array_equal(w["wqkv"], w2["wqkv"])
    assert not np.array_equal(w["d_wqkv"], w2["d_wqkv"])
