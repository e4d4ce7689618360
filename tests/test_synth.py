"""Host-side checks of the seeded input generator (no GPU)."""
import numpy as np
import torch

import synth
from synth import workloads as wl


def test_splitmix64_reference_outputs():
    # first outputs of SplitMix64 from state 0 (published reference sequence)
    got = [int(x) for x in synth.draw_u64(0, [0, 1, 2])]
    assert got == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3
    x[:4] = [1.00390625, 1.01171875, -1.00390625, 65504.0]     # ties and a large value
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_normal_moments_and_determinism():
    key = synth.stream_key(42, 3)
    a = synth.normal_f32(key, np.arange(400000), 0.5)
    b = synth.normal_f32(key, np.arange(400000), 0.5)
    np.testing.assert_array_equal(a, b)
    assert abs(a.mean()) < 3e-3 and abs(a.std() - 0.5) < 3e-3
    assert np.abs(a).max() <= 0.5 * 3.47
    c = synth.normal_f32(synth.stream_key(42, 4), np.arange(400000), 0.5)
    assert abs(np.corrcoef(a, c)[0, 1]) < 0.01


def test_uniform_int_and_bernoulli():
    key = synth.stream_key(7, 1)
    u = synth.uniform_int(key, np.arange(200000), 3, 9)
    assert u.min() == 3 and u.max() == 9
    assert np.all(np.abs(np.bincount(u - 3) / len(u) - 1 / 7) < 0.01)
    bern = synth.bernoulli(key, np.arange(200000), 0.25)
    assert abs(bern.mean() - 0.25) < 0.005


def test_geometric_accept_lengths():
    w = wl.RAGGED32
    m = np.concatenate([wl.accepted_lengths(w, r) for r in range(400)])
    assert m.min() >= 0 and m.max() <= w.B
    # truncated geometric: P(m = k) = (1-p)^k p for k < B, P(m = B) = (1-p)^B
    p = 0.25
    expect = sum(k * (1 - p) ** k * p for k in range(w.B)) + w.B * (1 - p) ** w.B
    assert abs(m.mean() - expect) < 0.15


def test_page_table_is_a_permutation():
    w = wl.RAGGED32.replace(rounds=4)
    pt = wl.page_table(w)
    assert sorted(pt.ravel().tolist()) == list(range(pt.size))


def test_anchors_sorted_distinct_in_range():
    a, u, a2 = wl.anchors(wl.TRAIN_FWD)
    assert a.shape == (8, 256) and u.shape == (8, 256) and a2.shape == (8, 256)
    for row in a:
        assert np.all(np.diff(row) > 0) and row[0] >= 0 and row[-1] <= 4096 - 16 - 1
    assert u.min() >= 0 and u.max() <= 16
    # shifted anchor: the next correction/bonus position, never past the response
    np.testing.assert_array_equal(a2, a + (16 - u) + 1)
    assert a2.min() >= 1 and a2.max() <= 4096


def test_grid_index_matches_layout():
    idx = synth.grid_index((2, 3, 4), (100, 10, 1), 5)
    assert idx[1, 2, 3] == 5 + 100 + 20 + 3


def test_c_host_generator_matches_numpy_definition():
    """The C build of the block generator gives the numpy definition's bits."""
    import synth
    if synth.host_lib() is None:
        synth.build_host()
    cases = [((3, 5, 7), (1000, 11, 1), 17), ((4, 2, 9, 16), (5000, 800, 16, 1), 123456789),
             ((64,), (3,), 0), ((2, 1, 130), (1 << 20, 7, 1), 5)]
    for shape, strides, base in cases:
        for dtype in ("f32", "bf16"):
            a = synth.normal_block(0x1234567890ABCDEF, shape, strides, base, 0.37, dtype, True)
            b = synth.normal_block(0x1234567890ABCDEF, shape, strides, base, 0.37, dtype, False)
            assert a.dtype == b.dtype and a.shape == b.shape
            np.testing.assert_array_equal(a.view(np.uint16 if dtype == "bf16" else np.uint32),
                                          b.view(np.uint16 if dtype == "bf16" else np.uint32))


def test_bf16_values_widened_in_c_match_numpy():
    """The C generator's bf16-as-fp32 mode gives the bf16 values, widened,
    bit for bit as the numpy definition."""
    import synth
    key = synth.stream_key(0xC0FFEE, 11)
    shape, strides = (3, 5, 70), (1 << 20, 131, 1)
    a = synth.normal_block(key, shape, strides, 777, 0.37, "bf16_f32")
    b = synth.bf16_bits_to_f32(synth.normal(key, synth.grid_index(shape, strides, 777), 0.37,
                                            "bf16"))
    assert a.dtype == np.float32
    np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))
