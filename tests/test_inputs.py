"""Seeded input generation and half-precision storage formats (CPU)."""
import numpy as np

from paper_2102_06725_amd import inputs as I


def test_fp16_quantisation_is_numpy_rne():
    v = np.array([0.0, 1.0, 1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, 65504.0, 65520.0, 1e-8, -2.5])
    bits = I.to_bits(v, I.F16)
    with np.errstate(over="ignore"):  # 65520 rounds to inf
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(bits, ref)
    # ties go to even: 1 + 2^-11 -> 1.0 ; 1 + 3*2^-11 -> 1 + 2^-9
    assert I.from_bits(bits, I.F16)[2] == 1.0
    assert I.from_bits(bits, I.F16)[3] == 1.0 + 2.0 ** -9
    assert np.isinf(I.from_bits(bits, I.F16)[5])


def test_bf16_round_to_nearest_even():
    ulp = 2.0 ** -7
    v = np.array([1.0, 1.0 + ulp / 2, 1.0 + 3 * ulp / 2, 1.0 + ulp / 2 + 2.0 ** -20,
                  -3.0, 3.4e38, np.inf, -np.inf], np.float64)
    got = I.from_bits(I.to_bits(v, I.BF16), I.BF16)
    assert got[0] == 1.0
    assert got[1] == 1.0                 # tie -> even mantissa (0)
    assert got[2] == 1.0 + 2 * ulp       # tie -> even mantissa (2)
    assert got[3] == 1.0 + ulp           # above the tie rounds up
    assert got[4] == -3.0
    assert np.isinf(got[5])              # overflows to inf, not saturation
    assert np.isinf(got[6]) and got[6] > 0 and np.isinf(got[7]) and got[7] < 0
    nan = I.to_bits(np.array([np.nan]), I.BF16)
    assert np.isnan(I.from_bits(nan, I.BF16)[0])


def test_bf16_exhaustive_representable_roundtrip():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = I.from_bits(bits, I.BF16)
    finite = np.isfinite(vals)
    assert np.array_equal(I.to_bits(vals[finite], I.BF16), bits[finite])


def test_seeds_reproduce_and_differ():
    a = I.draw(5, (4, 5), "normal")
    b = I.draw(5, (4, 5), "normal")
    c = I.draw(6, (4, 5), "normal")
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    assert np.all(I.from_bits(I.draw(1, (1000,), "absnormal"), I.F16) >= 0)


def test_resnet50_has_53_layers():
    layers = I.resnet50_layers(256)
    assert sum(c for _, c in layers) == 53
    assert len(layers) == 23
    stem = layers[0][0]
    assert (stem.p, stem.q) == (112, 112) and stem.c_alg == 3
    # conv forward FLOPs of one 224x224 image: sum over the 53 layers
    per_image = sum(l.with_batch(1).flops() * c for l, c in layers)
    assert abs(per_image / 1e9 - 8.17) < 0.02


def test_workload_tensors_layout_and_padding():
    wl = I.workload(4, batch=1)
    t = I.layer_tensors(wl, 0, 4)
    assert t["x"].shape == (1, 224, 224, 4)
    assert not t["x"][..., 3:].any() and not t["w"][..., 3:].any()
    wl1 = I.workload(1)
    t1 = I.layer_tensors(wl1, 0, 1)
    assert t1["x"].shape == (2, 16, 16, 16) and t1["dy"].shape == (2, 16, 16, 16)
