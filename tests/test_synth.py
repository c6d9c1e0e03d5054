"""Seeded workload generators and the selector-cache microscale encoders."""
import numpy as np

import oracle
from paper_2606_22874_amd import synth
from paper_2606_22874_amd.synth import bf16_bits, bf16_value


def test_bf16_rounding_is_rne():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 3.0e38],
                 dtype=np.float32)
    got = bf16_value(bf16_bits(x))
    want = np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5, 2.9913e38], dtype=np.float32)
    np.testing.assert_array_equal(got[:5], want[:5])
    assert abs(got[5] / 3.0e38 - 1) < 2 ** -8


def test_e2m1_rounding_ties_to_even():
    """OCP MX v1.0 E2M1 grid 0, .5, 1, 1.5, 2, 3, 4, 6 with RNE ties."""
    y = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 7.0, 0.3, 2.9, 6.0])
    grid = synth.E2M1_GRID[synth._e2m1_rne(y)]
    np.testing.assert_array_equal(grid, [0, 1, 1, 2, 2, 4, 4, 6, 0.5, 3, 6])


def test_mxfp4_encoder():
    x = np.zeros((1, 64), np.float32)
    x[0, :32] = np.linspace(-6, 6, 32)
    x[0, 32:] = np.linspace(-0.9, 1.0, 32)
    codes, e8 = synth.quantize_mxfp4_g32(bf16_bits(x))
    # amax 6 -> X = floor(log2 6) - 2 = 0 -> E8M0 127; amax 1 -> X = -2 -> 125.
    np.testing.assert_array_equal(e8[0], [127, 125])
    vals = oracle.key_values(codes, e8, "mxfp4", 64)
    xv = bf16_value(bf16_bits(x))[0].astype(np.float64)
    # Error at most half a grid step (grid step <= 2 * 2^X).
    step = np.repeat(np.ldexp(1.0, e8.astype(np.int64) - 127)[0], 32)
    assert np.all(np.abs(vals - xv) <= step + 1e-12)
    # An all-zero group encodes to E8M0 0 and zero codes.
    codes, e8 = synth.quantize_mxfp4_g32(np.zeros((2, 32), np.uint16))
    assert np.all(e8 == 0) and np.all(codes == 0)


def test_int4_encoder():
    rng = np.random.default_rng(1)
    x = bf16_bits(rng.standard_normal((50, 64)).astype(np.float32))
    codes, scales = synth.quantize_int4_g32(x)
    assert codes.shape == (50, 32) and scales.shape == (50, 2)
    vals = oracle.key_values(codes, scales, "int4", x.size).reshape(50, 64)
    xv = bf16_value(x).astype(np.float64)
    sc = np.repeat(scales.view(np.float16).astype(np.float64), 32, axis=-1)
    amax = np.repeat(np.abs(xv).reshape(50, 2, 32).max(-1), 32, axis=-1)
    assert np.all(np.abs(vals - xv) <= sc / 2 + amax * 2.0 ** -10)
    nib = np.stack([codes & 15, codes >> 4], -1)
    assert not np.any(nib == 8)           # codes stay within [-7, 7]
    codes, scales = synth.quantize_int4_g32(np.zeros((1, 32), np.uint16))
    assert np.all(codes == 0) and np.all(scales == 0)


def test_int8_encoder():
    rng = np.random.default_rng(2)
    x = bf16_bits(rng.standard_normal((50, 64)).astype(np.float32))
    codes, scales = synth.quantize_int8_g32(x)
    assert codes.shape == (50, 64) and scales.shape == (50, 2)
    vals = oracle.key_values(codes, scales, "int8", x.size).reshape(50, 64)
    xv = bf16_value(x).astype(np.float64)
    sc = np.repeat(scales.view(np.float16).astype(np.float64), 32, axis=-1)
    amax = np.repeat(np.abs(xv).reshape(50, 2, 32).max(-1), 32, axis=-1)
    assert np.all(np.abs(vals - xv) <= sc / 2 + amax * 2.0 ** -10)
    assert not np.any(codes.view(np.int8) == -128)   # codes stay within [-127, 127]
    codes, scales = synth.quantize_int8_g32(np.zeros((1, 32), np.uint16))
    assert np.all(codes == 0) and np.all(scales == 0)


def test_mxfp8_encoder():
    rng = np.random.default_rng(3)
    x = bf16_bits(rng.standard_normal((50, 64)).astype(np.float32))
    codes, e8 = synth.quantize_mxfp8_g32(x)
    assert codes.shape == (50, 64) and e8.shape == (50, 2)
    vals = oracle.key_values(codes, e8, "mxfp8", x.size).reshape(50, 64)
    xv = bf16_value(x).astype(np.float64)
    amax = np.repeat(np.abs(xv).reshape(50, 2, 32).max(-1), 32, axis=-1)
    # E4M3 keeps 3 fraction bits: within half a step of 2^-3 relative, or of
    # the smallest subnormal step (2^-9 of the scale) near zero
    X = e8.astype(np.int64) - 127
    s2 = np.repeat(np.ldexp(1.0, X), 32, axis=-1)
    sat = np.abs(xv) / s2 > 448                       # OCP MX: saturate at the max
    step = np.maximum(np.abs(xv) * 2.0 ** -3, amax * 2.0 ** -8 * 2.0 ** -9)
    assert np.all(np.abs(vals - xv)[~sat] <= step[~sat] / 2 + 1e-30)
    np.testing.assert_array_equal(vals[sat], np.sign(xv[sat]) * 448 * s2[sat])
    # the group maximum lands in [256, 512) after the scale
    top = np.abs(xv).reshape(50, 2, 32).max(-1) / np.ldexp(1.0, X)
    assert np.all((top >= 256) & (top < 512))
    assert np.all((codes & 0x7F) != 0x7F)            # no NaN codes
    # ties go to the even code: 1 + 1/16 lies halfway between codes 0x38 and 0x39
    c = synth._e4m3_rne(np.array([1.0625, 1.1875]))
    assert list(c) == [0x38, 0x3A]


def test_footprint_matches_paper():
    """Section 5.3: 4.50 GiB BF16 -> 1.27 GiB INT4 and 1.20 GiB FP4 (0.281x)."""
    ds = 64
    bf16 = 2 * ds
    int4 = ds // 2 + 2 * (ds // 32)
    mxfp4 = ds // 2 + 1 * (ds // 32)
    assert abs(int4 / bf16 - 0.281) < 5e-4
    assert round(4.50 * int4 / bf16, 2) == 1.27
    assert round(4.50 * mxfp4 / bf16, 2) == 1.20


def test_generators_deterministic():
    a = synth.decode_config(2, B=2, L=4096)
    b = synth.decode_config(2, B=2, L=4096)
    for f in ("q_sel", "w", "k_sel", "q", "k", "v"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    k1 = synth.normal_bf16(5, 2, (3, 2, 64, 8))
    k2 = synth.normal_bf16(5, 2, (3, 2, 64, 8))
    np.testing.assert_array_equal(k1, k2)


def _budgets(wl):
    s = oracle.selector_score(wl.q_sel, wl.w, wl.k_sel, n_valid=wl.n_valid)
    return oracle.select_blocks(s.astype(np.float32), wl.rule, wl.n_valid)


def test_realised_budgets():
    """Zipf workloads: ~21-22 blocks mass-terminated (L=32K), cap-bound at 128K."""
    _, cnt, mass = _budgets(synth.decode_config(2, backbone=False))
    assert 17 <= cnt.mean() <= 26 and np.all(mass >= 0.9)
    _, cnt, mass = _budgets(synth.decode_config(3, backbone=False))
    assert np.all(cnt == 128) and np.all(mass < 0.95)
    assert 0.65 < mass.mean() < 0.85
