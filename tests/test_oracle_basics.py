"""Pins of the oracle's rounding, random numbers and residual quantiser.

Each test checks the oracle against something other than itself: library
conversions, published known-answer vectors, textbook identities of the
Hadamard matrix, distributional facts, or properties the quantiser's
definition implies.
"""
import numpy as np
import pytest
import scipy.linalg
import scipy.stats
import torch

from conftest import golden
from oracle import philox, residual, rounding
from oracle.alloc import calibrate_eps2


# ----------------------------------------------------------------------------- rounding
def test_fp16_matches_numpy_conversion(rng):
    x = rng.standard_normal(200_000) * np.exp(rng.uniform(-25, 12, 200_000))
    # include exact ties between neighbouring fp16 values and overflow edges
    base = rng.standard_normal(5000).astype(np.float16).astype(np.float64)
    ulp = np.spacing(np.abs(base).astype(np.float16)).astype(np.float64)
    ties = base + 0.5 * ulp * np.sign(base)
    extra = np.array([65504.0, 65519.99, 65520.0, -65520.0, 1e-8, 2.0 ** -25, 3 * 2.0 ** -26, 0.0])
    for v in (x, ties, extra):
        with np.errstate(over="ignore"):
            ref = v.astype(np.float16).astype(np.float64)
        np.testing.assert_array_equal(rounding.to_fp16(v), ref)


def test_bf16_matches_torch_conversion(rng):
    x32 = (rng.standard_normal(200_000) * np.exp(rng.uniform(-80, 80, 200_000))).astype(np.float32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(rounding.to_bf16(x32.astype(np.float64)), ref)


def test_ceil_log2_exact_at_powers_of_two():
    for k in range(-30, 30):
        assert rounding.ceil_log2(2.0 ** k) == k
        assert rounding.ceil_log2(2.0 ** k * 1.0000001) == k + 1
        assert rounding.ceil_log2(2.0 ** k * 0.9999999) == k


# ----------------------------------------------------------------------------- philox
def test_philox_known_answer_vectors():
    for v in golden("philox4x32_10_kat.json")["vectors"]:
        ctr = [np.uint64(int(c, 16)) for c in v["ctr"]]
        key = [int(k, 16) for k in v["key"]]
        out = philox.philox4x32_10(*ctr, *key)
        assert ["%08x" % int(o) for o in out] == v["out"]


def test_signs_deterministic_and_balanced():
    s = philox.rotation_signs(7, 1 << 16)
    assert set(np.unique(s)) == {-1.0, 1.0}
    assert abs(s.mean()) < 0.02
    np.testing.assert_array_equal(s, philox.rotation_signs(7, 1 << 16))
    assert (philox.rotation_signs(8, 128) != philox.rotation_signs(7, 128)).any()


def test_sketch_is_bf16_standard_normal():
    om = philox.sketch_matrix(3, 512, 200)
    np.testing.assert_array_equal(rounding.to_bf16(om), om)
    ks = scipy.stats.kstest(om.ravel(), "norm")
    assert ks.pvalue > 1e-3
    # columns depend only on (row, column): a wider sketch extends a narrower one
    np.testing.assert_array_equal(philox.sketch_matrix(3, 512, 50), om[:, :50])
    assert not np.array_equal(philox.sketch_matrix(4, 512, 200), om)


def test_calibration_samples_gaussian():
    z = philox.calibration_samples(0, 1 << 16)
    assert scipy.stats.kstest(z, "norm").pvalue > 1e-3
    np.testing.assert_array_equal(rounding.to_fp32(z), z)


# ----------------------------------------------------------------------------- rotation
@pytest.mark.parametrize("d", [1, 2, 8, 64, 128, 256])
def test_sylvester_hadamard(d):
    H = residual.sylvester_hadamard(d)
    np.testing.assert_array_equal(H, scipy.linalg.hadamard(d))
    np.testing.assert_array_equal(H @ H.T, d * np.eye(d))


def test_rotation_orthogonal_and_invertible(rng):
    d = 128
    s = philox.rotation_signs(1, d)
    r = rng.standard_normal((50, d)) * np.exp(rng.uniform(-3, 3, (50, 1)))
    rp = residual.rotate(r, s)
    np.testing.assert_allclose(np.linalg.norm(rp, axis=1), np.linalg.norm(r, axis=1), rtol=1e-13)
    np.testing.assert_allclose(residual.unrotate(rp, s), r, atol=1e-12 * np.abs(r).max())
    # explicit matrix form: r' = (H diag(s) / sqrt(d)) r
    M = scipy.linalg.hadamard(d) @ np.diag(s) / np.sqrt(d)
    np.testing.assert_allclose(rp, r @ M.T, atol=1e-12 * np.abs(r).max())


def test_rotation_spreads_outlier_channel():
    d = 128
    r = np.zeros((1, d))
    r[0, 5] = 10.0
    rp = residual.rotate(r, philox.rotation_signs(0, d))
    np.testing.assert_allclose(np.abs(rp), 10.0 / np.sqrt(d), rtol=1e-14)


# ----------------------------------------------------------------------------- quantiser
@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantizer_properties(rng, bits):
    g = 64
    x = rng.standard_normal((40, 128)) * np.exp(rng.uniform(-4, 4, (40, 1)))
    codes, scales = residual.quantize(x, bits, g)
    L = (1 << bits) - 1
    assert codes.min() >= 0 and codes.max() <= L
    np.testing.assert_array_equal(rounding.to_fp16(scales), scales)      # fp16 scales
    xh = residual.dequantize(codes, scales, bits, g)
    err = np.abs(x - xh).reshape(40, 2, g)
    amax = np.abs(x).reshape(40, 2, g).max(-1)
    # inside the representable range the error is at most half a step; the
    # range edge a may exceed the outer level by the fp16 rounding of Delta
    lim = np.maximum(scales / 2, amax - (L / 2) * scales)
    assert (err <= lim[..., None] * (1 + 1e-12) + 1e-300).all()
    # monotone: a larger value never gets a smaller code within a group
    grp = x[0, :g]
    order = np.argsort(grp)
    assert (np.diff(codes[0, :g][order].astype(int)) >= 0).all()


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantizer_grid_points_roundtrip_exactly(bits):
    g, L = 64, (1 << bits) - 1
    delta = 0.375                                   # fp16-exact step
    k = np.arange(g) % (L + 1)
    k[0], k[1] = 0, L                               # extremes present: a = (L/2) delta
    x = ((k - L / 2.0) * delta)[None, :]
    codes, scales = residual.quantize(x, bits, g)
    assert scales[0, 0] == delta
    np.testing.assert_array_equal(codes[0], k)
    np.testing.assert_array_equal(residual.dequantize(codes, scales, bits, g), x)


def test_quantizer_zero_group():
    codes, scales = residual.quantize(np.zeros((1, 128)), 4, 64)
    assert (codes == 8).all() and (scales == 0).all()
    assert (residual.dequantize(codes, scales, 4, 64) == 0).all()


def test_pack_lsb_first():
    assert residual.pack(np.array([1, 2, 3, 0], np.uint8), 2).tolist() == [0b00111001]
    assert residual.pack(np.array([0xA, 0x5], np.uint8), 4).tolist() == [0x5A]
    c = np.random.default_rng(0).integers(0, 16, 4096).astype(np.uint8)
    np.testing.assert_array_equal(residual.unpack(residual.pack(c, 4), 4, c.size), c)


def test_eps2_monotone_and_rotation_invariant():
    """eq. (2): eps^2(0) = 1 and eps^2 decreasing in b.  Because the rotation is
    orthogonal and maps iid Gaussian rows to iid Gaussian rows, the calibrated
    value must equal the plain quantisation error of unrotated iid Gaussian
    groups (estimated here from numpy's own generator) within Monte-Carlo error."""
    e = calibrate_eps2(group=64, d=128, seed=0, n_samples=1 << 20)
    assert e[0] == 1.0 and 1.0 > e[2] > e[4] > e[8] > 0.0
    z = np.random.default_rng(99).standard_normal((1 << 14, 64))
    for b in (2, 4, 8):
        codes, sc = residual.quantize(z, b, 64)
        ref = np.sum((residual.dequantize(codes, sc, b, 64) - z) ** 2) / np.sum(z * z)
        assert abs(e[b] / ref - 1.0) < 0.03, (b, e[b], ref)


# ------------------------------------------------------------------ rotary embedding (appendix B)
def test_rope_two_features_is_a_plane_rotation():
    """d = 2: one pair with frequency base^0 = 1, so position p turns the row by p radians."""
    from oracle.rope import rope
    x = np.array([[0.3, -1.7], [2.0, 0.5], [-0.4, 0.9]])
    p = np.array([0.0, 1.0, 7.5])
    got = rope(x, 1e4, p)
    for r in range(3):
        c, s = np.cos(p[r]), np.sin(p[r])
        want = np.array([[c, -s], [s, c]]) @ x[r]
        np.testing.assert_allclose(got[r], want, rtol=0, atol=1e-15)


def test_rope_keeps_norms_and_inverts():
    from oracle.rope import rope
    rng = np.random.default_rng(4)
    X = rng.standard_normal((3, 50, 128))
    pos = np.arange(50) + 1000.0
    Y = rope(X, 1e6, pos)
    np.testing.assert_allclose(np.linalg.norm(Y, axis=-1), np.linalg.norm(X, axis=-1), rtol=1e-13)
    np.testing.assert_allclose(rope(Y, 1e6, -pos), X, rtol=0, atol=1e-12)
    np.testing.assert_allclose(rope(X, 1e6, np.zeros(50)), X, rtol=0, atol=0)


def test_rope_scores_depend_only_on_relative_position():
    """The defining property: <rope(q, p1), rope(k, p2)> depends on p2 - p1 alone."""
    from oracle.rope import rope
    rng = np.random.default_rng(5)
    q, k = rng.standard_normal((1, 64)), rng.standard_normal((1, 64))
    for p1, p2, shift in ((3, 10, 500), (0, 4000, 77), (123, 45, 9999)):
        a = float((rope(q, 1e4, [p1]) @ rope(k, 1e4, [p2]).T)[0, 0])
        b = float((rope(q, 1e4, [p1 + shift]) @ rope(k, 1e4, [p2 + shift]).T)[0, 0])
        assert abs(a - b) <= 1e-9 * (abs(a) + 1)
