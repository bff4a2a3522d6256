"""Pins of the oracle's RoPE strip / re-apply (content-space mapping, Sec. 3.3).

Each check uses something other than the oracle's own formula: the complex
exponential form of RoPE, dense rotation matrices inverted numerically, the
relative-position property, orthogonality, and the published Llama 3.1
frequency rescaling rule evaluated band by band.
"""

import math

import numpy as np
import pytest

from oracle import kvx_oracle as O

ROPES = [
    O.Rope(1e4), O.Rope(1e6), O.Rope(5e5, factor=8.0), O.Rope(1e4, style=1),
    O.Rope(5e5, style=1, factor=8.0),
]


def _x(rng, T, d, lead=()):
    return rng.standard_normal(lead + (T, d))


@pytest.mark.parametrize("rope", ROPES)
@pytest.mark.parametrize("d", [8, 64, 128])
def test_strip_then_apply_is_identity(rope, d):
    rng = np.random.default_rng(0)
    T = 37
    x = _x(rng, T, d, (3,))
    pos = rng.integers(0, 70000, size=T)
    y = O.rope_rotate(O.rope_rotate(x, pos, rope, inverse=True), pos, rope)
    assert np.max(np.abs(y - x)) < 1e-12
    y2 = O.rope_rotate(O.rope_rotate(x, pos, rope), pos, rope, inverse=True)
    assert np.max(np.abs(y2 - x)) < 1e-12


@pytest.mark.parametrize("rope", ROPES)
def test_position_zero_is_identity(rope):
    rng = np.random.default_rng(1)
    x = _x(rng, 5, 64)
    assert np.array_equal(O.rope_rotate(x, np.zeros(5, int), rope), x)


@pytest.mark.parametrize("rope", ROPES)
def test_norm_of_each_plane_is_preserved(rope):
    rng = np.random.default_rng(2)
    d, T = 64, 11
    x = _x(rng, T, d)
    pos = rng.integers(0, 40000, size=T)
    y = O.rope_rotate(x, pos, rope)
    if rope.style == 0:
        a, b = np.arange(d // 2), np.arange(d // 2) + d // 2
    else:
        a, b = np.arange(0, d, 2), np.arange(1, d, 2)
    np.testing.assert_allclose(x[:, a] ** 2 + x[:, b] ** 2,
                               y[:, a] ** 2 + y[:, b] ** 2, rtol=1e-12)


@pytest.mark.parametrize("rope", ROPES)
def test_rotations_compose_additively(rope):
    rng = np.random.default_rng(3)
    x = _x(rng, 9, 128)
    p = rng.integers(0, 30000, size=9)
    q = rng.integers(0, 30000, size=9)
    two = O.rope_rotate(O.rope_rotate(x, p, rope), q, rope)
    one = O.rope_rotate(x, p + q, rope)
    assert np.max(np.abs(two - one)) < 1e-9


def _base_freq(theta, d):
    return np.array([theta ** (-(2.0 * j) / d) for j in range(d // 2)])


@pytest.mark.parametrize("theta,style", [(1e4, 0), (1e6, 0), (1e4, 1)])
def test_matches_complex_exponential_form(theta, style):
    """RoPE is multiplication of each plane, read as u + i v, by exp(i p w_j)."""
    rng = np.random.default_rng(4)
    d, T = 128, 23
    x = _x(rng, T, d)
    pos = rng.integers(0, 65536, size=T)
    w = _base_freq(theta, d)
    if style == 0:
        z = x[:, : d // 2] + 1j * x[:, d // 2:]
    else:
        z = x[:, 0::2] + 1j * x[:, 1::2]
    z = z * np.exp(1j * pos[:, None] * w[None, :])
    want = np.empty_like(x)
    if style == 0:
        want[:, : d // 2], want[:, d // 2:] = z.real, z.imag
    else:
        want[:, 0::2], want[:, 1::2] = z.real, z.imag
    got = O.rope_rotate(x, pos, O.Rope(theta, style=style))
    assert np.max(np.abs(got - want)) < 1e-10


def test_relative_position_property():
    """<R(p) q, R(r) k> depends on p - r only (the defining RoPE property)."""
    rng = np.random.default_rng(5)
    d = 64
    rope = O.Rope(1e4)
    q = rng.standard_normal((1, d))
    k = rng.standard_normal((1, d))
    base = None
    for p, r in [(10, 3), (107, 100), (5007, 5000)]:
        v = float((O.rope_rotate(q, [p], rope) @ O.rope_rotate(k, [r], rope).T)[0, 0])
        base = v if base is None else base
        assert abs(v - base) < 1e-9


def test_base_frequencies():
    w = O.rope_inv_freq(O.Rope(1e4), 128)
    assert w.shape == (64,)
    assert w[0] == 1.0
    np.testing.assert_allclose(w[1:] / w[:-1], 1e4 ** (-2.0 / 128), rtol=1e-13)
    np.testing.assert_allclose(w[-1], 1e4 ** (-126.0 / 128), rtol=1e-13)


def test_llama3_rescaling_bands():
    """Published Llama 3.1 rule: short wavelengths kept, long ones divided by
    the factor, a linear blend in wavelength-ratio space in between."""
    d, theta, factor, C = 128, 5e5, 8.0, 8192
    base = _base_freq(theta, d)
    got = O.rope_inv_freq(O.Rope(theta, factor=factor, low_freq_factor=1.0,
                                  high_freq_factor=4.0, original_max_pos=C), d)
    wl = 2 * math.pi / base
    keep = wl < C / 4.0
    scaled = wl > C / 1.0
    mid = ~keep & ~scaled
    # band counts for theta 5e5, d 128
    assert keep.sum() == 29 and scaled.sum() == 29 and mid.sum() == 6
    np.testing.assert_allclose(got[keep], base[keep], rtol=1e-15)
    np.testing.assert_allclose(got[scaled], base[scaled] / factor, rtol=1e-15)
    # blend endpoints: s = 1 at C/wl = high, s = 0 at C/wl = low
    s = (C / wl[mid] - 1.0) / (4.0 - 1.0)
    assert np.all((s > 0) & (s < 1))
    np.testing.assert_allclose(got[mid], base[mid] / factor * (1 - s) + base[mid] * s,
                               rtol=1e-14)
    assert np.all(np.diff(got) < 0)          # still strictly decreasing
    assert np.all(got <= base * (1 + 1e-15)) and np.all(got >= base / factor * (1 - 1e-15))


def test_dense_matrix_form_is_orthogonal_and_matches():
    """Build R(t) as a dense d x d matrix from its plane definition; the oracle's
    rotation must equal R x, and R^T must be R^-1."""
    rng = np.random.default_rng(6)
    d = 16
    for style in (0, 1):
        rope = O.Rope(1e4, style=style)
        w = _base_freq(1e4, d)
        p = 1234
        R = np.zeros((d, d))
        for j in range(d // 2):
            a, b = (j, j + d // 2) if style == 0 else (2 * j, 2 * j + 1)
            c, s = math.cos(p * w[j]), math.sin(p * w[j])
            R[a, a], R[a, b], R[b, a], R[b, b] = c, -s, s, c
        np.testing.assert_allclose(R @ R.T, np.eye(d), atol=1e-14)
        x = rng.standard_normal(d)
        np.testing.assert_allclose(O.rope_rotate(x[None], [p], rope)[0], R @ x, atol=1e-13)
        np.testing.assert_allclose(O.rope_rotate(x[None], [p], rope, inverse=True)[0],
                                   np.linalg.solve(R, x), atol=1e-13)


def _hf_inv_freq(rope_type, theta, d, scaling=None):
    """Frequencies from the transformers library's own RoPE initialisers, built
    offline from an in-process config (no download).  transformers works in
    float32, so comparisons allow float32 rounding."""
    torch = pytest.importorskip("torch")
    rope_utils = pytest.importorskip("transformers.modeling_rope_utils")
    from transformers import LlamaConfig
    params = {"rope_type": rope_type, "factor": 1.0}
    if scaling:
        params.update(scaling)
    cfg = LlamaConfig(hidden_size=8 * d, num_attention_heads=8, head_dim=d, rope_theta=theta,
                      max_position_embeddings=131072, rope_scaling=params)
    inv, _ = rope_utils.ROPE_INIT_FUNCTIONS[rope_type](cfg, "cpu")
    return inv.to(torch.float64).numpy()


@pytest.mark.parametrize("theta", [1e4, 5e5, 1e6])
@pytest.mark.parametrize("d", [64, 128])
def test_base_frequencies_match_transformers(theta, d):
    """omega_j = theta^(-2j/d) as an independent library computes it."""
    want = _hf_inv_freq("linear", theta, d)
    np.testing.assert_allclose(O.rope_inv_freq(O.Rope(theta), d), want, rtol=2e-6)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("theta", [5e5, 1e6])
def test_llama3_rule_matches_transformers(theta, d):
    """The Llama 3.1 band rule (factor 8, low 1, high 4, context 8192) against
    the transformers library's implementation of it.  Every band is covered at
    d = 128, theta = 5e5: 29 kept, 6 blended, 29 divided."""
    scaling = {"factor": 8.0, "low_freq_factor": 1.0, "high_freq_factor": 4.0,
               "original_max_position_embeddings": 8192}
    want = _hf_inv_freq("llama3", theta, d, scaling)
    got = O.rope_inv_freq(O.Rope(theta, factor=8.0, low_freq_factor=1.0, high_freq_factor=4.0,
                                 original_max_pos=8192), d)
    np.testing.assert_allclose(got, want, rtol=2e-6)
    # the rescaling really changed something, so the comparison is not vacuous
    assert np.abs(got / O.rope_inv_freq(O.Rope(theta), d) - 1).max() > 0.5


def test_llama3_rule_other_parameters_match_transformers():
    """A second parameter set (factor 32, low 2, high 8, context 4096), so that
    no constant of the published default hides in the oracle."""
    scaling = {"factor": 32.0, "low_freq_factor": 2.0, "high_freq_factor": 8.0,
               "original_max_position_embeddings": 4096}
    want = _hf_inv_freq("llama3", 5e5, 128, scaling)
    got = O.rope_inv_freq(O.Rope(5e5, factor=32.0, low_freq_factor=2.0, high_freq_factor=8.0,
                                 original_max_pos=4096), 128)
    np.testing.assert_allclose(got, want, rtol=2e-6)
