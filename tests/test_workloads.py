"""The seeded input generators (CPU only): shapes, determinism, their own
real harmonics against scipy's, and the bf16 rounding helper."""

import numpy as np
import pytest

import workloads as W
from oracle.sh import real_sph_harm


def test_real_ylm_matches_scipy():
    x = np.random.default_rng(0).normal(size=(200, 3))
    assert np.abs(W.real_ylm(8, x) - real_sph_harm(8, x)).max() < 1e-13


@pytest.mark.parametrize("name", ["tiny", "nbody", "molecule"])
def test_small_workloads_shapes_and_determinism(name):
    w = W.WORKLOADS[name]
    q, k = W.make(name)
    assert q.shape == (w["B"], w["N"], (w["L"] + 1) ** 2, w["C"])
    assert q.dtype == np.float32 and k.dtype == np.float32
    q2, k2 = W.make(name)
    assert (q == q2).all() and (k == k2).all()
    assert not np.array_equal(q, k)


def test_molecule_padding_rows_are_zero():
    w = W.WORKLOADS["molecule"]
    q, k, n_real = W.molecule(w["B"], w["N"], w["L"], w["C"], w["seed"])
    assert ((n_real >= 9) & (n_real <= 29)).all()
    for b, n in enumerate(n_real):
        assert (q[b, n:] == 0).all() and (k[b, n:] == 0).all()
        assert np.abs(q[b, :n]).sum() > 0


def test_pointcloud_generator_small():
    q, k = W.pointcloud(2, 512, 3, 4, 77)
    assert q.shape == (2, 512, 16, 4)
    # features are Y(n) * w_c: every channel is a multiple of channel 0
    Y = q[0, :, :, 0]
    for c in range(1, 4):
        ratio = q[0, :, :, c] / np.where(Y == 0, 1, Y)
        assert np.allclose(ratio[np.abs(Y) > 1e-3], ratio[np.abs(Y) > 1e-3].flat[0], rtol=1e-5)
    # Y_00 is constant: 1/sqrt(4 pi)
    assert np.allclose(q[0, :, 0, 0] / q[0, 0, 0, 0], 1.0, rtol=1e-6)


def test_bf16_rounding():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.0e-5, 65504.0], dtype=np.float32)
    b = W.to_bf16_bits(x)
    back = W.bf16_bits_to_f32(b)
    # ties go to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> 1
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == np.float32(1.0 + 2 ** -6)
    assert back[3] == -2.5
    assert np.all(np.abs(back - x) <= np.abs(x) * 2 ** -8)
