"""The error model behind the training parity bar, checked on the CPU: on
seeded small layers, an emulation of the path's fp16 roundings lands within
four predicted standard deviations of the fp64 oracle for each scale
gradient, and not far inside one (the model does not overstate the error
by orders of magnitude either)."""
import numpy as np
import pytest

from paper_2609_06161_amd import synth
from rounding_model import emulate_gradients, rounding_noise

SHAPES = [(32, 64, 32, 279), (32, 32, 32, 45), (64, 160, 64, 78), (128, 96, 256, 54),
          (224, 224, 32, 118), (256, 320, 96, 200), (96, 128, 160, 123), (160, 192, 96, 293)]


@pytest.mark.parametrize("m,n,r,T", SHAPES)
def test_emulated_rounding_error_within_model(oracle, m, n, r, T):
    seed = 7000 + m + 3 * n + 5 * r + T
    lin = synth.make_linear(seed, m, n, r, T)
    dy = synth.make_output_grad(seed + 1, T, m)
    ref = oracle.backward(m, n, r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid, lin.s_in, lin.x, dy)[1:]
    sigma = rounding_noise(oracle, lin, dy)
    for name, got, want, s in zip(("ds_out", "ds_mid", "ds_in"),
                                  emulate_gradients(oracle, lin, dy), ref, sigma):
        err = float(np.linalg.norm(got - want))
        assert 0.05 * s <= err <= 4 * s, (name, err, s)
