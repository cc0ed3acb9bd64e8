"""Tolerances for comparing the HIP path with the oracle.

Conv / FC: a layer passes when both hold
  (i)  max |gpu - oracle| <= 1e-4 * sqrt(Kred), Kred = (C/G)*R*S or I;
  (ii) ||gpu - oracle||_2 / ||oracle||_2 <= 1e-4.
Pooling indices and max values, ReLU: bit-exact on identical inputs.
Average pooling and LRN: elementwise relative 1e-5 (plus an absolute floor
of 1e-6 times the input's largest magnitude for results that cancel to ~0).
"""
import math

import numpy as np


def assert_gemm_close(gpu, ref, kred, what=""):
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU output"
    err = np.abs(g - r)
    atol = 1e-4 * math.sqrt(kred)
    assert err.max(initial=0.0) <= atol, f"{what}: max abs err {err.max():.3e} > {atol:.3e}"
    nr = np.linalg.norm(r)
    if nr > 0:
        rel = np.linalg.norm(g - r) / nr
        assert rel <= 1e-4, f"{what}: relative L2 err {rel:.3e} > 1e-4"
    return float(err.max(initial=0.0))


def assert_elementwise_close(gpu, ref, x_absmax, what="", rtol=1e-5):
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    np.testing.assert_allclose(g, r, rtol=rtol, atol=1e-6 * max(float(x_absmax), 1e-30),
                               err_msg=what)
