"""Seeded random descriptors for the three normalisations (RMS, softmax,
layer), against the CPU oracle bit for bit (gfx950): leaf width and layout,
fold direction, the fma rule, output type, the pre-weight rounding, optional
weight and bias, and ragged rows and columns (including widths past the
one-pass kernels' 8192 columns)."""
import numpy as np
import pytest

import oracle
from paper_2609_11356_amd import inputs
from tests.gpu_util import assert_bits_equal
from tests import test_gpu_layernorm as ln
from tests import test_gpu_rmsnorm as rms
from tests import test_gpu_softmax as smx

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_11356_amd import dg as _dg
    _dg.lib()
    return _dg


def draw(seed, kind):
    rng = np.random.default_rng(80_000 + 3 * seed + ("rms", "smx", "ln").index(kind))
    desc = {}
    if rng.random() < 0.6:
        desc.update(leaf_layout="strided", leaf_w=int(rng.choice([8, 32, 64, 128, 256])),
                    lane_fold=str(rng.choice(["up", "down"])))
    else:
        desc["leaf_w"] = int(rng.choice([1, 7, 64, 100]))
    if kind != "smx" and rng.random() < 0.3:
        desc["fma"] = 0
    if rng.random() < 0.5:
        desc["out"] = "bf16"
        if kind != "smx" and rng.random() < 0.5:
            desc["norm_round"] = "pre_weight"
    rows = int(rng.choice([1, 3, 64, 130]))
    cols = int(rng.choice([1, 17, 256, 1000, 4096, 8192, 8200]))
    X = inputs.lognormal_f32(91_000 + 3 * seed, (rows, cols))
    w = inputs.normal_bf16(92_000 + seed, (cols,), 1.0) if rng.random() < 0.7 else None
    b = inputs.normal_bf16(93_000 + seed, (cols,), 1.0) if rng.random() < 0.7 else None
    eps = float(rng.choice([0.0, 1e-6, 1e-5]))
    return desc, X, w, b, eps


@pytest.mark.parametrize("kind", ["rms", "smx", "ln"])
@pytest.mark.parametrize("seed", range(24))
def test_norm_random_descriptor(dg, seed, kind):
    desc, X, w, b, eps = draw(seed, kind)
    print("%s seed %d shape %s desc %s w %s b %s eps %g" % (kind, seed, X.shape, desc, w is not None,
                                                          b is not None, eps), flush=True)
    if kind == "rms":
        got, want = rms.run(dg, desc, X, w, eps), oracle.rmsnorm(desc, X, w, eps=eps)
    elif kind == "smx":
        got, want = smx.run(dg, desc, X), oracle.softmax(desc, X)
    else:
        got, want = ln.run(dg, desc, X, w, b, eps), oracle.layernorm(desc, X, w, b, eps=eps)
    assert_bits_equal(got, want, "%s seed %d %s" % (kind, seed, desc))
