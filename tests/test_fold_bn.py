"""BN folding (fcm_fold_batchnorm): a convolution followed by inference batch
normalisation equals the convolution with folded weights and bias. Checked on the CPU
oracle in float64 against the normalisation applied explicitly after it (DW and PW), plus
hand values and the rejections."""
import numpy as np
import pytest

import oracle
from paper_2404_19331_amd import fcm


def _bn(y, gamma, beta, mean, var, eps, axis):
    shp = [1] * y.ndim
    shp[axis] = -1
    r = lambda a: np.asarray(a, np.float64).reshape(shp)
    return (y - r(mean)) / np.sqrt(r(var) + eps) * r(gamma) + r(beta)


@pytest.mark.parametrize("kind", ["dw", "pw"])
def test_folded_conv_equals_conv_then_batchnorm(kind):
    rng = np.random.default_rng(5)
    n, h, w, ci, co = 2, 7, 6, 12, 12 if kind == "dw" else 20
    x = rng.standard_normal((n, ci, h, w))
    wt = rng.standard_normal((ci, 3, 3) if kind == "dw" else (co, ci)).astype(np.float32)
    b = rng.standard_normal(co).astype(np.float32)
    gamma, beta = rng.uniform(0.5, 2, co), rng.standard_normal(co)
    mean, var = rng.standard_normal(co), rng.uniform(0.1, 3, co)
    eps = 1e-3
    case = dict(n=n, h=h, w=w, c_in=ci, c_mid=ci, c_out=co, k=3 if kind == "dw" else 1, stride=1,
                pad=1 if kind == "dw" else 0, dtype="f64", layout="nchw", act=["none"] * 3)
    run = oracle.dw if kind == "dw" else oracle.pw
    ref = _bn(run(case, x, wt.astype(np.float64), b.astype(np.float64)), gamma, beta, mean, var, eps, 1)
    wf, bf = fcm.fold_batchnorm(wt, b, gamma, beta, mean, var, eps)
    got = run(case, x, wf.astype(np.float64), bf.astype(np.float64))
    assert np.allclose(got, ref, rtol=1e-5, atol=1e-5)  # folded parameters are float32


def test_fold_hand_values_and_no_bias():
    # gamma 2, var 3 + eps 1 -> scale 1; mean 4, beta 5: w unchanged, b' = (b - 4) + 5
    wf, bf = fcm.fold_batchnorm(np.array([[1.5, -2.0]]), np.array([0.25]), [2.0], [5.0], [4.0], [3.0], eps=1.0)
    assert wf.tolist() == [[1.5, -2.0]] and bf.tolist() == [1.25]
    wf, bf = fcm.fold_batchnorm(np.array([[1.0]]), None, [1.0], [0.0], [2.0], [0.25], eps=0.0)
    assert wf.tolist() == [[2.0]] and bf.tolist() == [-4.0]  # scale 1/sqrt(0.25) = 2


def test_fold_rejects_bad_statistics():
    with pytest.raises(fcm.FcmError):
        fcm.fold_batchnorm(np.ones((1, 1)), None, [1.0], [0.0], [0.0], [0.0], eps=0.0)   # var + eps = 0
    with pytest.raises(fcm.FcmError):
        fcm.fold_batchnorm(np.ones((1, 1)), None, [1.0], [0.0], [0.0], [1.0], eps=-1.0)  # eps < 0
    with pytest.raises(ValueError):
        fcm.fold_batchnorm(np.ones((2, 1)), None, [1.0], [0.0], [0.0], [1.0])           # one statistic short
