"""Pin of the oracle's update and momentum step: a 2-2-1 net worked by hand.

The paper prints no worked example.  This one applies the method as the paper
states it (sections 3, 4.1, 6.2.1 and 9) to the smallest net with a hidden
layer, with the readings that the oracle follows: summed change over the batch,
delta = e y (1 - y) from E = 1/2 sum e^2, reported error sum e^2, true unit as
the last weight row, classical momentum V = lr G + alpha V_prev, W += V.  The
numbers below were worked out step by step in 40-digit decimal arithmetic,
independently of the oracle's code, and agree to every printed digit with the
values derived the same way for the design survey of this library.

Net 2-2-1.  W0 rows: input 0, input 1, true unit; W1 rows: hidden 0, hidden 1,
true unit.

    W0 = [[0.1, -0.2], [0.3, 0.4], [0.0, 0.1]]    W1 = [0.5, -0.6, 0.2]
    batch of two patterns: (1, 0) -> 0.9 and (0, 1) -> 0.1
    lr = 0.5, momentum = 0.9, V = 0 at the start; two updates on that batch.

Update 1, pattern (1, 0):
    hidden net  (0.1, -0.1)          h = (0.524979187479, 0.475020812521)
    output net  0.177477106227       y = 0.544253179814
    e = 0.355746820186               d2 = e y (1 - y) = 0.088240030423
    d1 = h (1 - h) W1[:2] d2 = (0.011002474687, -0.013202969624)
Update 1, pattern (0, 1):
    hidden net  (0.3, 0.5)           h = (0.574442516812, 0.622459331202)
    output net  0.113745659685       y = 0.528405795164
    e = -0.428405795164              d2 = -0.106755772782
    d1 = (-0.013048667989, 0.015052801742)
Summed changes (G = sum over the batch of a_l d_{l+1}; bias row: sum of d):
    G1 = (-0.015000875327, -0.024535275980, -0.018515742359)
    G0 = [[0.011002474687, -0.013202969624], [-0.013048667989, 0.015052801742],
          [-0.002046193302, 0.001849832118]]
    error = 0.355746820186^2 + 0.428405795164^2 = 0.310087325402
    V = 0.5 G (V_prev = 0);  W += V.
Update 2 (same batch, now with the momentum term 0.9 V_prev):
    outputs 0.539882792972, 0.522589405314;  error = 0.308266208281
    G1 = (-0.013307142910, -0.023469055785, -0.015975225946)
    V1 = 0.5 G1 + 0.9 V1_prev = (-0.013403965352, -0.022775402083, -0.016319697035)

The oracle takes float32 targets, so 0.9 and 0.1 enter as 0.89999998 and
0.10000000149; that moves every value below by a few 1e-8, hence the
tolerance of 1e-7.
"""
import numpy as np

import oracle

SIZES = (2, 2, 1)
W_INIT = [0.1, -0.2, 0.3, 0.4, 0.0, 0.1, 0.5, -0.6, 0.2]   # flat: W0 row-major, then W1
X = np.array([[1.0, 0.0], [0.0, 1.0]], np.float32)
T = np.array([[0.9], [0.1]], np.float32)
LR, MOM = 0.5, 0.9
TOL = 1e-7

# (outputs before the update, error of the update, weights after, momentum after)
STEPS = [
    {
        "outputs": [0.544253179814, 0.528405795164],
        "sse": 0.310087325402,
        "W": [0.1055012373, -0.2066014848, 0.2934756660, 0.4075264009, -0.0010230967, 0.1009249161,
              0.4924995623, -0.6122676380, 0.1907421288],
        "V": [0.005501237343, -0.006601484812, -0.006524333994, 0.007526400871, -0.001023096651, 0.000924916059,
              -0.007500437663, -0.012267637990, -0.009257871180],
    },
    {
        "outputs": [0.539882792972, 0.522589405314],
        "sse": 0.308266208281,
        "W": [0.1159445097, -0.2193701562, 0.2812499604, 0.4218693806, -0.0028055300, 0.1024992244,
              0.4790955970, -0.6350430401, 0.1744224318],
        "V": [0.010443272328, -0.012768671375, -0.012225705653, 0.014342979695, -0.001782433325, 0.001574308320,
              -0.013403965352, -0.022775402083, -0.016319697035],
    },
]


def _run(storage):
    net = oracle.OracleNet(SIZES, storage)
    net.set_weights(np.array(W_INIT, np.float64))
    got = []
    for _ in STEPS:
        y = net.forward(x=X)[:, 0]
        sse = net.train_epoch(T, 2, LR, MOM, x=X)
        got.append((y, sse, net.get_weights(), net.get_momentum()))
    return got


def test_two_updates_match_hand_computed_steps():
    for k, ((y, sse, w, v), ref) in enumerate(zip(_run(64), STEPS)):
        np.testing.assert_allclose(y, ref["outputs"], rtol=0, atol=TOL, err_msg=f"outputs before update {k + 1}")
        assert abs(sse - ref["sse"]) <= TOL, (k + 1, sse, ref["sse"])
        np.testing.assert_allclose(w, ref["W"], rtol=0, atol=TOL, err_msg=f"weights after update {k + 1}")
        np.testing.assert_allclose(v, ref["V"], rtol=0, atol=TOL, err_msg=f"momentum after update {k + 1}")


def test_float_storage_tracks_hand_computed_steps():
    # float storage rounds a, delta, G, V and W to fp32: a few ulp of 0.6
    for k, ((y, sse, w, v), ref) in enumerate(zip(_run(32), STEPS)):
        np.testing.assert_allclose(y, ref["outputs"], rtol=0, atol=1e-6)
        assert abs(sse - ref["sse"]) <= 1e-6
        np.testing.assert_allclose(w, ref["W"], rtol=0, atol=1e-6)
        np.testing.assert_allclose(v, ref["V"], rtol=0, atol=1e-6)
