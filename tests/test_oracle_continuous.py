"""Pins of the continuous-time EventProp model (test-only oracle).

The exact EventProp gradients of Table 1 (weights and delays, with the delayed
postsynaptic adjoints in the lambda_V jump) must equal central finite
differences of the exactly simulated loss.  A dropped theta term, a swapped
(lambda_V - lambda_I) sign, adjoints taken at the emission instead of the
arrival time, or a wrong denominator all break these equalities.
"""
import math

import pytest

from oracle.continuous import ContNet


def _cmp(g, f, rtol=2e-6, atol=1e-9):
    for ga, fa in zip(g, f):                 # dW, dD
        for gp, fp in zip(ga, fa):           # projections
            for gr, fr in zip(gp, fp):       # rows
                for x, y in zip(gr, fr):
                    assert abs(x - y) <= atol + rtol * abs(y), (x, y)


@pytest.mark.parametrize("w1,T,nspk", [(10.0, 60.0, 1), (25.0, 80.0, 5)])
def test_chain_eventprop_equals_fd(w1, T, nspk):
    net = ContNet([1, 1, 1], [(0, 1, [[w1]], [[2.0]]), (1, 2, [[1.5]], [[3.0]])], T=T)
    inp = [(1.0, 0)]
    L, rec = net.forward(inp)
    assert len(rec["spikes"]) == nspk
    _cmp(net.backward(inp, rec), net.fd(inp, h=1e-6), rtol=5e-6)


def test_recurrent_delays_two_readouts_integral_loss():
    W_in = [[6.0, 4.5], [3.0, 7.0]]
    D_in = [[1.3, 4.1], [2.2, 0.7]]
    W_rec = [[0.0, 2.5], [1.8, 0.0]]
    D_rec = [[0.5, 3.3], [6.1, 1.1]]
    W_out = [[1.2, -0.7], [0.4, 0.9]]
    D_out = [[2.5, 0.9], [3.7, 5.2]]
    net = ContNet([2, 2, 2], [(0, 1, W_in, D_in), (1, 1, W_rec, D_rec), (1, 2, W_out, D_out)],
                  T=70.0)
    inp = [(0.5, 0), (3.1, 1), (9.4, 0), (17.2, 1)]
    c = [0.8, -1.3]
    L, rec = net.forward(inp, "integral", c)
    assert len(rec["spikes"]) >= 4
    _cmp(net.backward(inp, rec), net.fd(inp, "integral", c, h=1e-6), rtol=2e-5, atol=1e-8)


def test_max_voltage_loss_source_at_tmax():
    W_in = [[9.0]]
    D_in = [[1.5]]
    W_out = [[1.1, 0.6]]
    D_out = [[2.0, 6.5]]
    net = ContNet([1, 1, 2], [(0, 1, W_in, D_in), (1, 2, W_out, D_out)], T=60.0)
    inp = [(2.0, 0)]
    c = [1.0, -0.5]
    L, rec = net.forward(inp, "max", c)
    assert len(rec["spikes"]) >= 1
    _cmp(net.backward(inp, rec), net.fd(inp, "max", c, h=1e-6), rtol=2e-5, atol=1e-8)


def test_time_translation_identity():
    """Shifting every input delay by eps shifts the whole trajectory, so with an
    integral readout sum_ij dL/dd_ij (input projection) = -sum_k c_k V_k(T)."""
    W_in = [[8.0, 3.0]]
    D_in = [[1.0, 2.5]]
    W_out = [[1.0], [0.5]]
    D_out = [[2.0], [1.0]]
    net = ContNet([1, 2, 1], [(0, 1, W_in, D_in), (1, 2, W_out, D_out)], T=40.0)
    inp = [(1.0, 0)]
    L, rec = net.forward(inp, "integral", [1.0])
    dW, dD = net.backward(inp, rec)
    # V_out(T) from the derivative of L with respect to T
    h = 1e-6
    net.T = 40.0 + h
    Lp, _ = net.forward(inp, "integral", [1.0])
    net.T = 40.0 - h
    Lm, _ = net.forward(inp, "integral", [1.0])
    VT = (Lp - Lm) / (2 * h)
    assert abs(sum(dD[0][0]) + VT) <= 1e-6 * abs(VT) + 1e-9
