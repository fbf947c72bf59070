"""Pins of the hidden spike-count regulariser (CPU only).

The Results train the SHD/SSC/Braille models with a target of 14 spikes per
example and a layer-wise regularisation strength, and defer the formula to
earlier EventProp work.  Reading (the same in the oracle and the library):
with cbar_i the batch-mean spike count of neuron i of a regularised LIF layer,
the penalty is R = rho/2 sum_i (cbar_i - nu)^2, and every spike k of neuron i
adds dl_p/dt_k = -rho (cbar_i - nu) / B to the numerator of its lambda_V jump.
Counts are piecewise constant, so this is the gradient, with the counts held
fixed, of -(rho / B) sum_i (cbar_i - nu) sum_k t_k.

* Continuous time: EventProp with these terms equals central finite
  differences of that function (one sample), on a recurrent net.
* The terms and R by hand for a small record set.
* The reading's direction: plain gradient steps on the regulariser alone move
  the mean hidden count toward the target, from above and from below.
* A zero strength changes nothing, bit for bit.
"""
import numpy as np
import pytest

import oracle
from oracle.continuous import ContNet
from oracle.grid import ForwardResult
from workloads import make_workload

from .test_oracle_continuous import _cmp


def _rec_net(T=40.0):
    W_in, D_in = [[6.0, 4.5], [3.0, 7.0]], [[1.3, 4.1], [2.2, 0.7]]
    W_rec, D_rec = [[0.0, 2.5], [1.8, 0.0]], [[0.5, 3.3], [6.1, 1.1]]
    W_out, D_out = [[1.2, -0.7], [0.4, 0.9]], [[2.5, 0.9], [3.7, 5.2]]
    return ContNet([2, 2, 2], [(0, 1, W_in, D_in), (1, 1, W_rec, D_rec), (1, 2, W_out, D_out)], T=T)


INP = [(0.5, 0), (3.1, 1), (9.4, 0), (17.2, 1)]
C = [0.8, -1.3]


def test_regulariser_terms_equal_fd_in_continuous_time():
    net = _rec_net()
    kw = dict(spike_reg={1: (0.03, 4.0)})
    L, rec = net.forward(INP, "integral", C, **kw)
    counts = [sum(1 for s in rec["spikes"] if s[1] == 1 and s[2] == j) for j in range(2)]
    assert counts[0] != 4 and counts[1] != 4 and counts[0] != counts[1]
    g = net.backward(INP, rec)
    _cmp(g, net.fd(INP, "integral", C, h=1e-6, **kw), rtol=2e-5, atol=1e-8)
    L0, rec0 = net.forward(INP, "integral", C)
    g0 = net.backward(INP, rec0)
    assert abs(g[0][0][0][0] - g0[0][0][0][0]) > 1e-4        # the terms matter


def test_regulariser_terms_by_hand():
    """One LIF layer of 3 neurons, B = 2: records (neurons) [0, 0, 2] and
    [1, 0] give counts (3, 1, 1), cbar = (1.5, 0.5, 0.5); with nu = 1,
    rho = 2: R = 2/2 (0.25 + 0.25 + 0.25) = 0.75 and the per-neuron term
    -2 (cbar - 1) / 2 = (-0.5, 0.5, 0.5)."""
    net = oracle.OracleNet(((2, 0, 0), (3, 1, 0), (2, 2, 0)), 20.0, 5.0, 1.0, 1.0, 5, 10, 0, 0.1)
    cap = 4
    count = np.array([[3, 2]], np.int32)
    neuron = np.zeros((1, 2, cap), np.int32)
    neuron[0, 0, :3] = [0, 0, 2]
    neuron[0, 1, :2] = [1, 0]
    z = np.zeros((2, 2), np.float32)
    fwd = ForwardResult(0, count, np.zeros_like(neuron), neuron, np.zeros((1, 2, cap), np.float32), z,
                        np.zeros((2, 2), np.int32), np.zeros((2, 5), np.float32),
                        np.zeros((2, 5), np.float32), None, 0, cap)
    R, dlp = oracle.spike_count_reg(net, fwd, [2.0], 1.0)
    assert R == 0.75
    assert dlp[0, 0, :3].tolist() == [-0.5, -0.5, 0.5]
    assert dlp[0, 1, :2].tolist() == [0.5, -0.5]
    assert np.all(dlp[0, 0, 3:] == 0) and np.all(dlp[0, 1, 2:] == 0)
    R0, dlp0 = oracle.spike_count_reg(net, fwd, [0.0], 1.0)
    assert R0 == 0.0 and not dlp0.any()


def _reg_only_steps(nu, steps=3, rho=0.05, lr=2e-5):
    wl = make_workload(3, B=8)
    c = wl.cfg
    net = oracle.OracleNet(c.layers, c.tau_m, c.tau_s, c.theta, c.dt, c.max_delay, wl.T, c.loss,
                           c.readout_scale, list(c.delay_range))
    W = [w.copy() for w in wl.W]
    g = np.zeros((wl.B, c.n_classes), np.float32)        # the regulariser alone
    means = []
    for _ in range(steps + 1):
        f = oracle.forward(net, wl.in_off, wl.in_step, wl.in_neuron, W, wl.D, cap=300 * 128)
        means.append(float(f.count[0].sum()) / wl.B / 128)
        R, dlp = oracle.spike_count_reg(net, f, [rho], nu)
        dW, _, _ = oracle.backward(net, wl.in_off, wl.in_step, wl.in_neuron, W, wl.D, f, g, dlp=dlp)
        W = [(w - lr * d).astype(np.float32) for w, d in zip(W, dW)]
    return means


@pytest.mark.parametrize("nu", [4.0, 30.0])
def test_regulariser_moves_counts_toward_target(nu):
    """The 12-128rec-27 net starts near 13.4 spikes per neuron and sample;
    three small gradient steps on the regulariser alone lower the mean count
    toward a target of 4 and raise it toward 30, every step (a flipped sign
    of the term moves it away)."""
    m = np.array(_reg_only_steps(nu))
    assert 12.0 < m[0] < 15.0
    d = np.diff(m) * np.sign(nu - m[0])
    assert np.all(d > 0.2), m


def test_zero_strength_changes_nothing():
    wl = make_workload(3, B=4)
    c = wl.cfg
    net = oracle.OracleNet(c.layers, c.tau_m, c.tau_s, c.theta, c.dt, c.max_delay, wl.T, c.loss,
                           c.readout_scale, list(c.delay_range))
    f = oracle.forward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, cap=64 * 128)
    lo, g = oracle.loss(f.z, wl.labels)
    R, dlp = oracle.spike_count_reg(net, f, [0.0], 14.0)
    a = oracle.backward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, f, g)
    b = oracle.backward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, f, g, dlp=dlp)
    for x, y in zip(a[0] + a[1], b[0] + b[1]):
        assert np.array_equal(x, y)
