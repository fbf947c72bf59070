"""Pins of the spike-time loss terms (CPU only): the time-invariant MSE on
first output spike times and a general dl_p/dt_k added to the lambda_V jump
(Table 1 backward transition; Methods, "Time-invariant mean squared error
loss").

* Continuous time: EventProp with the l_p term equals central finite
  differences of the exactly simulated loss (a wrong sign, a dropped term or
  the term applied at a later spike fails), and the loss's invariance to a
  common time shift makes the input-delay gradients sum to zero.
* Grid: the loss and its time derivatives in closed form; the grid gradient
  converges to the continuous one as dt halves; a zero l_p term changes
  nothing; the gradients are affine in the l_p term.
"""
import numpy as np
import pytest

import oracle
from oracle.continuous import ContNet
from workloads import INPUT, LIF, LI, LOSS_CE_SUM, make_workload

from .test_oracle_continuous import _cmp
from .test_oracle_grid import TM, TS, one_sample_csr

W_IN = [[9.0, 6.0], [5.0, 8.5]]
D_IN = [[1.0, 3.0], [2.2, 0.4]]
W_OUT = [[7.0, 3.0], [4.0, 6.5]]
D_OUT = [[1.5, 3.0], [2.5, 0.8]]
INP = [(0.5, 0), (2.0, 1), (7.5, 0)]


def _cont():
    return ContNet([2, 2, 2], [(0, 1, W_IN, D_IN), (1, 2, W_OUT, D_OUT)], T=60.0, out_lif=True)


@pytest.mark.parametrize("label,delta", [(0, 3.0), (1, 0.5)])
def test_dmse_eventprop_equals_fd(label, delta):
    net = _cont()
    L, rec = net.forward(INP, "dmse", label=label, delta=delta)
    assert all(f < net.T for f in rec["first"])              # both outputs fire
    assert sum(1 for s in rec["spikes"] if s[1] == 2) > 2     # later output spikes carry no l_p
    _cmp(net.backward(INP, rec), net.fd(INP, "dmse", label=label, delta=delta), rtol=2e-6, atol=1e-8)


def test_dmse_is_time_invariant():
    """A common shift of every input delay moves every spike by the same
    amount and leaves t_i - t_c unchanged: the input-delay gradients sum to 0
    (while they are individually far from 0)."""
    net = _cont()
    L, rec = net.forward(INP, "dmse", label=0, delta=3.0)
    dW, dD = net.backward(INP, rec)
    s = sum(sum(r) for r in dD[0])
    big = max(abs(x) for r in dD[0] for x in r)
    assert big > 0.1 and abs(s) < 1e-9 * big


def test_linear_hidden_spike_time_term_equals_fd():
    W_in = [[8.0, 4.5], [3.0, 7.0]]
    D_in = [[1.3, 4.1], [2.2, 0.7]]
    W_out = [[1.2, -0.7], [0.4, 0.9]]
    D_out = [[2.5, 0.9], [3.7, 5.2]]
    net = ContNet([2, 2, 2], [(0, 1, W_in, D_in), (1, 2, W_out, D_out)], T=50.0)
    inp = [(0.5, 0), (3.1, 1), (9.4, 0)]
    c = [0.8, -1.3]
    kw = dict(lp_lin={1: 0.35})
    L, rec = net.forward(inp, "integral", c, **kw)
    assert len(rec["spikes"]) >= 3
    g = net.backward(inp, rec)
    _cmp(g, net.fd(inp, "integral", c, h=1e-6, **kw), rtol=2e-5, atol=1e-8)
    # and the term matters: without it the gradient differs
    L0, rec0 = net.forward(inp, "integral", c)
    g0 = net.backward(inp, rec0)
    assert abs(g[0][0][0][0] - g0[0][0][0][0]) > 1e-3


def test_dmse_loss_closed_form():
    # c = 0, t = (5, 8, 12), delta = 2: errors 8-5-2 = 1 and 12-5-2 = 5,
    # L = (1 + 25) / 2 = 13; dL/dt = (-(1 + 5), 1, 5) / B
    z = np.array([[5.0, 8.0, 12.0], [3.0, 3.0, 1.0]], np.float32)
    lo, dl = oracle.loss_dmse(z, [0, 2], 2.0)
    # second sample, c = 2: errors 3-1-2 = 0, 3-1-2 = 0
    assert lo[0] == 13.0 and lo[1] == 0.0 and lo[2] == 6.5
    assert np.array_equal(dl[0], np.array([-6.0, 1.0, 5.0]) / 2)
    assert np.array_equal(dl[1], np.zeros(3))


def _grid_run(dt, label=0, delta=3.0, mode="f64", dlp_scale=1.0):
    T = int(round(60.0 / dt))
    net = oracle.OracleNet(((2, INPUT, 0), (2, LIF, 0), (2, LIF, 0)), TM, TS, 1.0, dt,
                           int(round(3.0 / dt)), T, oracle.LOSS_DMSE, 0.0)
    off, st, ne = one_sample_csr([(int(round(t / dt)), i) for t, i in INP])
    W = [np.array(W_IN, np.float32), np.array(W_OUT, np.float32)]
    D = [np.array(D_IN, np.float32) / np.float32(dt), np.array(D_OUT, np.float32) / np.float32(dt)]
    D = [np.rint(d).astype(np.float32) for d in D]
    f = oracle.forward(net, off, st, ne, W, D)
    lo, dl = oracle.loss_dmse(f.z, [label], delta)
    dlp = oracle.first_spike_dlp(net, f, dl) * dlp_scale
    dW, dD, _ = oracle.backward(net, off, st, ne, W, D, f, np.zeros_like(f.z), mode=mode, dlp=dlp)
    return net, f, lo, dW, dD


def test_first_spike_dlp_sits_on_first_spikes_only():
    net, f, lo, _, _ = _grid_run(0.1)
    _, dl = oracle.loss_dmse(f.z, [0], 3.0)
    dlp = oracle.first_spike_dlp(net, f, dl)
    c = int(f.count[1, 0])
    assert c > 2
    nz = np.flatnonzero(dlp[1, 0, :c])
    first = [int(np.flatnonzero(f.neuron[1, 0, :c] == k)[0]) for k in (0, 1)]
    assert sorted(nz.tolist()) == sorted(first)
    assert np.all(dlp[0] == 0)
    # z holds the first spike times in ms (n times the fp32 dt, in fp64)
    for k in (0, 1):
        assert f.z[0, k] == np.float32(f.step[1, 0, first[k]] * np.float64(np.float32(0.1)))


def test_grid_dmse_converges_to_continuous():
    cont = _cont()
    L, rec = cont.forward(INP, "dmse", label=0, delta=3.0)
    cW, cD = cont.backward(INP, rec)
    ref = np.concatenate([np.ravel(cW[0]), np.ravel(cW[1]), np.ravel(cD[0]), np.ravel(cD[1])])
    errs = []
    for dt in (0.1, 0.05, 0.025, 0.0125):
        _, _, _, dW, dD = _grid_run(dt)
        grid = np.concatenate([np.ravel(dW[0]), np.ravel(dW[1]), np.ravel(dD[0]) / dt,
                               np.ravel(dD[1]) / dt])
        errs.append(np.abs(grid - ref).max() / np.abs(ref).max())
    errs = np.array(errs)
    assert errs[-1] < 2e-2
    assert np.all(errs[:-1] / errs[1:] > 1.6), errs


def test_zero_lp_term_changes_nothing_and_gradients_are_affine_in_it():
    wl = make_workload(3, B=4)
    c = wl.cfg
    net = oracle.OracleNet(c.layers, c.tau_m, c.tau_s, c.theta, c.dt, c.max_delay, wl.T, c.loss,
                           c.readout_scale)
    f = oracle.forward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, cap=8192)
    lo, g = oracle.loss(f.z, wl.labels)
    args = (net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, f, g)
    base = oracle.backward(*args, mode="f32")
    zero = oracle.backward(*args, mode="f32", dlp=np.zeros((1, wl.B, f.cap)))
    for a, b in zip(base[0] + base[1], zero[0] + zero[1]):
        assert np.array_equal(a, b)
    rng = np.random.default_rng(3)
    x = rng.normal(0, 1e-3, size=(1, wl.B, f.cap))
    g0 = oracle.backward(*args)
    g1 = oracle.backward(*args, dlp=x)
    g2 = oracle.backward(*args, dlp=2 * x)
    P = len(wl.W)
    for p, (a0, a1, a2) in enumerate(zip(g0[0] + g0[1], g1[0] + g1[1], g2[0] + g2[1])):
        d1, d2 = a1 - a0, a2 - a0
        if p % P == P - 1:
            # the readout's adjoints never see a hidden jump
            assert np.all(d1 == 0) and np.all(d2 == 0)
            continue
        assert np.abs(d1).max() > 1e-3 * np.abs(a0).max()
        assert np.allclose(d2, 2 * d1, rtol=1e-9, atol=1e-12 * np.abs(d1).max())
