"""Pins of the grid oracle against closed forms, the continuous-time model,
invariants and the paper's sequence-detection example (all on the CPU)."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle.continuous import ContNet
from workloads import CONFIGS, LIF, LI, INPUT, LOSS_CE_SUM, LOSS_CE_MAX, make_workload

TM, TS = 20.0, 5.0


def kappa(x, tm=TM, ts=TS):
    return ts / (ts - tm) * (math.exp(-x / ts) - math.exp(-x / tm))


def dkappa(x, tm=TM, ts=TS):
    return ts / (ts - tm) * (-math.exp(-x / ts) / ts + math.exp(-x / tm) / tm)


def one_sample_csr(events):
    ev = sorted(events)
    return (np.array([0, len(ev)], np.int32), np.array([e[0] for e in ev], np.int32),
            np.array([e[1] for e in ev], np.int32))


def net_of(layers, T, dt=1.0, max_delay=10, loss=LOSS_CE_SUM, scale=None, theta=1.0):
    return oracle.OracleNet(layers, TM, TS, theta, dt, max_delay, T, loss,
                            1.0 / T if scale is None else scale)


# ---------------------------------------------------------------- constants, rounding


def test_constants_are_exact_one_step_propagators():
    a, b, g, c = oracle.constants(TM, TS, 1.0)
    assert a == np.float32(math.exp(-1 / TM)) and b == np.float32(math.exp(-1 / TS))
    # gamma is the one-step voltage response to unit current: kappa(dt)
    assert abs(g - kappa(1.0)) <= 1e-7 * abs(kappa(1.0))
    # c is the lambda_V -> lambda_I coupling; c = (tau_m/tau_s) gamma
    assert abs(c - TM / TS * kappa(1.0)) <= 1e-7 * abs(c)
    with pytest.raises(ValueError):
        oracle.constants(10.0, 10.0, 1.0)


def test_delay_rounding_half_even_and_clamp():
    # 1 input -> LI with 6 posts; delays exercise rint ties and clamps
    D = np.array([[0.5, 1.5, 2.5, -0.7, 12.6, np.nan]], np.float32)
    W = np.ones((1, 6), np.float32)
    net = net_of(((1, INPUT, 0), (6, LI, 0)), T=30, max_delay=10)
    off, st, ne = one_sample_csr([(0, 0)])
    f = oracle.forward(net, off, st, ne, [W], [D], trace=True)
    # first nonzero V- of post j is at step slot_j + 1
    first = [int(np.nonzero(f.V_trace[0, :, j])[0][0]) - 1 for j in range(6)]
    assert first == [0, 2, 2, 0, 10, 0]
    assert f.clamped == 3


def test_per_projection_delay_clamp():
    """A projection's own largest delay clamps its delays (and is counted),
    below the network-wide max_delay."""
    D = np.array([[0.5, 1.5, 2.5, -0.7, 12.6, np.nan, 4.4, 4.6]], np.float32)
    W = np.ones((1, 8), np.float32)
    net = net_of(((1, INPUT, 0), (8, LI, 0)), T=30, max_delay=10)
    net.proj_max_delay = [4]
    off, st, ne = one_sample_csr([(0, 0)])
    f = oracle.forward(net, off, st, ne, [W], [D], trace=True)
    first = [int(np.nonzero(f.V_trace[0, :, j])[0][0]) - 1 for j in range(8)]
    assert first == [0, 2, 2, 0, 4, 0, 4, 4]
    assert f.clamped == 4
    net.proj_max_delay = [11]          # beyond max_delay: refused
    with pytest.raises(ValueError):
        oracle.forward(net, off, st, ne, [W], [D])


# ---------------------------------------------------------------- P-1 closed-form PSP


@pytest.mark.parametrize("s0,d,w", [(3, 5, 0.7), (0, 0, -1.3), (7, 10, 2.0)])
def test_psp_matches_closed_form(s0, d, w):
    T = 120
    net = net_of(((1, INPUT, 0), (1, LI, 0)), T=T, max_delay=10)
    off, st, ne = one_sample_csr([(s0, 0)])
    f = oracle.forward(net, off, st, ne, [np.array([[w]], np.float32)],
                       [np.array([[d]], np.float32)], trace=True)
    V = f.V_trace[0, :, 0].astype(np.float64)
    m = s0 + d
    ref = np.array([0.0 if n <= m else w * kappa((n - m) * 1.0) for n in range(T)])
    assert np.all(V[:m + 1] == 0.0)
    assert np.allclose(V, ref, rtol=2e-5, atol=1e-12)


def test_lif_spike_train_matches_closed_form():
    """One strong input: spikes at m + k1, then from reset with I_r = I- ..."""
    T, s0, d, w = 200, 2, 4, 9.0
    net = net_of(((1, INPUT, 0), (1, LIF, 0), (1, LI, 0)), T=T, max_delay=10)
    off, st, ne = one_sample_csr([(s0, 0)])
    f = oracle.forward(net, off, st, ne, [np.array([[w]], np.float32), np.zeros((1, 1), np.float32)],
                       [np.array([[d]], np.float32), np.zeros((1, 1), np.float32)])
    beta = math.exp(-1.0 / TS)
    n, I, spikes, margins = s0 + d, w, [], []
    while True:
        k = 1
        while n + k < T and I * kappa(k) < 1.0:
            k += 1
        if n + k >= T:
            break
        margins.append(min(I * kappa(k) - 1.0, 1.0 - I * kappa(k - 1) if k > 1 else 1.0))
        n, I = n + k, I * beta ** k
        spikes.append((n, I))
    assert min(margins) > 1e-4       # fp32 cannot flip any decision
    st_, ne_ = f.spikes(0, 0)
    assert [int(x) for x in st_] == [s for s, _ in spikes]
    assert np.allclose(f.I_minus[0, 0, :len(spikes)], [i for _, i in spikes], rtol=1e-5)


# ---------------------------------------------------------------- P-2/P-3 exact grid adjoint


@pytest.mark.parametrize("mode", ["f64", "f32"])
def test_subthreshold_dw_dd_closed_forms(mode):
    """LI only, sum readout, linear loss L = g z: dW = s g sum_k kappa(k dt),
    dD (per step) = -w s g dt sum_k kappa'(k dt), k = 1 .. T-1-m."""
    T, s0, d, w = 80, 3, 5, 0.7
    net = net_of(((1, INPUT, 0), (1, LI, 0)), T=T, max_delay=10)
    off, st, ne = one_sample_csr([(s0, 0)])
    W, D = [np.array([[w]], np.float32)], [np.array([[d]], np.float32)]
    f = oracle.forward(net, off, st, ne, W, D)
    g = np.array([[1.0]], np.float32)
    dW, dD, deg = oracle.backward(net, off, st, ne, W, D, f, g, mode=mode)
    m = s0 + d
    s = float(np.float32(1.0 / T))       # the readout scale the oracle receives
    ks = range(1, T - m)
    dW_ref = s * sum(kappa(k) for k in ks)
    dD_ref = -float(np.float32(w)) * s * sum(dkappa(k) for k in ks)
    # the fp32 model's dD loses digits to the cancellation in lambda_I - lambda_V
    tol_w, tol_d = (1e-12, 1e-12) if mode == "f64" else (2e-6, 3e-5)
    assert abs(dW[0][0, 0] - dW_ref) <= tol_w * abs(dW_ref)
    assert abs(dD[0][0, 0] - dD_ref) <= tol_d * abs(dD_ref)
    assert deg == 0


def test_max_readout_subthreshold_closed_forms():
    """LI only, max-over-time readout, linear loss L = sum_k c_k z_k: the loss
    source sits at the first maximiser n* = m + k* (k* maximises kappa(k dt)),
    so dW_k = c_k kappa(k* dt) and dD_k (per step, the right-derivative in the
    arrival time) = -w_k c_k kappa'(k* dt) dt, exactly on the grid; a source
    one step early or late gives kappa((k* -+ 1) dt) instead.  An output whose
    voltage never rises above 0 keeps n* = 0 (strict >) and a zero gradient."""
    T, s0 = 60, 3
    net = net_of(((1, INPUT, 0), (2, LI, 0)), T=T, max_delay=10, loss=LOSS_CE_MAX, scale=1.0)
    off, st, ne = one_sample_csr([(s0, 0)])
    w = np.array([[0.7, -0.4]], np.float32)
    W, D = [w], [np.array([[5.0, 2.0]], np.float32)]
    f = oracle.forward(net, off, st, ne, W, D)
    c = np.array([[1.0, -0.5]], np.float32)
    dW, dD, deg = oracle.backward(net, off, st, ne, W, D, f, c)
    ks = max(range(1, T), key=lambda k: kappa(float(k)))
    assert ks == 9 and int(f.nstar[0, 0]) == s0 + 5 + ks and int(f.nstar[0, 1]) == 0
    assert abs(dW[0][0, 0] - kappa(ks)) <= 1e-12 * kappa(ks)
    ref_d = -float(w[0, 0]) * dkappa(ks)
    assert abs(dD[0][0, 0] - ref_d) <= 1e-10 * abs(ref_d)
    assert dW[0][0, 1] == 0.0 and dD[0][0, 1] == 0.0
    for k in (ks - 1, ks + 1):          # what a misplaced source would give
        assert abs(kappa(k) - kappa(ks)) > 1e-4 * kappa(ks)


# ---------------------------------------------------------------- P-5 grid -> continuous


def _grid_vs_continuous(layers, projs, inp, T_ms, dt, loss, c):
    """Grid oracle gradients (fp64) of L = sum_k c_k z_k on the continuous net's
    parameters: z the sum readout with scale dt (so z ~ the integral of V) or
    the max readout; delays and input times on the grid, dD per ms."""
    T = int(round(T_ms / dt))
    md = max(int(round(float(np.max(d)) / dt)) for _, _, _, d in projs)
    net = oracle.OracleNet(layers, TM, TS, 1.0, dt, md, T, loss, dt)
    off, st, ne = one_sample_csr([(int(round(t / dt)), i) for t, i in inp])
    W = [np.array(w, np.float32) for _, _, w, _ in projs]
    D = [np.array(np.round(np.array(d) / dt), np.float32) for _, _, _, d in projs]
    f = oracle.forward(net, off, st, ne, W, D)
    dW, dD, _ = oracle.backward(net, off, st, ne, W, D, f, np.array([c], np.float32))
    return dW, [x / dt for x in dD], f


def _tensor_err(grid, cont):
    """max |grid - cont| / max |cont| per tensor (absolute where cont is 0)."""
    out = []
    for g, r in zip(grid, cont):
        r = np.asarray(r, np.float64)
        sc = np.abs(r).max()
        out.append(np.abs(np.asarray(g) - r).max() / (sc if sc > 0 else 1.0))
    return out


def test_recurrent_delays_grid_converges_to_continuous():
    """Two recurrent LIF neurons with recurrent delays and two LI readouts
    (13 hidden spikes in 40 ms, the first cut of the continuous net of the
    recurrent FD test before a grazing crossing at 45 ms): every dW and dD of
    the three projections approaches continuous EventProp at first order in
    dt, which pins the recurrent adjoint ring and the jump sums over
    recurrent arrivals."""
    W_in, D_in = [[6.0, 4.5], [3.0, 7.0]], [[1.3, 4.1], [2.2, 0.7]]
    W_rec, D_rec = [[0.0, 2.5], [1.8, 0.0]], [[0.5, 3.3], [6.1, 1.1]]
    W_out, D_out = [[1.2, -0.7], [0.4, 0.9]], [[2.5, 0.9], [3.7, 5.2]]
    projs = [(0, 1, W_in, D_in), (1, 1, W_rec, D_rec), (1, 2, W_out, D_out)]
    inp = [(0.5, 0), (3.1, 1), (9.4, 0), (17.2, 1)]
    c = [0.8, -1.3]
    T = 40.0
    cont = ContNet([2, 2, 2], projs, T=T)
    L, rec = cont.forward(inp, "integral", c)
    assert len(rec["spikes"]) == 13
    cW, cD = cont.backward(inp, rec)
    worst = []
    for dt in (0.1, 0.05, 0.025):
        gW, gD, f = _grid_vs_continuous(((2, INPUT, 0), (2, LIF, 1), (2, LI, 0)), projs, inp, T, dt,
                                        LOSS_CE_SUM, c)
        assert int(f.count.sum()) == 13
        worst.append(max(_tensor_err(gW, cW) + _tensor_err(gD, cD)))
    worst = np.array(worst)
    assert np.all(worst[:-1] / worst[1:] > 1.6), worst
    assert worst[-1] < 0.1, worst


def test_max_readout_grid_converges_to_continuous():
    """One hidden spike into two LI readouts, max-over-time loss: the readout
    weights' gradients (the PSP value at the maximum) match continuous
    EventProp to 1e-3 at dt <= 0.1 ms, and the gradients that vanish in
    continuous time (a shift of the hidden spike or of an arrival only moves
    the maximum) shrink with dt."""
    W_in, D_in = [[9.0]], [[1.5]]
    W_out, D_out = [[1.1, 0.6]], [[2.0, 6.5]]
    projs = [(0, 1, W_in, D_in), (1, 2, W_out, D_out)]
    inp = [(2.0, 0)]
    c = [1.0, -0.5]
    cont = ContNet([1, 1, 2], projs, T=60.0)
    L, rec = cont.forward(inp, "max", c)
    cW, cD = cont.backward(inp, rec)
    ro = np.asarray(cW[1], np.float64)
    zero = [np.asarray(cW[0]), np.asarray(cD[0]), np.asarray(cD[1])]
    assert all(np.abs(z).max() < 1e-12 for z in zero)
    vanish = []
    for dt in (0.1, 0.05):
        gW, gD, _ = _grid_vs_continuous(((1, INPUT, 0), (1, LIF, 0), (2, LI, 0)), projs, inp, 60.0,
                                        dt, LOSS_CE_MAX, c)
        assert np.abs(gW[1] - ro).max() <= 1e-3 * np.abs(ro).max()
        vanish.append(max(np.abs(gW[0]).max(), np.abs(gD[0]).max(), np.abs(gD[1]).max()))
    assert vanish[1] < vanish[0] / 2 and vanish[0] < 1e-3 * np.abs(ro).max()


def test_grid_converges_to_continuous_eventprop():
    cont = ContNet([1, 1, 1], [(0, 1, [[10.0]], [[2.0]]), (1, 2, [[1.5]], [[3.0]])], T=60.0)
    inp = [(1.0, 0)]
    L, rec = cont.forward(inp)
    cW, cD = cont.backward(inp, rec)
    ref = np.array([cW[0][0][0], cD[0][0][0], cW[1][0][0], cD[1][0][0]])
    errs = []
    for dt in (0.1, 0.05, 0.025, 0.0125):
        T = int(round(60.0 / dt))
        net = oracle.OracleNet(((1, INPUT, 0), (1, LIF, 0), (1, LI, 0)), TM, TS, 1.0, dt,
                               int(round(3.0 / dt)), T, LOSS_CE_SUM, dt)
        off, st, ne = one_sample_csr([(int(round(1.0 / dt)), 0)])
        W = [np.array([[10.0]], np.float32), np.array([[1.5]], np.float32)]
        D = [np.array([[2.0 / dt]], np.float32), np.array([[3.0 / dt]], np.float32)]
        f = oracle.forward(net, off, st, ne, W, D)
        dW, dD, _ = oracle.backward(net, off, st, ne, W, D, f, np.array([[1.0]], np.float32))
        grid = np.array([dW[0][0, 0], dD[0][0, 0] / dt, dW[1][0, 0], dD[1][0, 0] / dt])
        errs.append(np.abs(grid - ref) / np.abs(ref))
    worst = np.array(errs).max(axis=1)     # spike times are quantised to the grid: O(dt)
    assert worst[-1] < 1.5e-2
    assert np.all(worst[:-1] / worst[1:] > 1.8)


# ---------------------------------------------------------------- P-6 invariants


def _run(wl, mode="f64", layers=None, max_delay=None, D=None, B_sel=None):
    c = wl.cfg
    net = oracle.OracleNet(layers or c.layers, c.tau_m, c.tau_s, c.theta, c.dt,
                           c.max_delay if max_delay is None else max_delay, wl.T, c.loss,
                           c.readout_scale)
    D = wl.D if D is None else D
    f = oracle.forward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, D)
    lo, g = oracle.loss(f.z, wl.labels)
    dW, dD, deg = oracle.backward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, D, f, g, mode=mode)
    return f, lo, g, dW, dD


@pytest.mark.parametrize("cid", [1, 3])
def test_zero_input_gives_zero_everything(cid):
    wl = make_workload(cid, B=4)
    wl.in_off[:] = 0
    wl.in_step, wl.in_neuron = wl.in_step[:0], wl.in_neuron[:0]
    f, lo, g, dW, dD = _run(wl)
    assert f.count.sum() == 0 and np.all(f.z == 0)
    assert abs(lo[-1] - math.log(wl.cfg.n_classes)) < 1e-6
    assert all(np.all(x == 0) for x in dW + dD)


@pytest.mark.parametrize("cid", [2, 3])
def test_input_delay_shift_shifts_spike_train_exactly(cid):
    """Adding k to every input-projection delay shifts every hidden spike and
    its I- by exactly k steps, bit-exact also with recurrence: every
    projection has its own delay ring, so each cell keeps its summation
    order; with the max readout the readout value is unchanged."""
    wl = make_workload(cid, B=4)
    k = 7
    f0, *_ = _run(wl, max_delay=wl.cfg.max_delay + k)
    D = [d.copy() for d in wl.D]
    D[0] = D[0] + np.float32(k)
    f1, *_ = _run(wl, max_delay=wl.cfg.max_delay + k, D=D)
    assert f0.count.sum() > 50
    for b in range(wl.B):
        s0, n0 = f0.spikes(0, b)
        s1, n1 = f1.spikes(0, b)
        keep = s0 + k <= wl.T - 1
        assert np.array_equal(s0[keep] + k, s1) and np.array_equal(n0[keep], n1)
        assert np.array_equal(f0.I_minus[0, b, :keep.sum()], f1.I_minus[0, b, :keep.sum()])
    if cid == 2:
        inner = f0.nstar + k <= wl.T - 1
        assert np.array_equal(f0.z[inner], f1.z[inner])
        assert np.array_equal(f0.nstar[inner] + k, f1.nstar[inner])


def test_input_time_shift_shifts_recurrent_net_exactly():
    """Recurrent net: delaying every input spike by k steps delays everything
    by k steps, bit-exact."""
    wl = make_workload(3, B=4)
    k = 9
    f0, *_ = _run(wl)
    wl.in_step = (wl.in_step + k).astype(np.int32)
    keep_in = wl.in_step <= wl.T - 1
    counts = [int(keep_in[wl.in_off[b]:wl.in_off[b + 1]].sum()) for b in range(wl.B)]
    wl.in_off = np.cumsum([0] + counts).astype(np.int32)
    wl.in_step, wl.in_neuron = wl.in_step[keep_in], wl.in_neuron[keep_in]
    f1, *_ = _run(wl)
    assert f0.count.sum() > 100
    for b in range(wl.B):
        s0, n0 = f0.spikes(0, b)
        s1, n1 = f1.spikes(0, b)
        keep = s0 + k <= wl.T - 1
        assert np.array_equal(s0[keep] + k, s1) and np.array_equal(n0[keep], n1)
        assert np.array_equal(f0.I_minus[0, b, :keep.sum()], f1.I_minus[0, b, :keep.sum()])


def test_batch_permutation_and_sample_independence():
    wl = make_workload(3, B=6)
    f, lo, g, dW, dD = _run(wl)
    perm = [3, 0, 5, 1, 4, 2]
    off, st, ne = wl.in_off, wl.in_step, wl.in_neuron
    segs = [(st[off[b]:off[b + 1]], ne[off[b]:off[b + 1]]) for b in range(wl.B)]
    wl2 = make_workload(3, B=6)
    wl2.in_off = np.cumsum([0] + [segs[p][0].size for p in perm]).astype(np.int32)
    wl2.in_step = np.concatenate([segs[p][0] for p in perm])
    wl2.in_neuron = np.concatenate([segs[p][1] for p in perm])
    wl2.labels = wl.labels[perm]
    f2, lo2, g2, dW2, dD2 = _run(wl2)
    assert np.array_equal(f2.z, f.z[perm]) and np.array_equal(g2, g[perm])
    for i, p in enumerate(perm):
        assert np.array_equal(f2.spikes(0, i)[0], f.spikes(0, p)[0])
    for a, b in zip(dW + dD, dW2 + dD2):
        assert np.allclose(a, b, rtol=1e-12, atol=1e-15 * np.abs(a).max())
    # one sample alone equals the same sample inside the batch
    wl1 = make_workload(3, B=6)
    wl1.in_off = np.array([0, segs[2][0].size], np.int32)
    wl1.in_step, wl1.in_neuron, wl1.labels = segs[2][0], segs[2][1], wl.labels[2:3]
    f1, *_ = _run(wl1)
    assert np.array_equal(f1.spikes(0, 0)[0], f.spikes(0, 2)[0])
    assert np.array_equal(f1.z[0], f.z[2])


def test_zero_delays_recurrent_runs_and_sub_half_delays_round_to_zero():
    wl = make_workload(3, B=3)
    D0 = [np.zeros_like(d) for d in wl.D]
    Dh = [np.full_like(d, 0.49) for d in wl.D]
    fa, la, ga, dWa, dDa = _run(wl, D=D0)
    fb, lb, gb, dWb, dDb = _run(wl, D=Dh)
    assert fa.count.sum() > 0
    assert np.array_equal(fa.count, fb.count) and np.array_equal(fa.z, fb.z)
    for a, b in zip(dWa + dDa, dWb + dDb):
        assert np.array_equal(a, b)


def test_degenerate_crossings_are_counted():
    wl = make_workload(3, B=8)
    c = wl.cfg
    net = oracle.OracleNet(c.layers, c.tau_m, c.tau_s, c.theta, c.dt, c.max_delay, wl.T, c.loss,
                           c.readout_scale)
    f = oracle.forward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D)
    lo, g = oracle.loss(f.z, wl.labels)
    _, _, deg = oracle.backward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, f, g)
    n_deg = sum(int((f.I_minus[0, b, :f.count[0, b]] <= c.theta).sum()) for b in range(wl.B))
    assert deg == n_deg


# ---------------------------------------------------------------- loss


def test_cross_entropy_closed_forms():
    z = np.zeros((3, 4), np.float32)
    lo, g = oracle.loss(z, [0, 1, 3])
    assert np.allclose(lo, math.log(4))
    exp = np.full((3, 4), 0.25 / 3)
    exp[[0, 1, 2], [0, 1, 3]] -= 1 / 3
    assert np.allclose(g, exp, rtol=1e-7)
    z = np.array([[2.0, -1.0]], np.float32)
    lo, g = oracle.loss(z, [1])
    ref = math.log(math.exp(2) + math.exp(-1)) + 1.0
    assert abs(lo[0] - ref) < 1e-6 and abs(g[0, 0] + g[0, 1]) < 1e-7


# ---------------------------------------------------------------- fp32 model vs fp64


@pytest.mark.parametrize("cid", [2, 3])
def test_f32_model_tracks_f64_definition(cid):
    """The kernel-precision model (fp32 state, fp64 sums) stays within
    1e-4 of each gradient tensor's scale of the fp64 definition."""
    wl = make_workload(cid, B=16)
    _, _, _, dW, dD = _run(wl, "f64")
    _, _, _, dW1, dD1 = _run(wl, "f32")
    for a, b in zip(dW + dD, dW1 + dD1):
        s = np.abs(a).max()
        assert s > 0
        assert np.abs(a - b).max() <= 1e-4 * s


# ---------------------------------------------------------------- P-7 sequence detection


GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "sequence_detection.json")))


def _seq_net():
    return oracle.OracleNet(((2, INPUT, 0), (2, LI, 0)), TM, TS, 1.0, 1.0, 30, 60, LOSS_CE_MAX, 1.0)


def _seq_example(cls):
    # dt = 1 ms, so times in ms are steps
    return one_sample_csr([(int(t), int(i)) for t, i in GOLDEN["class_inputs_ms"][str(cls)]])


def test_sequence_detection_first_gradient_signs():
    net = _seq_net()
    W = [np.array(GOLDEN["weights"], np.float32)]
    D = [np.array(GOLDEN["initial_delays_ms"], np.float32)]
    off, st, ne = _seq_example(0)
    f = oracle.forward(net, off, st, ne, W, D)
    lo, g = oracle.loss(f.z, [0])
    _, dD, _ = oracle.backward(net, off, st, ne, W, D, f, g)
    dD = dD[0]
    # correct output 0: the update (-dL/dd) to the delay from the earlier input is
    # positive and to the delay from the later input negative (Fig. 3 caption).
    assert dD[0, 0] < 0 < dD[1, 0]
    # The wrong output starts with coincident EPSPs; its max sits at the PSP
    # peak, where both delay gradients vanish up to grid effects, so the
    # caption's "opposite" direction is not a robust sign there.
    assert abs(dD[0, 1]) < 0.2 * abs(dD[0, 0]) and abs(dD[1, 1]) < 0.2 * abs(dD[1, 0])


def test_sequence_detection_learns_with_delays_only():
    net = _seq_net()
    W = [np.array(GOLDEN["weights"], np.float32)]
    D = np.array(GOLDEN["initial_delays_ms"], np.float32)
    # The paper reaches 100 % after 6 presentations of each class with learning
    # rate 1 under time constants and loss scaling it does not state.  With
    # tau_m = 20 ms, tau_s = 5 ms and the CE gradient used here the delay
    # gradients are ~300x smaller, so the equivalent step is lr = 300.
    lr = 300.0

    def accuracy(D):
        ok = 0
        for cls in (0, 1):
            off, st, ne = _seq_example(cls)
            f = oracle.forward(net, off, st, ne, W, [D])
            ok += int(np.argmax(f.z[0]) == cls)
        return ok / 2

    assert accuracy(D) == 0.0
    assert accuracy(np.array(GOLDEN["solving_delays_ms"], np.float32)) == 1.0
    seen = 0
    while accuracy(D) < 1.0:
        assert seen < 10
        for cls in (0, 1):
            off, st, ne = _seq_example(cls)
            f = oracle.forward(net, off, st, ne, W, [D])
            lo, g = oracle.loss(f.z, [cls])
            _, dD, _ = oracle.backward(net, off, st, ne, W, [D], f, g)
            D = np.maximum(D - lr * dD[0].astype(np.float32), 0.0).astype(np.float32)
        seen += 1
