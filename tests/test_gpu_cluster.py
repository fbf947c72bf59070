"""Cluster mode of the LIF cores: a sample spread over ceil(widest LIF layer /
64) one-wave workgroups, each holding the LDS ring columns of its 64 neurons,
which exchange the step's spike masks (forward) and the partial jump sums of
the step's spikes (backward) through device memory.

* Forced on the smaller networks (SNN_FLAG_CLUSTER): the forward bit-exact
  with the oracle and with one workgroup per sample; every dW and dD element
  within 1e-6 + 1e-4 |ref| of the oracle's fp64 definition (the jump sums add
  the workgroups' shares in workgroup order, another order than one
  workgroup's).
* The two 1024-neuron recurrent layers, whose rings fit no single workgroup,
  run their forward core in cluster mode by themselves (their rings are
  reported in LDS); forward and backward in cluster mode agree with one
  workgroup per sample and rings in device memory.
* More samples than one launch holds (several passes) and repeated calls
  (fresh exchange tags): per-sample results equal those of separate smaller
  batches, repeated calls bit-identical.
"""
import dataclasses

import numpy as np
import pytest

from workloads import LOSS_DMSE, make_variant, make_workload

from .gpu_util import (assert_backward_close, assert_forward_bitexact, grad_close, run_gpu,
                       run_oracle)

pytestmark = pytest.mark.gpu

FWD_KEYS = ("count", "step", "neuron", "z", "V", "I", "loss")


def _same_forward(a, b, wl):
    for k in FWD_KEYS:
        assert np.array_equal(np.asarray(a[k]).view(np.uint8), np.asarray(b[k]).view(np.uint8)), k
    for li in range(a["count"].shape[0]):
        for s in range(wl.B):
            c = min(int(a["count"][li, s]), a["net"].record_capacity)
            assert np.array_equal(a["I_minus"][li, s, :c].view(np.uint32),
                                  b["I_minus"][li, s, :c].view(np.uint32))


def _latency_lif_out(B):
    return make_variant(2, B=B, layers=((4, 0, 0), (200, 1, 0), (3, 1, 0)), loss=LOSS_DMSE,
                        dmse_delta=1.0, name="latency-4-200-3lif")


@pytest.mark.parametrize("case", ["cfg3", "cfg4", "lif-out"])
def test_forced_cluster_mode_parity(case):
    """12-128rec-27 (2 workgroups per sample), 700-256rec-20 (4) and the
    4-200-3 network with a LIF output layer and the spike-time loss (4
    workgroups; the 3 output neurons all in the first)."""
    import paper_2501_07331_amd as snn
    wl = {"cfg3": lambda: make_workload(3, B=16), "cfg4": lambda: make_workload(4, B=8),
          "lif-out": lambda: _latency_lif_out(16)}[case]()
    print(f"[cluster] {case} B={wl.B}", flush=True)
    gpu = run_gpu(wl, flags=snn.SNN_FLAG_CLUSTER)
    assert gpu["rc"] == 0
    orc = run_oracle(wl, modes=("f64",))
    assert_forward_bitexact(gpu, orc, wl)
    assert np.allclose(gpu["loss"], orc["loss"], rtol=1e-6, atol=1e-7)
    assert_backward_close(gpu, orc)
    one = run_gpu(wl)
    _same_forward(gpu, one, wl)


def test_wide_recurrent_layers_run_in_cluster_mode():
    """700-1024rec-1024rec-35 at B = 16 (its oracle parity is in the parity
    tests): every LIF -> LIF ring in LDS, which only cluster mode can hold
    (1.9 MB per sample), and the same forward as one workgroup per sample
    with its rings in device memory, bit for bit; gradients within the
    tolerance of each other."""
    import paper_2501_07331_amd as snn
    wl = make_workload(5, B=16)
    print("[cluster] cfg5 B=16 against device-memory rings", flush=True)
    gpu = run_gpu(wl)
    assert gpu["rc"] == 0
    lif_lif = [p for p, (pre, post) in enumerate(_projections(wl))
               if pre > 0 and post < len(wl.layers) - 1]
    assert all((gpu["stats"]["lds_rings"] >> p) & 1 for p in lif_lif), gpu["stats"]["lds_rings"]
    hbm = run_gpu(wl, flags=snn.SNN_FLAG_HBM_RINGS)
    assert hbm["stats"]["lds_rings"] == 0
    both = run_gpu(wl, flags=snn.SNN_FLAG_CLUSTER)        # the backward core in cluster mode too
    for x in (gpu, both):
        _same_forward(x, hbm, wl)
        for p in range(len(x["dW"])):
            for nm in ("dW", "dD"):
                ok, worst, rel = grad_close(x[nm][p], hbm[nm][p])
                print(f"[cluster] {nm}[{p}] vs device-memory rings: worst {worst:.3g}", flush=True)
                assert ok, (nm, p, worst, rel)


def _projections(wl):
    out = []
    for l in range(1, len(wl.layers)):
        out.append((l - 1, l))
        if wl.layers[l][2]:
            out.append((l, l))
    return out


def _slice(wl, s0, s1):
    o = wl.in_off
    return dataclasses.replace(wl, B=s1 - s0, in_off=(o[s0:s1 + 1] - o[s0]).astype(o.dtype),
                               in_step=wl.in_step[o[s0]:o[s1]], in_neuron=wl.in_neuron[o[s0]:o[s1]],
                               labels=wl.labels[s0:s1])


def test_several_launches_and_repeated_calls():
    """700-1024rec-1024rec-35 at B = 40: 16 samples per launch on 256 CUs, so
    three launches.  Each sample's forward equals that of a 20-sample batch
    holding it, bit for bit; dW and dD equal the sum of the two halves'
    (the loss is a batch mean: halves weigh 1/2 each); a second call on the
    same handle repeats the first bit for bit."""
    import paper_2501_07331_amd as snn
    wl = make_workload(5, B=40)
    print("[cluster] cfg5 B=40, twice, and two halves", flush=True)
    a = run_gpu(wl, flags=snn.SNN_FLAG_CLUSTER)
    assert a["rc"] == 0
    again = run_gpu(wl, net=a["net"])
    _same_forward(a, again, wl)
    for x, y in zip(a["dW"] + a["dD"], again["dW"] + again["dD"]):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    h = [run_gpu(_slice(wl, s0, s0 + 20), flags=snn.SNN_FLAG_CLUSTER) for s0 in (0, 20)]
    for k in ("count",):
        assert np.array_equal(a[k], np.concatenate([x[k] for x in h], axis=1))
    for k in ("z", "V", "I"):
        assert np.array_equal(a[k].view(np.uint32), np.concatenate([x[k] for x in h]).view(np.uint32)), k
    for li in range(a["count"].shape[0]):
        for s in range(wl.B):
            x, i = h[s // 20], s % 20
            c = min(int(a["count"][li, s]), a["net"].record_capacity)
            assert np.array_equal(a["step"][li, s, :c], x["step"][li, i, :c])
            assert np.array_equal(a["neuron"][li, s, :c], x["neuron"][li, i, :c])
            assert np.array_equal(a["I_minus"][li, s, :c].view(np.uint32),
                                  x["I_minus"][li, i, :c].view(np.uint32))
    for p in range(len(a["dW"])):
        for nm in ("dW", "dD"):
            ref = 0.5 * (h[0][nm][p].astype(np.float64) + h[1][nm][p].astype(np.float64))
            ok, worst, rel = grad_close(a[nm][p], ref)
            print(f"[cluster] {nm}[{p}] halves: worst {worst:.3g}", flush=True)
            assert ok, (nm, p, worst, rel)
