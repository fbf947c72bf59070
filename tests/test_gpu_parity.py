"""GPU (HIP library through its C ABI) vs the CPU oracle on the same seeded
inputs.  Spike records (step, neuron, I- at the spike), readout z and final
V/I must be bit-exact; the loss within rel 1e-6; every element of dW and dD
within 1e-6 + 1e-4 |ref| of the oracle's fp64 definition."""
import math

import numpy as np
import pytest

from workloads import make_workload

from .gpu_util import (assert_backward_close, assert_forward_bitexact, default_cap, grad_close,
                       make_gpu_net, run_gpu, run_oracle, to_device)

pytestmark = pytest.mark.gpu


def _parity(wl, flags=0, cap=None, per_proj=True):
    print(f"[parity] cfg{wl.cfg.cid} B={wl.B} T={wl.T} flags={flags} per_proj={per_proj}",
          flush=True)
    gpu = run_gpu(wl, cap=cap, flags=flags, per_proj=per_proj)
    orc = run_oracle(wl, cap=cap, per_proj=per_proj)
    assert gpu["rc"] == 0
    assert_forward_bitexact(gpu, orc, wl)
    assert np.allclose(gpu["loss"], orc["loss"], rtol=1e-6, atol=1e-7)
    assert_backward_close(gpu, orc)
    return gpu, orc


CASES = [
    (1, None, 1.0), (1, None, 6.0),      # config 1 as stated (no hidden spikes), and an active variant
    (2, None, 1.0), (3, None, 1.0),
    (4, 16, 1.0),                          # full T and widths, 16 samples
    (5, 16, 1.0),                          # two 1024-neuron recurrent layers, 16 samples
]


@pytest.mark.parametrize("cid,B,scale", CASES)
def test_parity_lds_rings(cid, B, scale):
    wl = make_workload(cid, B=B, weight_scale=scale)
    gpu, orc = _parity(wl)
    if scale != 1.0 or cid in (2, 3, 4, 5):
        assert orc["fwd"].count.sum() > 0


@pytest.mark.parametrize("cid,B", [(3, 32), (4, 16)])
def test_parity_network_wide_ring_depth(cid, B):
    """Every ring as deep as the network-wide largest delay (no per-projection
    depths): the same results as the per-projection rings, bit for bit in
    the forward, and within tolerance (the same fp64 sums) in the backward."""
    wl = make_workload(cid, B=B)
    gpu, orc = _parity(wl, per_proj=False)
    gpu2 = run_gpu(wl, per_proj=True)
    for k in ("count", "step", "neuron", "z", "V", "I"):
        assert np.array_equal(np.asarray(gpu[k]).view(np.uint8), np.asarray(gpu2[k]).view(np.uint8)), k
    for li in range(gpu["count"].shape[0]):      # I- of the stored records (the rest is unspecified)
        for b in range(wl.B):
            c = min(int(gpu["count"][li, b]), gpu["net"].record_capacity)
            assert np.array_equal(gpu["I_minus"][li, b, :c].view(np.uint32),
                                  gpu2["I_minus"][li, b, :c].view(np.uint32))
    for x, y in zip(gpu["dW"] + gpu["dD"], gpu2["dW"] + gpu2["dD"]):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))


@pytest.mark.parametrize("cid,B", [(2, 64), (4, 16), (1, 32)])
def test_fused_readout_equals_separate_readout_kernel(cid, B):
    """The LI readout run as one more wave of the forward core gives what the
    separate readout kernel gives, bit for bit: records, z, the LI state, the
    loss and the gradients (max readout on config 2, sum readout on 1 and 4)."""
    import paper_2501_07331_amd as snn
    wl = make_workload(cid, B=B, weight_scale=6.0 if cid == 1 else 1.0)
    a = run_gpu(wl)
    b = run_gpu(wl, flags=snn.SNN_FLAG_SEPARATE_READOUT)
    for k in ("count", "step", "neuron", "z", "V", "I", "loss"):
        assert np.array_equal(np.asarray(a[k]).view(np.uint8), np.asarray(b[k]).view(np.uint8)), k
    for x, y in zip(a["dW"] + a["dD"], b["dW"] + b["dD"]):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    orc = run_oracle(wl, modes=("f64",))
    assert_forward_bitexact(a, orc, wl)


@pytest.mark.parametrize("cid,B,T,scale", [(3, 8, 5, 1.0), (1, 8, 7, 6.0), (1, 8, 8, 6.0), (3, 8, 9, 1.0)])
def test_parity_short_trials(cid, B, T, scale):
    """Trials of 5 to 9 steps: fewer steps than most delays (arrivals past
    the end are dropped, rings never wrap), and the records, state, loss and
    gradients still match the oracle."""
    wl = make_workload(cid, B=B, T=T, weight_scale=scale)
    _parity(wl)


def test_per_projection_delay_clamp():
    """Delays past their projection's own largest delay are clamped to it
    (and counted) exactly as by the oracle, on a recurrent net whose
    recurrent projection is capped well below the feed-forward ones."""
    wl = make_workload(4, B=4)
    D = wl.D[1].copy()                 # recurrent projection, range 50
    D[0, :4] = [50.4, 50.6, 80.0, 200.0]
    wl.D[1] = D
    gpu, orc = _parity(wl)
    assert gpu["stats"]["clamped_delays"] == orc["fwd"].clamped == 3


@pytest.mark.parametrize("cid,B,scale", [(1, None, 6.0), (2, None, 1.0), (3, 32, 1.0), (4, 4, 1.0)])
def test_parity_hbm_rings(cid, B, scale):
    import paper_2501_07331_amd as snn
    wl = make_workload(cid, B=B, weight_scale=scale)
    gpu, _ = _parity(wl, flags=snn.SNN_FLAG_HBM_RINGS)
    assert gpu["stats"]["lds_rings"] == 0


def test_full_size_audio_256rec_b256():
    """The benchmark workload in the bench's launch configuration, against the
    oracle on the full batch."""
    wl = make_workload(4)
    gpu, orc = _parity(wl)
    st = gpu["stats"]
    assert st["lds_rings"] & 2      # the recurrent LIF layer's rings in LDS
    f = orc["fwd"]
    ev = wl.in_off[-1] * 256 + f.count.sum() * (256 + 20)
    assert st["events"] == ev


def test_full_size_two_layer_1024_sampled_and_batch_linearity():
    """Config 5 at B = 256: spikes of 8 sampled samples bit-exact against the
    oracle run on those samples alone; the B = 256 gradient equals the mean of
    the 16 gradients of its B = 16 sub-batches (exact in real arithmetic: g and
    every adjoint scale by the power of two 256/16)."""
    import torch
    wl = make_workload(5)
    d = to_device(wl)
    full = run_gpu(wl, dev_in=d)
    assert full["rc"] == 0
    pick = [0, 37, 101, 128, 199, 230, 254, 255]
    for b in pick:
        sub = make_workload(5, B=1)
        lo, hi = wl.in_off[b], wl.in_off[b + 1]
        sub.in_off = np.array([0, hi - lo], np.int32)
        sub.in_step, sub.in_neuron = wl.in_step[lo:hi], wl.in_neuron[lo:hi]
        sub.labels = wl.labels[b:b + 1]
        orc = run_oracle(sub, cap=full["net"].record_capacity, modes=())
        f = orc["fwd"]
        for li in range(2):
            c = int(f.count[li, 0])
            assert full["count"][li, b] == c
            assert np.array_equal(full["step"][li, b, :c], f.step[li, 0, :c])
            assert np.array_equal(full["neuron"][li, b, :c], f.neuron[li, 0, :c])
        assert np.array_equal(full["z"][b], f.z[0])
    acc_W = [np.zeros_like(w, dtype=np.float64) for w in full["dW"]]
    acc_D = [np.zeros_like(w, dtype=np.float64) for w in full["dD"]]
    for s in range(16):
        sub = make_workload(5, B=16)
        lo, hi = wl.in_off[16 * s], wl.in_off[16 * s + 16]
        sub.in_off = (wl.in_off[16 * s:16 * s + 17] - lo).astype(np.int32)
        sub.in_step, sub.in_neuron = wl.in_step[lo:hi], wl.in_neuron[lo:hi]
        sub.labels = wl.labels[16 * s:16 * s + 16]
        r = run_gpu(sub)
        for p in range(len(acc_W)):
            acc_W[p] += r["dW"][p] / 16.0
            acc_D[p] += r["dD"][p] / 16.0
    for p in range(len(acc_W)):
        for g, ref in ((full["dW"][p], acc_W[p]), (full["dD"][p], acc_D[p])):
            ok, worst, _ = grad_close(g, ref, rtol=1e-5, atol_rel=1e-7)
            assert ok, worst


def test_forward_is_deterministic():
    wl = make_workload(3, B=32)
    a = run_gpu(wl, backward=True)
    b = run_gpu(wl, backward=True)
    for k in ("count", "step", "neuron", "z", "V", "I", "loss"):
        assert np.array_equal(np.asarray(a[k]).view(np.uint8), np.asarray(b[k]).view(np.uint8)), k
    for x, y in zip(a["dW"] + a["dD"], b["dW"] + b["dD"]):
        assert np.allclose(x, y, rtol=1e-12, atol=1e-12 * np.abs(x).max())


# ------------------------------------------------------------------ edge cases


def test_empty_input_and_empty_samples():
    wl = make_workload(3, B=5)
    off = wl.in_off
    # samples 1 and 3 empty, the others keep their spikes
    keep = np.ones(wl.in_step.size, bool)
    for b in (1, 3):
        keep[off[b]:off[b + 1]] = False
    counts = [int(keep[off[b]:off[b + 1]].sum()) for b in range(wl.B)]
    wl.in_off = np.cumsum([0] + counts).astype(np.int32)
    wl.in_step, wl.in_neuron = wl.in_step[keep], wl.in_neuron[keep]
    gpu, orc = _parity(wl)
    assert gpu["count"][0, 1] == 0 and gpu["count"][0, 3] == 0
    # all samples empty
    wl.in_off = np.zeros(wl.B + 1, np.int32)
    wl.in_step, wl.in_neuron = wl.in_step[:0], wl.in_neuron[:0]
    gpu = run_gpu(wl)
    assert gpu["count"].sum() == 0 and np.all(gpu["z"] == 0)
    assert abs(gpu["loss"][-1] - math.log(wl.cfg.n_classes)) < 1e-6
    assert all(np.all(x == 0) for x in gpu["dW"] + gpu["dD"])


def test_single_step_single_sample_and_zero_max_delay():
    wl = make_workload(1, B=1, T=1, weight_scale=6.0)
    _parity(wl, cap=4)
    wl = make_workload(3, B=3)
    wl.D = [np.zeros_like(d) for d in wl.D]
    gpu = run_gpu(wl, max_delay=0)
    orc = run_oracle(wl, max_delay=0)
    assert_forward_bitexact(gpu, orc, wl)
    assert_backward_close(gpu, orc)


def test_out_of_range_delays_are_clamped_like_the_oracle():
    wl = make_workload(2, B=8)
    D = wl.D[0].copy()
    D[0, :5] = [-3.0, 50.6, 1e9, np.nan, -0.4]
    wl.D[0] = D
    gpu, orc = _parity(wl)
    assert gpu["stats"]["clamped_delays"] == orc["fwd"].clamped == 4


def test_record_overflow_is_reported_and_blocks_backward():
    import paper_2501_07331_amd as snn
    wl = make_workload(3, B=4)
    orc = run_oracle(wl, modes=())
    gpu = run_gpu(wl, cap=3, backward=False)
    assert gpu["rc"] == snn.SNN_EOVERFLOW
    assert np.array_equal(gpu["count"], orc["fwd"].count)
    for b in range(wl.B):
        assert np.array_equal(gpu["step"][0, b, :3], orc["fwd"].step[0, b, :3])
    import torch
    dW = [torch.zeros(w.shape, device="cuda") for w in wl.W]
    with pytest.raises(snn.SNNError) as e:
        gpu["net"].backward(dW, [x.clone() for x in dW])
    assert e.value.code == snn.SNN_EOVERFLOW


def test_backward_before_forward_and_invalid_inputs():
    import torch
    import paper_2501_07331_amd as snn
    wl = make_workload(3, B=4)
    net = make_gpu_net(wl)
    dW = [torch.zeros(w.shape, device="cuda") for w in wl.W]
    with pytest.raises(snn.SNNError) as e:
        net.backward(dW, [x.clone() for x in dW])
    assert e.value.code == snn.SNN_ESTATE
    d = to_device(wl)
    B, cap = wl.B, net.record_capacity
    recs = [(torch.zeros(B, dtype=torch.int32, device="cuda"),
             torch.zeros(B, cap, dtype=torch.int32, device="cuda"),
             torch.zeros(B, cap, dtype=torch.int32, device="cuda"))]
    loss = torch.zeros(B + 1, device="cuda")

    def fwd(**kw):
        a = dict(d)
        a.update(kw)
        return net.forward(a["off"], a["step"], a["neuron"], a["W"], a["D"], a["labels"], recs, loss)

    bad_order = d["step"].clone()
    lo = int(wl.in_off[1])
    bad_order[lo], bad_order[lo + 1] = d["step"][lo + 1].clone(), d["step"][lo].clone()
    if int(wl.in_step[lo]) == int(wl.in_step[lo + 1]):
        bad_neuron = d["neuron"].clone()
        bad_neuron[lo], bad_neuron[lo + 1] = d["neuron"][lo + 1].clone(), d["neuron"][lo].clone()
        cases = [dict(neuron=bad_neuron)]
    else:
        cases = [dict(step=bad_order)]
    big = d["neuron"].clone()
    big[3] = wl.cfg.layers[0][0]
    late = d["step"].clone()
    late[-1] = wl.T
    bad_off = d["off"].clone()
    bad_off[2] = bad_off[3] + 1
    bad_lab = d["labels"].clone()
    bad_lab[0] = wl.cfg.n_classes
    cases += [dict(neuron=big), dict(step=late), dict(off=bad_off), dict(labels=bad_lab)]
    for kw in cases:
        with pytest.raises(snn.SNNError) as e:
            fwd(**kw)
        assert e.value.code == snn.SNN_EINVAL, kw.keys()
        with pytest.raises(snn.SNNError) as e:
            net.backward(dW, [x.clone() for x in dW])
        assert e.value.code == snn.SNN_ESTATE
    assert fwd() == 0      # the handle is still usable


def test_parity_two_layers_of_unequal_width():
    """A 32-neuron recurrent layer feeding a 96-neuron recurrent one: the
    narrow layer has two LIF-post projections and the wide one a single one,
    so the wide layer's unused projection entry stands in with the 32-row
    recurrent matrix of the narrow layer (its loads must stay in its rows).
    Both layers spike (about 15 and 20 spikes per neuron and sample)."""
    import dataclasses

    from workloads import Workload
    from workloads.configs import CONFIGS
    from workloads.generators import input_spikes, labels

    cfg = dataclasses.replace(CONFIGS[3], name="uneven-12-32rec-96rec-27",
                              layers=((12, 0, 0), (32, 1, 1), (96, 1, 1), (27, 2, 0)),
                              delay_range=(25, 25, 25, 25, 25))
    B, T = 6, 300
    off, st, ne = input_spikes(cfg, B, T=T)
    shapes = [(12, 32), (32, 32), (32, 96), (96, 96), (96, 27)]
    mus = (1.4, 0.0, 0.25, 0.0, 0.05)
    rng = np.random.default_rng(77)
    W = [rng.normal(m, 0.3 if p in (0, 2) else 0.05, size=s).astype(np.float32)
         for p, (m, s) in enumerate(zip(mus, shapes))]
    D = [rng.uniform(0.0, 25.0, size=s).astype(np.float32) for s in shapes]
    wl = Workload(cfg, B, T, off, st, ne, W, D, labels(cfg, B))
    import paper_2501_07331_amd as snn
    gpu, orc = _parity(wl)
    assert all(int(c.sum()) > 0 for c in orc["fwd"].count)
    _parity(wl, flags=snn.SNN_FLAG_HBM_RINGS)


# ------------------------------------------------- long delays, fine grids


@pytest.mark.parametrize("cid,B,rng_,flags", [
    (4, 4, (255, 255, 255), 0),          # S = 256: delay and adjoint rings in device memory
    (4, 4, (255, 50, 255), 0),
    (4, 4, (0, 0, 0), 0),                # every delay zero (plain EventProp)
    (3, 16, (255, 255, 255), 0),         # 128 posts: S = 256 rings still fit in LDS
    (3, 16, (255, 255, 255), 1),
])
def test_parity_max_delay_sweep_shapes(cid, B, rng_, flags):
    from workloads import make_variant
    wl = make_variant(cid, B=B, delay_range=rng_)
    gpu, orc = _parity(wl, flags=flags)
    assert orc["fwd"].count.sum() > 0


def test_parity_fine_dt_long_T():
    """dt = 0.1 ms, T = 10^4 steps (the same 1 s trials at ten times the
    resolution), delays up to 255 steps: the gradient kernel's trajectories
    no longer fit 8 or 4 posts per workgroup, the readout tables leave LDS."""
    from workloads import make_variant
    wl = make_variant(4, B=2, T=10000, dt=0.1, delay_range=(255, 50, 255))
    print(f"[parity] fine dt B={wl.B} T={wl.T}", flush=True)
    gpu = run_gpu(wl)
    orc = run_oracle(wl)
    assert gpu["rc"] == 0 and orc["fwd"].count.sum() > 0
    assert_forward_bitexact(gpu, orc, wl)
    assert np.allclose(gpu["loss"], orc["loss"], rtol=1e-6, atol=1e-7)
    assert_backward_close(gpu, orc)


def test_parity_synchronous_bursts():
    """Input spikes that drive every hidden neuron over threshold within a
    step or two: steps with up to all 256 neurons spiking at once, so the
    step's spike list is filled by every wave and read in many chunks by the
    scatter and the readout wave (the 700-256rec-20 network, B = 2)."""
    import dataclasses

    from workloads import Workload
    from workloads.configs import CONFIGS
    from workloads.generators import labels

    cfg = dataclasses.replace(CONFIGS[4], name="bursts-700-256rec-20")
    B, T = 2, 200
    rng = np.random.default_rng(2024)
    steps, neurons, off = [], [], [0]
    for b in range(B):
        t = np.sort(rng.choice(np.arange(5, T - 20), size=6, replace=False))
        steps.append(t)
        neurons.append(rng.integers(0, 700, size=t.size))
        off.append(off[-1] + t.size)
    st = np.concatenate(steps).astype(np.int32)
    ne = np.concatenate(neurons).astype(np.int32)
    off = np.array(off, dtype=np.int32)
    W = [rng.uniform(9.5, 10.5, size=(700, 256)).astype(np.float32),
         rng.normal(0.0, 0.02, size=(256, 256)).astype(np.float32),
         rng.normal(0.0, 0.1, size=(256, 20)).astype(np.float32)]
    D = [np.zeros((700, 256), dtype=np.float32),
         rng.uniform(0.0, 50.0, size=(256, 256)).astype(np.float32),
         rng.uniform(0.0, 150.0, size=(256, 20)).astype(np.float32)]
    wl = Workload(cfg, B, T, off, st, ne, W, D, labels(cfg, B))
    gpu, orc = _parity(wl)
    f = orc["fwd"]
    most = 0
    for b in range(B):
        c = int(f.count[0, b])
        most = max(most, int(np.bincount(f.step[0, b, :c], minlength=T).max()))
    print(f"[bursts] most spikes in one step of a sample: {most}", flush=True)
    assert most >= 200
