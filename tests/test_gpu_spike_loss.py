"""Spike-time loss terms on the GPU (through the C ABI) against the oracle:
the time-invariant MSE on first output spikes of a LIF output layer
(Methods, "Time-invariant mean squared error loss") and per-record
dl_p/dt_k terms added to the lambda_V jumps of any LIF layer
(snn_backward_lp).  Spikes, first-spike times (z) and the loss are
bit-exact; dW and dD within the usual tolerance of the fp32 model and the
fp64 definition."""
import numpy as np
import pytest

from workloads import LOSS_DMSE, make_variant

from .gpu_util import assert_backward_close, assert_forward_bitexact, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

YY_LIF_OUT = ((4, 0, 0), (200, 1, 0), (3, 1, 0))


def _dmse(B=16, delta=1.0, **kw):
    return make_variant(2, B=B, layers=YY_LIF_OUT, loss=LOSS_DMSE, dmse_delta=delta,
                        name="latency-4-200-3lif", **kw)


def _check(wl, gpu, orc):
    assert gpu["rc"] == 0
    assert_forward_bitexact(gpu, orc, wl)
    assert np.array_equal(gpu["loss"].view(np.uint32), orc["loss"].view(np.uint32))
    assert_backward_close(gpu, orc)


@pytest.mark.parametrize("B,delta,flags", [(16, 1.0, 0), (64, 2.5, 0), (16, 1.0, 1)])
def test_dmse_parity(B, delta, flags):
    print(f"[dmse] B={B} delta={delta} flags={flags}", flush=True)
    wl = _dmse(B, delta)
    gpu = run_gpu(wl, flags=flags)
    orc = run_oracle(wl)
    assert orc["fwd"].count[1].min() > 0          # every sample's output layer fires
    _check(wl, gpu, orc)
    # z holds the first output spike times in ms
    f = orc["fwd"]
    b = 0
    c = int(f.count[1, b])
    k = int(f.neuron[1, b, 0])
    assert gpu["z"][b, k] == np.float32(f.step[1, b, 0] * np.float64(np.float32(wl.cfg.dt)))
    assert c > 3


def test_dmse_silent_output_neuron():
    """An output neuron that never fires: its time is T dt in the loss and it
    carries no jump; the others still get theirs."""
    wl = _dmse(8)
    wl.W[1][:, 2] = -1.0                            # output 2 is silenced
    gpu = run_gpu(wl)
    orc = run_oracle(wl)
    assert np.all(orc["fwd"].z[:, 2] == np.float32(wl.T * np.float64(np.float32(wl.cfg.dt))))
    _check(wl, gpu, orc)


@pytest.mark.parametrize("cid,B", [(3, 16), (1, 32)])
def test_hidden_spike_time_terms(cid, B):
    """Random dl_p/dt_k on every hidden record of a CE-trained net: the jump
    terms of the layer that feeds the readout are summed with the readout
    part of its jump sums."""
    from workloads import make_workload
    wl = make_workload(cid, B=B, weight_scale=6.0 if cid == 1 else 1.0)
    from .gpu_util import default_cap
    cap = default_cap(wl)
    rng = np.random.default_rng(9)
    x = rng.normal(0, 1e-3, size=(1, B, cap)).astype(np.float32)
    gpu = run_gpu(wl, dlp=[x[0]])
    orc = run_oracle(wl, dlp=x.astype(np.float64))
    _check(wl, gpu, orc)
    # and the term matters
    base = run_oracle(wl, modes=("f64",))
    assert np.abs(base["f64"][0][0] - orc["f64"][0][0]).max() > 1e-3 * np.abs(base["f64"][0][0]).max()


def test_dmse_with_terms_on_both_layers_and_zero_terms_change_nothing():
    wl = _dmse(16)
    from .gpu_util import default_cap
    cap = default_cap(wl)
    rng = np.random.default_rng(4)
    x = rng.normal(0, 1e-2, size=(2, wl.B, cap)).astype(np.float32)
    gpu = run_gpu(wl, dlp=[x[0], x[1]])
    orc = run_oracle(wl, dlp=x.astype(np.float64))
    _check(wl, gpu, orc)
    a = run_gpu(wl)
    z = run_gpu(wl, dlp=[np.zeros((wl.B, cap), np.float32), None])
    for u, v in zip(a["dW"] + a["dD"], z["dW"] + z["dD"]):
        assert np.array_equal(u.view(np.uint32), v.view(np.uint32))


def test_dmse_training_lowers_the_loss():
    """Adam on weights and delays with the spike-time loss, all on the GPU."""
    import torch
    import paper_2501_07331_amd as snn
    from .gpu_util import make_gpu_net, to_device
    wl = _dmse(64, 1.0)
    net = make_gpu_net(wl)
    d = to_device(wl)
    W, D = d["W"], d["D"]
    B, cap = wl.B, net.record_capacity
    recs = [(torch.zeros(B, dtype=torch.int32, device="cuda"),
             torch.zeros(B, cap, dtype=torch.int32, device="cuda"),
             torch.zeros(B, cap, dtype=torch.int32, device="cuda")) for _ in net.lif_layers]
    loss = torch.zeros(B + 1, device="cuda")
    dW = [torch.zeros_like(w) for w in W]
    dD = [torch.zeros_like(w) for w in W]
    losses = []
    for it in range(30):
        net.forward(d["off"], d["step"], d["neuron"], W, D, d["labels"], recs, loss)
        net.backward(dW, dD)
        losses.append(float(loss[-1].item()))
        net.optimizer_step(W, D, dW, dD, kind=snn.SNN_OPT_ADAM, lr_w=2e-3, lr_d=0.5)
    print(f"[dmse train] loss {losses[0]:.4f} -> {losses[-1]:.4f}", flush=True)
    assert losses[-1] < 0.7 * losses[0]
