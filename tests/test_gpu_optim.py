"""Optimiser step on the GPU (through the C ABI) against the fp64 optimiser
oracle, and the training loop closed on the GPU: the paper's sequence-detection
example (Results, "Sequence detection task") learned with delay updates only,
step for step beside the oracle, and a synthetic-task learning curve."""
import numpy as np
import pytest

import oracle
from oracle.optim import Optimiser
from workloads import make_workload

from .gpu_util import assert_backward_close, assert_forward_bitexact, run_gpu, run_oracle, to_device

pytestmark = pytest.mark.gpu


def _ulp(x):
    return np.spacing(np.abs(np.asarray(x, np.float32))).astype(np.float64)


def _check_update(new_gpu, old, new_ref, rtol=1e-5):
    """The GPU's fp32 update (new - old) within rtol of the fp64 update, plus
    the rounding of the result to fp32 (two ulps of it)."""
    new_gpu = np.asarray(new_gpu, np.float64)
    old = np.asarray(old, np.float64)
    du_g, du_r = new_gpu - old, np.asarray(new_ref, np.float64) - old
    tol = rtol * np.abs(du_r) + 2.0 * _ulp(new_ref) + 2.0 * _ulp(old)
    err = np.abs(du_g - du_r)
    assert np.all(err <= tol), float((err / tol).max())


def _rand_params(wl, rng):
    dW = [rng.normal(0, 1e-3, size=w.shape).astype(np.float32) for w in wl.W]
    dD = [rng.normal(0, 1e-4, size=w.shape).astype(np.float32) for w in wl.W]
    return dW, dD


@pytest.mark.parametrize("kind", ["sgd", "adam"])
def test_optimizer_step_matches_oracle(kind):
    import torch
    import paper_2501_07331_amd as snn
    from .gpu_util import make_gpu_net
    print(f"[optim] {kind}", flush=True)
    wl = make_workload(3, B=4)
    net = make_gpu_net(wl)
    rng = np.random.default_rng(11)
    W = [torch.from_numpy(w.copy()).cuda() for w in wl.W]
    D = [torch.from_numpy(d.copy()).cuda() for d in wl.D]
    ref = Optimiser(kind)
    Wr, Dr = [w.astype(np.float64) for w in wl.W], [d.astype(np.float64) for d in wl.D]
    k = snn.SNN_OPT_SGD if kind == "sgd" else snn.SNN_OPT_ADAM
    lr_w, lr_d = (0.5, 100.0) if kind == "sgd" else (1e-3, 0.5)
    sw, sd = [1.0, 0.5, 2.0], [1.0, 0.0, 1.0]
    for it in range(3):
        dW, dD = _rand_params(wl, rng)
        old_W = [w.cpu().numpy() for w in W]
        old_D = [d.cpu().numpy() for d in D]
        net.optimizer_step(W, D, [torch.from_numpy(x).cuda() for x in dW],
                           [torch.from_numpy(x).cuda() for x in dD], kind=k, lr_w=lr_w, lr_d=lr_d,
                           d_min=0.0, d_max=25.0, lr_scale_w=sw, lr_scale_d=sd)
        torch.cuda.synchronize()
        # the oracle steps from the GPU's previous fp32 state, as the GPU does
        Wr, Dr = ref.step(old_W, old_D, dW, dD, lr_w, lr_d, 0.0, 25.0, sw, sd)
        for p in range(len(W)):
            _check_update(W[p].cpu().numpy(), old_W[p], Wr[p])
            _check_update(D[p].cpu().numpy(), old_D[p], Dr[p])
            assert D[p].min().item() >= 0.0 and D[p].max().item() <= 25.0
        assert np.array_equal(D[1].cpu().numpy(), np.clip(old_D[1], 0.0, 25.0))   # frozen
    # reset: the next Adam step is a first step again
    if kind == "adam":
        net.optimizer_reset()
        ref = Optimiser(kind)
        dW, dD = _rand_params(wl, rng)
        old_W = [w.cpu().numpy() for w in W]
        old_D = [d.cpu().numpy() for d in D]
        net.optimizer_step(W, D, [torch.from_numpy(x).cuda() for x in dW],
                           [torch.from_numpy(x).cuda() for x in dD], kind=k, lr_w=lr_w, lr_d=lr_d,
                           d_min=0.0, d_max=25.0)
        torch.cuda.synchronize()
        Wr, Dr = ref.step(old_W, old_D, dW, dD, lr_w, lr_d, 0.0, 25.0)
        for p in range(len(W)):
            _check_update(W[p].cpu().numpy(), old_W[p], Wr[p])


def test_optimizer_rejects_bad_arguments():
    import torch
    import paper_2501_07331_amd as snn
    from .gpu_util import make_gpu_net
    wl = make_workload(1, B=2)
    net = make_gpu_net(wl)
    W = [torch.from_numpy(w.copy()).cuda() for w in wl.W]
    D = [torch.from_numpy(d.copy()).cuda() for d in wl.D]
    for kw in (dict(kind=7), dict(lr_w=-1.0), dict(lr_d=float("inf")), dict(d_min=5.0, d_max=1.0),
               dict(beta1=1.0), dict(eps=0.0), dict(lr_scale_w=[-1.0] * len(W))):
        with pytest.raises(snn.SNNError) as e:
            net.optimizer_step(W, D, W, D, **kw)
        assert e.value.code == snn.SNN_EINVAL


# ------------------------------------------------------- sequence detection


def test_sequence_detection_learns_on_the_gpu_like_the_oracle():
    """Delay-only SGD on the paper's two-input / two-output example, every
    forward, backward and update on the GPU, beside the same loop on the
    oracle: spikes bit-exact (inputs only here), z bit-exact while the delays
    agree, delays within the update tolerance, and the same number of
    presentations to 100 % accuracy (at most 10)."""
    import json
    import os
    import torch
    import paper_2501_07331_amd as snn
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "sequence_detection.json")))
    TM, TS, T, MAXD, LR = 20.0, 5.0, 60, 30, 300.0
    layers = ((2, snn.SNN_INPUT, 0), (2, snn.SNN_LI, 0))
    net = snn.Network(layers, TM, TS, 1.0, 1.0, MAXD, 1, T, snn.SNN_LOSS_CE_MAX, 1.0, 4)
    onet = oracle.OracleNet(layers, TM, TS, 1.0, 1.0, MAXD, T, snn.SNN_LOSS_CE_MAX, 1.0)
    W = np.array(g["weights"], np.float32)
    D = np.array(g["initial_delays_ms"], np.float32)
    Wd = [torch.from_numpy(W.copy()).cuda()]
    Dd = [torch.from_numpy(D.copy()).cuda()]
    dW = [torch.zeros_like(Wd[0])]
    dD = [torch.zeros_like(Wd[0])]
    ref = Optimiser("sgd")
    Dr = D.copy()

    def example(cls):
        ev = sorted((int(t), int(i)) for t, i in g["class_inputs_ms"][str(cls)])
        return (np.array([0, len(ev)], np.int32), np.array([e[0] for e in ev], np.int32),
                np.array([e[1] for e in ev], np.int32))

    def gpu_fwd(cls):
        off, st, ne = (torch.from_numpy(a).cuda() for a in example(cls))
        lab = torch.tensor([cls], dtype=torch.int32, device="cuda")
        loss = torch.zeros(2, device="cuda")
        z = torch.zeros(1, 2, device="cuda")
        net.forward(off, st, ne, Wd, Dd, lab, [], loss, z)
        return z.cpu().numpy()[0], (off, st, ne, lab, loss)

    def accuracy():
        return sum(int(np.argmax(gpu_fwd(c)[0]) == c) for c in (0, 1)) / 2

    assert accuracy() == 0.0
    seen = 0
    while accuracy() < 1.0:
        assert seen < 10
        for cls in (0, 1):
            z, keep = gpu_fwd(cls)
            net.backward(dW, dD)
            f = oracle.forward(onet, *example(cls), [W], [Dr])
            assert np.array_equal(z.view(np.uint32), f.z[0].view(np.uint32))
            lo, gg = oracle.loss(f.z, [cls])
            _, dDr, _ = oracle.backward(onet, *example(cls), [W], [Dr], f, gg)
            old = Dd[0].cpu().numpy()
            net.optimizer_step(Wd, Dd, dW, dD, kind=snn.SNN_OPT_SGD, lr_w=0.0, lr_d=LR,
                               d_min=0.0, d_max=float(MAXD))
            torch.cuda.synchronize()
            _, Dn = ref.step([W], [old], [np.zeros_like(W)], dDr, 0.0, LR, 0.0, float(MAXD))
            # dD agrees to 1e-4 of its scale, so the step agrees to 1e-4 of lr * |dD|
            tol = 1e-4 * LR * np.abs(dDr[0]).max() + 2 * _ulp(Dn[0])
            assert np.all(np.abs(Dd[0].cpu().numpy() - Dn[0]) <= tol)
            assert np.array_equal(Wd[0].cpu().numpy(), W)
            Dr = Dd[0].cpu().numpy()      # both loops continue from the GPU's delays
        seen += 1
    print(f"[seqdet] 100 % after {seen} presentations of each class; delays {Dd[0].cpu().numpy().tolist()}",
          flush=True)


def test_training_loop_learning_curve_tactile():
    """Adam with the paper's SHD learning rates (weights 1e-3 eased in, delays
    0.1) on a fixed synthetic batch of the 12-128rec-27 config: the first
    full step (forward, backward, update) matches the oracle, and 40 steps
    lower the loss."""
    import torch
    import paper_2501_07331_amd as snn
    from paper_2501_07331_amd import schedules
    from .gpu_util import make_gpu_net
    wl = make_workload(3, B=32)
    gpu = run_gpu(wl)
    orc = run_oracle(wl)
    assert_forward_bitexact(gpu, orc, wl)
    assert_backward_close(gpu, orc)
    net = gpu["net"]
    d = to_device(wl)
    W, D = d["W"], d["D"]
    B, cap = wl.B, net.record_capacity
    recs = [(torch.zeros(B, dtype=torch.int32, device="cuda"),
             torch.zeros(B, cap, dtype=torch.int32, device="cuda"),
             torch.zeros(B, cap, dtype=torch.int32, device="cuda")) for _ in net.lif_layers]
    loss = torch.zeros(B + 1, device="cuda")
    dW = [torch.zeros_like(w) for w in W]
    dD = [torch.zeros_like(w) for w in W]
    ref = Optimiser("adam")
    losses = []
    for it in range(40):
        lr_w = schedules.ease_in(1e-2, it, start=0.1, growth=1.1)
        net.forward(d["off"], d["step"], d["neuron"], W, D, d["labels"], recs, loss)
        net.backward(dW, dD)
        losses.append(float(loss[-1].item()))
        if it == 0:
            old_W = [w.cpu().numpy() for w in W]
            old_D = [x.cpu().numpy() for x in D]
            Wr, Dr = ref.step(old_W, old_D, orc["f64"][0], orc["f64"][1], lr_w, 0.1, 0.0,
                              float(wl.cfg.max_delay))
        net.optimizer_step(W, D, dW, dD, kind=snn.SNN_OPT_ADAM, lr_w=lr_w, lr_d=0.1)
        if it == 0:
            torch.cuda.synchronize()
            # Adam divides by sqrt(v): near-zero gradients give steps of lr
            # whichever way rounding tips them, so compare where |g| is not
            # tiny against its own tensor, and bound every step by lr
            for p in range(len(W)):
                for new, old, rf, gr, lr in ((W[p], old_W[p], Wr[p], orc["f64"][0][p], lr_w),
                                             (D[p], old_D[p], Dr[p], orc["f64"][1][p], 0.1)):
                    new = new.cpu().numpy().astype(np.float64)
                    big = np.abs(gr) > 1e-2 * np.abs(gr).max()
                    du_g, du_r = new - old, rf - old
                    assert np.all(np.abs(du_g) <= lr * (1 + 1e-5) + 2 * _ulp(new))
                    assert np.all(np.abs(du_g - du_r)[big] <= 1e-3 * lr + 2 * _ulp(rf)[big])
    print(f"[train] loss {losses[0]:.4f} -> {losses[-1]:.4f}", flush=True)
    assert losses[-1] < 0.9 * losses[0]
