"""Helpers that drive the HIP library (through its C ABI) and the oracle on the
same seeded workload, and compare them."""
from __future__ import annotations

import numpy as np

import oracle
from workloads import Workload


def default_cap(wl: Workload) -> int:
    """Record capacity per sample and LIF layer: 64 spikes per neuron."""
    lif = [l[0] for l in wl.cfg.layers if l[1] == 1]
    return 64 * max(lif + [1])


def oracle_net(wl: Workload, max_delay=None):
    c = wl.cfg
    return oracle.OracleNet(c.layers, c.tau_m, c.tau_s, c.theta, c.dt,
                            c.max_delay if max_delay is None else max_delay, wl.T, c.loss,
                            c.readout_scale)


def run_oracle(wl: Workload, cap=None, modes=("f64", "f32"), max_delay=None, dlp=None):
    """dlp: extra per-record dl_p/dt_k [n_lif][B][cap] (fp64) or None."""
    cap = default_cap(wl) if cap is None else cap
    net = oracle_net(wl, max_delay)
    f = oracle.forward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, cap=cap)
    if wl.cfg.loss == oracle.LOSS_DMSE:
        lo, dl = oracle.loss_dmse(f.z, wl.labels, wl.cfg.dmse_delta)
        g = np.zeros_like(f.z)
        x = oracle.first_spike_dlp(net, f, dl)
        x = x if dlp is None else x + dlp
    else:
        lo, g = oracle.loss(f.z, wl.labels)
        x = dlp
    out = {"fwd": f, "loss": lo, "g": g}
    for m in modes:
        dW, dD, deg = oracle.backward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, f, g,
                                      mode=m, dlp=x)
        out[m] = (dW, dD, deg)
    return out


def make_gpu_net(wl: Workload, cap=None, flags=0, max_delay=None):
    import paper_2501_07331_amd as snn
    c = wl.cfg
    cap = default_cap(wl) if cap is None else cap
    return snn.Network(c.layers, c.tau_m, c.tau_s, c.theta, c.dt,
                       c.max_delay if max_delay is None else max_delay, wl.B, wl.T, c.loss,
                       c.readout_scale, cap, flags, dmse_delta=c.dmse_delta)


def to_device(wl: Workload):
    import torch
    dev = torch.device("cuda")
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(device=dev, dtype=dt)
    return {
        "off": t(wl.in_off, torch.int32), "step": t(wl.in_step, torch.int32),
        "neuron": t(wl.in_neuron, torch.int32),
        "W": [t(w, torch.float32) for w in wl.W], "D": [t(d, torch.float32) for d in wl.D],
        "labels": t(wl.labels, torch.int32),
    }


def run_gpu(wl: Workload, net=None, cap=None, flags=0, backward=True, max_delay=None, dev_in=None,
            dlp=None):
    """Forward (+ backward) through the library; returns numpy results.
    dlp: per LIF layer None or an fp32 [B][cap] array of dl_p/dt_k."""
    import torch
    import paper_2501_07331_amd as snn
    net = make_gpu_net(wl, cap, flags, max_delay) if net is None else net
    cap = net.record_capacity
    d = to_device(wl) if dev_in is None else dev_in
    dev = torch.device("cuda")
    B, C = wl.B, wl.cfg.n_classes
    recs = [(torch.zeros(B, dtype=torch.int32, device=dev),
             torch.full((B, cap), -1, dtype=torch.int32, device=dev),
             torch.full((B, cap), -1, dtype=torch.int32, device=dev)) for _ in net.lif_layers]
    loss = torch.zeros(B + 1, dtype=torch.float32, device=dev)
    z = torch.zeros(B, C, dtype=torch.float32, device=dev)
    out = {"net": net}
    try:
        net.forward(d["off"], d["step"], d["neuron"], d["W"], d["D"], d["labels"], recs, loss, z)
        out["rc"] = 0
    except snn.SNNOverflow:
        out["rc"] = snn.SNN_EOVERFLOW
    torch.cuda.synchronize()
    out["count"] = np.stack([r[0].cpu().numpy() for r in recs]) if recs else np.zeros((0, B), np.int32)
    out["step"] = np.stack([r[1].cpu().numpy() for r in recs]) if recs else None
    out["neuron"] = np.stack([r[2].cpu().numpy() for r in recs]) if recs else None
    out["loss"] = loss.cpu().numpy()
    out["z"] = z.cpu().numpy()
    Vs, Is = [], []
    for l in range(1, len(wl.cfg.layers)):
        n = wl.cfg.layers[l][0]
        V = torch.zeros(B, n, dtype=torch.float32, device=dev)
        I = torch.zeros(B, n, dtype=torch.float32, device=dev)
        net.state(l, V, I)
        Vs.append(V.cpu().numpy())
        Is.append(I.cpu().numpy())
    out["V"] = np.concatenate(Vs, axis=1)
    out["I"] = np.concatenate(Is, axis=1)
    if backward and out["rc"] == 0:
        dW = [torch.full_like(w, np.nan) for w in d["W"]]
        dD = [torch.full_like(w, np.nan) for w in d["W"]]
        if dlp is None:
            net.backward(dW, dD)
        else:
            net.backward(dW, dD, [None if x is None else
                                  torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(dev)
                                  for x in dlp])
        torch.cuda.synchronize()
        out["dW"] = [x.cpu().numpy() for x in dW]
        out["dD"] = [x.cpu().numpy() for x in dD]
    out["stats"] = net.stats()
    return out


def grad_close(gpu, ref, rtol=1e-4, atol_rel=1e-6):
    """|gpu - ref| <= atol_rel * max|ref| + rtol * |ref| elementwise (the abs
    tolerance is taken relative to the tensor's scale: the gradients of a
    batch-mean loss with a time-averaged readout are far below 1)."""
    ref = np.asarray(ref, np.float64)
    gpu = np.asarray(gpu, np.float64)
    scale = np.abs(ref).max()
    err = np.abs(gpu - ref)
    ok = err <= atol_rel * scale + rtol * np.abs(ref)
    worst = float((err / (atol_rel * scale + rtol * np.abs(ref) + 1e-300)).max()) if err.size else 0.0
    return bool(ok.all()), worst, float(err.max() / scale) if scale > 0 else float(err.max())


def assert_forward_bitexact(gpu, orc, wl):
    f = orc["fwd"]
    nl = gpu["count"].shape[0]
    assert np.array_equal(gpu["count"], f.count[:nl]), "spike counts differ"
    for li in range(nl):
        for b in range(wl.B):
            c = min(int(f.count[li, b]), f.cap)
            assert np.array_equal(gpu["step"][li, b, :c], f.step[li, b, :c]), (li, b, "steps")
            assert np.array_equal(gpu["neuron"][li, b, :c], f.neuron[li, b, :c]), (li, b, "neurons")
    assert np.array_equal(gpu["z"].view(np.uint32), f.z.view(np.uint32)), "readout z differs"
    assert np.array_equal(gpu["V"].view(np.uint32), f.V_final.view(np.uint32)), "final V differs"
    assert np.array_equal(gpu["I"].view(np.uint32), f.I_final.view(np.uint32)), "final I differs"


def assert_backward_close(gpu, orc, rtol=1e-4, atol_rel=1e-6, f64_bound=1e-4, model_gap=False):
    """GPU vs the fp32 kernel-precision model at the stated tolerance, and vs
    the fp64 definition within f64_bound of each tensor's scale.  With
    model_gap, the fp64 bound of a tensor is at least twice the distance of
    the oracle's own fp32 model from its fp64 definition (fp32 adjoints lose
    accuracy over long, spike-dense trials: about 1e-3 of scale at T = 10^4)."""
    dW32, dD32, deg32 = orc["f32"]
    assert gpu["stats"]["degenerate_jumps"] == deg32
    for p in range(len(dW32)):
        for nm, g, r in (("dW", gpu["dW"][p], dW32[p]), ("dD", gpu["dD"][p], dD32[p])):
            ok, worst, _ = grad_close(g, r, rtol, atol_rel)
            assert ok, f"{nm}[{p}] vs fp32 model: worst error / tolerance = {worst:.3g}"
    if "f64" in orc:
        dW64, dD64, _ = orc["f64"]
        for p in range(len(dW64)):
            for nm, g, r in (("dW", gpu["dW"][p], dW64[p]), ("dD", gpu["dD"][p], dD64[p])):
                scale = np.abs(r).max()
                err = np.abs(g.astype(np.float64) - r).max()
                bound = f64_bound
                if model_gap:
                    m32 = (dW32 if nm == "dW" else dD32)[p]
                    bound = max(bound, 2.0 * np.abs(m32.astype(np.float64) - r).max() / scale)
                assert err <= bound * scale + 1e-30, f"{nm}[{p}] vs fp64: {err / scale:.3g} of scale"
