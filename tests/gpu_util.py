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


def proj_delays(wl: Workload, max_delay=None, per_proj=True):
    """(network-wide max delay, per-projection largest delays or None): each
    projection's delay range of the config, capped at max_delay if given."""
    c = wl.cfg
    md = c.max_delay if max_delay is None else max_delay
    return md, ([min(r, md) for r in c.delay_range] if per_proj else None)


def oracle_net(wl: Workload, max_delay=None, per_proj=True):
    c = wl.cfg
    md, pm = proj_delays(wl, max_delay, per_proj)
    return oracle.OracleNet(c.layers, c.tau_m, c.tau_s, c.theta, c.dt, md, wl.T, c.loss,
                            c.readout_scale, pm)


def run_oracle(wl: Workload, cap=None, modes=("f64", "f32"), max_delay=None, dlp=None,
               per_proj=True, reg=None):
    """dlp: extra per-record dl_p/dt_k [n_lif][B][cap] (fp64) or None; reg:
    (strength per LIF layer, target) of the spike-count regulariser or None."""
    cap = default_cap(wl) if cap is None else cap
    net = oracle_net(wl, max_delay, per_proj)
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
    if reg is not None:
        # the parameter values the library receives (fp32 in its options)
        R, rd = oracle.spike_count_reg(net, f, [float(np.float32(x)) for x in reg[0]],
                                       float(np.float32(reg[1])))
        out["reg_loss"] = R
        x = rd if x is None else x + rd
    for m in modes:
        dW, dD, deg = oracle.backward(net, wl.in_off, wl.in_step, wl.in_neuron, wl.W, wl.D, f, g,
                                      mode=m, dlp=x)
        out[m] = (dW, dD, deg)
    return out


def make_gpu_net(wl: Workload, cap=None, flags=0, max_delay=None, per_proj=True, reg=None):
    """reg: (strength per LIF layer, target) of the spike-count regulariser."""
    import paper_2501_07331_amd as snn
    c = wl.cfg
    cap = default_cap(wl) if cap is None else cap
    md, pm = proj_delays(wl, max_delay, per_proj)
    kw = {} if reg is None else dict(reg_strength=list(reg[0]), reg_target=float(reg[1]))
    return snn.Network(c.layers, c.tau_m, c.tau_s, c.theta, c.dt, md, wl.B, wl.T, c.loss,
                       c.readout_scale, cap, flags, dmse_delta=c.dmse_delta, proj_max_delay=pm, **kw)


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
            dlp=None, per_proj=True, reg=None, noalloc=False):
    """Forward (+ backward) through the library; returns numpy results.
    dlp: per LIF layer None or an fp32 [B][cap] array of dl_p/dt_k; reg as
    make_gpu_net; noalloc: the backward through snn_backward_noalloc."""
    import torch
    import paper_2501_07331_amd as snn
    net = make_gpu_net(wl, cap, flags, max_delay, per_proj, reg) if net is None else net
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
    if out["rc"] in (0, snn.SNN_EOVERFLOW) and recs:
        Im = []
        for l in net.lif_layers:
            x = torch.zeros(B, cap, dtype=torch.float32, device=dev)
            net.record_currents(l, x)
            Im.append(x.cpu().numpy())
        out["I_minus"] = np.stack(Im)
    if backward and out["rc"] == 0:
        dW = [torch.full_like(w, np.nan) for w in d["W"]]
        dD = [torch.full_like(w, np.nan) for w in d["W"]]
        if noalloc:
            assert dlp is None
            net.backward_noalloc(dW, dD)
        elif dlp is None:
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
    """|gpu - ref| <= atol_rel * max|ref| + rtol * |ref| elementwise, for
    comparisons of GPU results with each other (batch linearity)."""
    ref = np.asarray(ref, np.float64)
    gpu = np.asarray(gpu, np.float64)
    scale = np.abs(ref).max()
    err = np.abs(gpu - ref)
    ok = err <= atol_rel * scale + rtol * np.abs(ref)
    worst = float((err / (atol_rel * scale + rtol * np.abs(ref) + 1e-300)).max()) if err.size else 0.0
    return bool(ok.all()), worst, float(err.max() / scale) if scale > 0 else float(err.max())


def assert_forward_bitexact(gpu, orc, wl):
    """Spike counts, records (step, neuron, I- at the spike), z and the final
    V and I equal to the oracle's, bit for bit."""
    f = orc["fwd"]
    nl = gpu["count"].shape[0]
    assert np.array_equal(gpu["count"], f.count[:nl]), "spike counts differ"
    for li in range(nl):
        for b in range(wl.B):
            c = min(int(f.count[li, b]), f.cap)
            assert np.array_equal(gpu["step"][li, b, :c], f.step[li, b, :c]), (li, b, "steps")
            assert np.array_equal(gpu["neuron"][li, b, :c], f.neuron[li, b, :c]), (li, b, "neurons")
            if "I_minus" in gpu:
                assert np.array_equal(gpu["I_minus"][li, b, :c].view(np.uint32),
                                      f.I_minus[li, b, :c].view(np.uint32)), (li, b, "I- records")
    assert np.array_equal(gpu["z"].view(np.uint32), f.z.view(np.uint32)), "readout z differs"
    assert np.array_equal(gpu["V"].view(np.uint32), f.V_final.view(np.uint32)), "final V differs"
    assert np.array_equal(gpu["I"].view(np.uint32), f.I_final.view(np.uint32)), "final I differs"


RTOL, ATOL = 1e-4, 1e-6


def assert_backward_close(gpu, orc, rtol=RTOL, atol=ATOL):
    """Every element of every dW and dD within atol + rtol |ref| of the
    oracle's fp64 definition (absolute atol, not scaled), and the same count
    of skipped degenerate jumps.  The oracle's fp32 evaluation of the same
    expressions, where computed, is printed beside it as the noise floor."""
    dW64, dD64, deg = orc["f64"]
    assert gpu["stats"]["degenerate_jumps"] == deg
    for p in range(len(dW64)):
        for nm, g, r, i in (("dW", gpu["dW"][p], dW64[p], 0), ("dD", gpu["dD"][p], dD64[p], 1)):
            g = np.asarray(g, np.float64)
            tol = atol + rtol * np.abs(r)
            err = np.abs(g - r)
            worst = float((err / tol).max()) if err.size else 0.0
            floor = ""
            if "f32" in orc:
                r32 = np.asarray(orc["f32"][i][p], np.float64)
                floor = f", fp32 evaluation {float((np.abs(r32 - r) / tol).max()):.3g}"
            print(f"[grad] {nm}[{p}] worst |gpu - fp64| / tol = {worst:.3g}{floor}", flush=True)
            bad = ~(err <= tol)
            assert not bad.any(), (f"{nm}[{p}]: {int(bad.sum())} of {bad.size} elements off the "
                                   f"fp64 definition, worst error / tolerance {worst:.3g}")
