"""ctypes marshalling for libsnn (names follow include/snn.h)."""
from __future__ import annotations

import ctypes as C
import os
from typing import List, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))

SNN_OK, SNN_EINVAL, SNN_ENOMEM, SNN_ESTATE, SNN_EOVERFLOW, SNN_EDEVICE = 0, -1, -2, -3, -4, -5
SNN_INPUT, SNN_LIF, SNN_LI = 0, 1, 2
SNN_LOSS_CE_SUM, SNN_LOSS_CE_MAX, SNN_LOSS_DMSE = 0, 1, 2
SNN_FLAG_HBM_RINGS = 1
SNN_FLAG_TIMING = 2
SNN_FLAG_SEPARATE_READOUT = 4
SNN_FLAG_CLUSTER = 8
SNN_NOALLOC_SCRATCH_BYTES = 32 << 20
SNN_OPT_SGD, SNN_OPT_ADAM = 0, 1
_NAMES = {0: "SNN_OK", -1: "SNN_EINVAL", -2: "SNN_ENOMEM", -3: "SNN_ESTATE", -4: "SNN_EOVERFLOW",
          -5: "SNN_EDEVICE"}


class SNNError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_NAMES.get(code, code)}: {msg}")
        self.code = code


class SNNOverflow(SNNError):
    pass


class snn_layer(C.Structure):
    _fields_ = [("n", C.c_int32), ("kind", C.c_int32), ("recurrent", C.c_int32)]


class snn_opts(C.Structure):
    _fields_ = [("batch", C.c_int32), ("T", C.c_int32), ("loss", C.c_int32),
                ("readout_scale", C.c_float), ("record_capacity", C.c_int32),
                ("flags", C.c_int32), ("hip_stream", C.c_void_p), ("dmse_delta", C.c_float),
                ("proj_max_delay", C.c_void_p), ("reg_target", C.c_float),
                ("reg_strength", C.c_void_p)]


class snn_spikes_in(C.Structure):
    _fields_ = [("offsets", C.c_void_p), ("step", C.c_void_p), ("neuron", C.c_void_p),
                ("nnz", C.c_int32)]


class snn_spikes_out(C.Structure):
    _fields_ = [("count", C.c_void_p), ("step", C.c_void_p), ("neuron", C.c_void_p)]


class snn_stats(C.Structure):
    _fields_ = [("input_spikes", C.c_int64), ("lif_spikes", C.c_int64), ("events", C.c_int64),
                ("clamped_delays", C.c_int64), ("degenerate_jumps", C.c_int64),
                ("overflow", C.c_int32), ("lds_rings", C.c_int32),
                ("kernel_ms", C.c_float * 8), ("reg_loss", C.c_double)]


class snn_optim(C.Structure):
    _fields_ = [("kind", C.c_int32), ("lr_w", C.c_float), ("lr_d", C.c_float),
                ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("d_min", C.c_float), ("d_max", C.c_float),
                ("lr_scale_w", C.c_void_p), ("lr_scale_d", C.c_void_p)]


# order of snn_stats.kernel_ms
KERNELS = ("input_scan", "forward_core", "readout_forward", "readout_adjoint", "backward_core",
           "group", "gradients")


_lib = None


def lib_path() -> str:
    return os.path.join(HERE, "libsnn.so")


def load_library():
    """Load libsnn.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    path = lib_path()
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2501_07331_amd.build` "
                          "(there is no CPU fallback)")
    lib = C.CDLL(path)
    P = C.c_void_p
    lib.snn_create.argtypes = [C.POINTER(snn_layer), C.c_int32, C.c_float, C.c_float, C.c_float,
                               C.c_float, C.c_int32, C.POINTER(snn_opts), C.POINTER(P)]
    lib.snn_num_projections.argtypes = [P, C.POINTER(C.c_int32)]
    lib.snn_projection_info.argtypes = [P, C.c_int32] + [C.POINTER(C.c_int32)] * 4
    lib.snn_forward.argtypes = [P, C.POINTER(snn_spikes_in), C.POINTER(P), C.POINTER(P), P,
                                C.POINTER(snn_spikes_out), P, P]
    lib.snn_backward.argtypes = [P, C.POINTER(P), C.POINTER(P)]
    lib.snn_backward_lp.argtypes = [P, C.POINTER(P), C.POINTER(P), C.POINTER(P)]
    lib.snn_backward_noalloc.argtypes = [P, C.POINTER(P), C.POINTER(P)]
    lib.snn_optimizer_step.argtypes = [P, C.POINTER(snn_optim), C.POINTER(P), C.POINTER(P),
                                       C.POINTER(P), C.POINTER(P)]
    lib.snn_optimizer_reset.argtypes = [P]
    lib.snn_get_state.argtypes = [P, C.c_int32, P, P]
    lib.snn_get_record_currents.argtypes = [P, C.c_int32, P]
    lib.snn_get_stats.argtypes = [P, C.POINTER(snn_stats)]
    lib.snn_last_error.argtypes = [P]
    lib.snn_last_error.restype = C.c_char_p
    lib.snn_destroy.argtypes = [P]
    lib.snn_destroy.restype = None
    for f in ("snn_create", "snn_num_projections", "snn_projection_info", "snn_forward",
              "snn_backward", "snn_backward_lp", "snn_backward_noalloc", "snn_optimizer_step", "snn_optimizer_reset", "snn_get_state",
              "snn_get_record_currents", "snn_get_stats"):
        getattr(lib, f).restype = C.c_int
    _lib = lib
    return lib


def _ptr(t, dtype=None, what="tensor"):
    import torch
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    return C.c_void_p(t.data_ptr())


def _ptr_array(ts, dtype, what):
    arr = (C.c_void_p * len(ts))()
    for i, t in enumerate(ts):
        arr[i] = _ptr(t, dtype, f"{what}[{i}]")
    return arr


class Network:
    """One snn_net handle: a topology, constants and scratch for `batch`
    samples of `T` steps, bound to the current torch stream at creation."""

    def __init__(self, layers: Sequence[Tuple[int, int, int]], tau_m: float, tau_s: float,
                 theta: float, dt: float, max_delay: int, batch: int, T: int, loss: int,
                 readout_scale: float, record_capacity: int, flags: int = 0, stream=None,
                 dmse_delta: float = 0.0, proj_max_delay: Optional[Sequence[int]] = None,
                 reg_strength: Optional[Sequence[float]] = None, reg_target: float = 14.0):
        import torch
        self._lib = load_library()
        self.layers = [tuple(int(x) for x in l) for l in layers]
        self.batch, self.T = int(batch), int(T)
        self.record_capacity = int(record_capacity)
        self.max_delay = int(max_delay)
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        arr = (snn_layer * len(layers))(*[snn_layer(*l) for l in self.layers])
        self.proj_max_delay = None if proj_max_delay is None else [int(x) for x in proj_max_delay]
        pmd = (C.c_int32 * len(self.proj_max_delay))(*self.proj_max_delay) \
            if self.proj_max_delay is not None else None
        self.reg_strength = None if reg_strength is None else [float(x) for x in reg_strength]
        n_lif = sum(1 for l in self.layers if l[1] == SNN_LIF)
        if self.reg_strength is not None and len(self.reg_strength) != n_lif:
            raise ValueError(f"reg_strength needs one value per LIF layer ({n_lif})")
        rs = (C.c_float * len(self.reg_strength))(*self.reg_strength) \
            if self.reg_strength is not None else None
        opts = snn_opts(self.batch, self.T, int(loss), float(readout_scale), self.record_capacity,
                        int(flags), C.c_void_p(stream.cuda_stream), float(dmse_delta),
                        C.cast(pmd, C.c_void_p) if pmd is not None else None, float(reg_target),
                        C.cast(rs, C.c_void_p) if rs is not None else None)
        h = C.c_void_p()
        rc = self._lib.snn_create(arr, len(layers), tau_m, tau_s, theta, dt, int(max_delay),
                                  C.byref(opts), C.byref(h))
        if rc != SNN_OK:
            why = self._lib.snn_last_error(None).decode()
            raise SNNError(rc, "snn_create failed" + (f" ({why})" if why else ""))
        self._h = h
        n = C.c_int32()
        self._check(self._lib.snn_num_projections(h, C.byref(n)))
        self.projections = []
        for p in range(n.value):
            v = [C.c_int32() for _ in range(4)]
            self._check(self._lib.snn_projection_info(h, p, *[C.byref(x) for x in v]))
            self.projections.append(tuple(x.value for x in v))   # (pre, post, n_pre, n_post)

    def _check(self, rc):
        if rc == SNN_OK:
            return rc
        msg = self._lib.snn_last_error(self._h).decode() if getattr(self, "_h", None) else ""
        if rc == SNN_EOVERFLOW:
            raise SNNOverflow(rc, msg)
        raise SNNError(rc, msg)

    @property
    def lif_layers(self) -> List[int]:
        return [l for l, y in enumerate(self.layers) if y[1] == SNN_LIF]

    def forward(self, offsets, step, neuron, W, D, labels, records, loss, z=None):
        """records: one (count [B], step [B][cap], neuron [B][cap]) int32 triple
        per LIF layer; loss: fp32 [B+1]; z: fp32 [B][C] or None."""
        import torch
        i32, f32 = torch.int32, torch.float32
        inp = snn_spikes_in(_ptr(offsets, i32, "offsets"), _ptr(step, i32, "step"),
                            _ptr(neuron, i32, "neuron"), int(step.numel()))
        if offsets.numel() != self.batch + 1 or neuron.numel() != step.numel():
            raise ValueError("offsets must hold batch+1 entries and step/neuron the same count")
        if len(W) != len(self.projections) or len(D) != len(self.projections):
            raise ValueError("one W and one D tensor per projection")
        for p, (_, _, npre, npost) in enumerate(self.projections):
            for t_, nm in ((W[p], "W"), (D[p], "D")):
                if t_.numel() != npre * npost:
                    raise ValueError(f"{nm}[{p}] must hold {npre}x{npost} elements")
        if labels.numel() != self.batch or loss.numel() != self.batch + 1:
            raise ValueError("labels [B] and loss [B+1]")
        C_ = self.layers[-1][0]
        if z is not None and z.numel() != self.batch * C_:
            raise ValueError("z must hold B x C elements")
        if len(records) != len(self.lif_layers):
            raise ValueError("one record triple per LIF layer")
        recs = (snn_spikes_out * max(len(records), 1))()
        for i, (cnt, st, ne) in enumerate(records):
            if cnt.numel() != self.batch or st.numel() != self.batch * self.record_capacity \
                    or ne.numel() != self.batch * self.record_capacity:
                raise ValueError("record buffers must be [B] and [B][record_capacity]")
            recs[i] = snn_spikes_out(_ptr(cnt, i32, "count"), _ptr(st, i32, "rec step"),
                                     _ptr(ne, i32, "rec neuron"))
        self._keep = (offsets, step, neuron, list(W), list(D), labels)
        rc = self._lib.snn_forward(self._h, C.byref(inp), _ptr_array(W, f32, "W"),
                                   _ptr_array(D, f32, "D"), _ptr(labels, i32, "labels"), recs,
                                   _ptr(loss, f32, "loss"), _ptr(z, f32, "z") if z is not None else None)
        return self._check(rc)

    def backward(self, dW, dD, dlp=None):
        """dlp: None, or one entry per LIF layer: None or an fp32 [B][cap]
        device tensor of dl_p/dt_k per record (snn_backward_lp)."""
        import torch
        f32 = torch.float32
        for p, (_, _, npre, npost) in enumerate(self.projections):
            if dW[p].numel() != npre * npost or dD[p].numel() != npre * npost:
                raise ValueError(f"dW/dD[{p}] must hold {npre}x{npost} elements")
        if dlp is None:
            rc = self._lib.snn_backward(self._h, _ptr_array(dW, f32, "dW"), _ptr_array(dD, f32, "dD"))
            return self._check(rc)
        if len(dlp) != len(self.lif_layers):
            raise ValueError("one dlp entry (or None) per LIF layer")
        arr = (C.c_void_p * max(len(dlp), 1))()
        for i, x in enumerate(dlp):
            if x is not None and x.numel() != self.batch * self.record_capacity:
                raise ValueError("dlp entries must be [B][record_capacity]")
            arr[i] = _ptr(x, f32, f"dlp[{i}]") if x is not None else None
        rc = self._lib.snn_backward_lp(self._h, arr, _ptr_array(dW, f32, "dW"),
                                       _ptr_array(dD, f32, "dD"))
        return self._check(rc)

    def backward_noalloc(self, dW, dD):
        """snn_backward_noalloc: the backward pass with its input-sized scratch
        in the library's fixed per-device array (no device allocation)."""
        import torch
        f32 = torch.float32
        for p, (_, _, npre, npost) in enumerate(self.projections):
            if dW[p].numel() != npre * npost or dD[p].numel() != npre * npost:
                raise ValueError(f"dW/dD[{p}] must hold {npre}x{npost} elements")
        rc = self._lib.snn_backward_noalloc(self._h, _ptr_array(dW, f32, "dW"),
                                            _ptr_array(dD, f32, "dD"))
        return self._check(rc)

    def optimizer_step(self, W, D, dW, dD, kind: int = SNN_OPT_ADAM, lr_w: float = 1e-3,
                       lr_d: float = 0.1, beta1: float = 0.9, beta2: float = 0.999,
                       eps: float = 1e-8, d_min: float = 0.0, d_max: Optional[float] = None,
                       lr_scale_w: Optional[Sequence[float]] = None,
                       lr_scale_d: Optional[Sequence[float]] = None):
        """One SGD or Adam step on W and D in place, then D clamped to
        [d_min, d_max] (default d_max: the handle's max_delay)."""
        import torch
        f32 = torch.float32
        P_ = len(self.projections)
        for nm, ts in (("W", W), ("D", D), ("dW", dW), ("dD", dD)):
            if len(ts) != P_:
                raise ValueError(f"one {nm} tensor per projection")
        for p, (_, _, npre, npost) in enumerate(self.projections):
            for t_ in (W[p], D[p], dW[p], dD[p]):
                if t_.numel() != npre * npost:
                    raise ValueError(f"parameters of projection {p} must hold {npre}x{npost} elements")
        sw = (C.c_float * P_)(*lr_scale_w) if lr_scale_w is not None else None
        sd = (C.c_float * P_)(*lr_scale_d) if lr_scale_d is not None else None
        o = snn_optim(int(kind), float(lr_w), float(lr_d), float(beta1), float(beta2), float(eps),
                      float(d_min), float(self.max_delay if d_max is None else d_max),
                      C.cast(sw, C.c_void_p) if sw is not None else None,
                      C.cast(sd, C.c_void_p) if sd is not None else None)
        rc = self._lib.snn_optimizer_step(self._h, C.byref(o), _ptr_array(W, f32, "W"),
                                          _ptr_array(D, f32, "D"), _ptr_array(dW, f32, "dW"),
                                          _ptr_array(dD, f32, "dD"))
        return self._check(rc)

    def optimizer_reset(self):
        return self._check(self._lib.snn_optimizer_reset(self._h))

    def state(self, layer: int, V, I):
        import torch
        rc = self._lib.snn_get_state(self._h, int(layer), _ptr(V, torch.float32, "V"),
                                     _ptr(I, torch.float32, "I"))
        return self._check(rc)

    def record_currents(self, layer: int, I):
        """I- of every stored record of LIF layer `layer`: fp32 [B][cap] device tensor."""
        import torch
        if I.numel() != self.batch * self.record_capacity:
            raise ValueError("I must hold B x record_capacity elements")
        rc = self._lib.snn_get_record_currents(self._h, int(layer), _ptr(I, torch.float32, "I"))
        return self._check(rc)

    def stats(self) -> dict:
        s = snn_stats()
        self._check(self._lib.snn_get_stats(self._h, C.byref(s)))
        out = {f: getattr(s, f) for f, _ in snn_stats._fields_ if f != "kernel_ms"}
        out["kernel_ms"] = {k: float(s.kernel_ms[i]) for i, k in enumerate(KERNELS)}
        return out

    def close(self):
        if getattr(self, "_h", None):
            self._lib.snn_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
