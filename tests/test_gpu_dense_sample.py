"""A sample whose input and hidden spikes exceed what the LDS stages hold:
the grouping by presynaptic neuron sorts it in device memory, and the
gradient pass reads its spike steps from device memory (the other sample of
the batch takes the LDS paths).  Forward bit-exact, every dW and dD element within 1e-6 +
1e-4 |ref| of the oracle's fp64 definition."""
import dataclasses

import numpy as np
import pytest

from workloads import make_workload

from .gpu_util import assert_backward_close, assert_forward_bitexact, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


def _dense_pair(wl):
    """Sample 0: the union of samples 0, 1 and 2 (sorted by step, then
    channel, duplicates once); sample 1: sample 3 as drawn."""
    o = wl.in_off
    keys = []
    for s in range(3):
        keys.append(wl.in_step[o[s]:o[s + 1]].astype(np.int64) * 100000 + wl.in_neuron[o[s]:o[s + 1]])
    k = np.unique(np.concatenate(keys))
    st0, ne0 = (k // 100000).astype(wl.in_step.dtype), (k % 100000).astype(wl.in_neuron.dtype)
    st1, ne1 = wl.in_step[o[3]:o[4]], wl.in_neuron[o[3]:o[4]]
    off = np.array([0, len(st0), len(st0) + len(st1)], dtype=o.dtype)
    return dataclasses.replace(wl, B=2, in_off=off, in_step=np.concatenate([st0, st1]),
                               in_neuron=np.concatenate([ne0, ne1]), labels=wl.labels[:2])


def test_dense_sample_takes_the_device_memory_paths():
    wl = _dense_pair(make_workload(4, B=4))
    n0 = int(wl.in_off[1])
    print(f"[dense] cfg4 B=2: {n0} and {int(wl.in_off[2]) - n0} input spikes", flush=True)
    assert n0 > 16384                      # more than the grouping's LDS stage holds
    cap = 32768                            # (about 20k hidden spikes in sample 0)
    gpu = run_gpu(wl, cap=cap)
    assert gpu["rc"] == 0
    assert gpu["count"][0, 0] > 16384
    orc = run_oracle(wl, cap=cap, modes=("f64",))
    assert_forward_bitexact(gpu, orc, wl)
    assert np.allclose(gpu["loss"], orc["loss"], rtol=1e-6, atol=1e-7)
    assert_backward_close(gpu, orc)
