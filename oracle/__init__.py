"""CPU oracle for grid EventProp with learnable delays.

TEST INFRASTRUCTURE ONLY: the checker, not the product.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
it.  It shares no code with the HIP library (``paper_2501_07331_amd``), and the
library never imports it.

* ``snn_oracle.c`` (built into ``liboracle.so`` by ``oracle/build.py``): the
  plain single-threaded grid forward (fp32), CE loss (fp64) and backward
  (fp64 definition, or an fp32 evaluation of it as a noise floor); the
  spike-count regulariser's per-spike terms (``grid.spike_count_reg``).
* ``continuous.py``: an fp64 event-driven simulator of the continuous-time
  system of Table 1 for tiny networks, with the exact EventProp backward and
  a finite-difference check; it pins the grid oracle.
"""
from .grid import (OracleNet, constants, forward, loss, loss_dmse, first_spike_dlp, backward,
                   spike_count_reg, lib_path, ForwardResult, LOSS_DMSE)

__all__ = ["OracleNet", "constants", "forward", "loss", "loss_dmse", "first_spike_dlp", "backward",
           "spike_count_reg", "lib_path", "ForwardResult", "LOSS_DMSE"]
