// Forward core instantiations for workgroups of up to 1024 threads.
#include "snn_fwd_core.h"

bool launch_forward_core_1024(const CoreFwdArgs& a, int n_lif, int np, bool rl, int threads,
                             size_t lds, hipStream_t s) {
    return launch_ft<1024>(a, n_lif, np, rl, threads, lds, s);
}

hipError_t set_core_lds_limits_1024(size_t bytes, int* bad) {
    hipError_t e = set_lds_limits_t<1024, true, false>(bytes, bad);
    if (e == hipSuccess) {
        e = set_lds_limits_t<1024, false, false>(bytes, bad);
        if (e != hipSuccess && bad) *bad += 8;   // kernels with rings in HBM: 8 .. 15
    }
    return e;
}
