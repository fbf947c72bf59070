// Forward core instantiations for workgroups of up to 256 threads.
#include "snn_fwd_core.h"

bool launch_forward_core_256(const CoreFwdArgs& a, int n_lif, int np, bool rl, int threads,
                             size_t lds, hipStream_t s) {
    return launch_ft<256>(a, n_lif, np, rl, threads, lds, s);
}

hipError_t set_core_lds_limits_256(size_t bytes, int* bad) {
    // kernels 0 .. 7: LDS rings; 8 .. 15: rings in HBM; 16 .. 31: the same
    // with the fused readout wave
    hipError_t e = set_lds_limits_t<256, true, false>(bytes, bad);
    int base = 0;
    if (e == hipSuccess) {
        base = 8;
        e = set_lds_limits_t<256, false, false>(bytes, bad);
    }
    if (e == hipSuccess) {
        base = 16;
        e = set_lds_limits_t<256, true, true>(bytes, bad);
    }
    if (e == hipSuccess) {
        base = 24;
        e = set_lds_limits_t<256, false, true>(bytes, bad);
    }
    if (e != hipSuccess && bad) *bad += base;
    return e;
}
