// Forward core instantiations in cluster mode: workgroups of one neuron wave
// and one wave per LIF -> LIF ring, every ring in LDS, G workgroups per
// sample, one cooperative launch (the runtime refuses a grid that cannot be
// resident at once, so every wait of a cluster ends).
#include "snn_fwd_core.h"

namespace {

template <int NL, int NP>
const void* fcl_fn() {
    return (const void*)forward_core_kernel<64, NL, NP, true, false, true>;
}

const void* fcl_kernel(int n_lif, int np) {
    switch (n_lif * 4 + np) {
        case 4 + 1: return fcl_fn<1, 1>();
        case 8 + 1: return fcl_fn<2, 1>();
        case 8 + 2: return fcl_fn<2, 2>();
        case 12 + 1: return fcl_fn<3, 1>();
        case 12 + 2: return fcl_fn<3, 2>();
        case 16 + 1: return fcl_fn<4, 1>();
        case 16 + 2: return fcl_fn<4, 2>();
        default: return nullptr;
    }
}

}  // namespace

hipError_t launch_forward_core_cluster(const CoreFwdArgs& a, int n_lif, int np, int grid, int threads,
                                       size_t lds, hipStream_t s) {
    const void* f = fcl_kernel(n_lif, np);
    int rings = 0;
    for (int l = 0; l < n_lif; ++l) rings += a.ly[l].npost;
    if (!f || a.ro_C != 0 || a.cl.G < 1 || a.NW != a.cl.G || grid < a.cl.G || grid % a.cl.G ||
        threads != 64 * (1 + rings) || rings > n_lif * np)
        return hipErrorInvalidValue;
    CoreFwdArgs arg = a;
    void* args[] = {&arg};
    return hipLaunchCooperativeKernel(f, dim3(grid), dim3(threads), args, (unsigned)lds, s);
}

hipError_t forward_cluster_occupancy(int n_lif, int np, int threads, size_t lds, int* blocks_per_cu) {
    const void* f = fcl_kernel(n_lif, np);
    if (!f) return hipErrorInvalidValue;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, f, threads, lds);
}

hipError_t set_core_lds_limits_cl(size_t bytes, int* bad) {
    for (int k = 0; k < 7; ++k) {
        static const int cases[7][2] = {{1, 1}, {2, 1}, {2, 2}, {3, 1}, {3, 2}, {4, 1}, {4, 2}};
        const hipError_t e = hipFuncSetAttribute(fcl_kernel(cases[k][0], cases[k][1]),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
        if (e != hipSuccess) {
            if (bad) *bad = k;
            return e;
        }
    }
    return hipSuccess;
}
