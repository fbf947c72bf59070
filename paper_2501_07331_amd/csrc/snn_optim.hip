// Optimiser step over every weight and delay of the network (SGD or Adam),
// followed by the delay clamp.  One launch covers all projections; a lane
// owns one parameter, so the loads and stores of a wave are coalesced.
#include "snn_device.h"

namespace {

__global__ void __launch_bounds__(256) optimizer_kernel(OptArgs a) {
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= a.nparams) return;
    int p = 0;
    while (p + 1 < a.P && g >= a.woff[p + 1]) ++p;
    const long long k = g - a.woff[p];
    const float gw = a.dW[p][k], gd = a.dD[p][k];
    float w = a.W[p][k], d = a.D[p][k];
    if (a.kind == SNN_OPT_SGD) {
        w = __fsub_rn(w, __fmul_rn(a.lr_w[p], gw));
        d = __fsub_rn(d, __fmul_rn(a.lr_d[p], gd));
    } else {
        // moments: [m_w, v_w, m_d, v_d] blocks of nparams each
        float* mw = a.mom;
        float* vw = a.mom + a.nparams;
        float* md = a.mom + 2 * a.nparams;
        float* vd = a.mom + 3 * a.nparams;
        const float ob1 = a.one_m_b1, ob2 = a.one_m_b2;
        float m1 = __fadd_rn(__fmul_rn(a.b1, mw[g]), __fmul_rn(ob1, gw));
        float v1 = __fadd_rn(__fmul_rn(a.b2, vw[g]), __fmul_rn(ob2, __fmul_rn(gw, gw)));
        float m2 = __fadd_rn(__fmul_rn(a.b1, md[g]), __fmul_rn(ob1, gd));
        float v2 = __fadd_rn(__fmul_rn(a.b2, vd[g]), __fmul_rn(ob2, __fmul_rn(gd, gd)));
        mw[g] = m1;
        vw[g] = v1;
        md[g] = m2;
        vd[g] = v2;
        const float uw = __fdiv_rn(__fmul_rn(m1, a.c1), __fadd_rn(__fsqrt_rn(__fmul_rn(v1, a.c2)), a.eps));
        const float ud = __fdiv_rn(__fmul_rn(m2, a.c1), __fadd_rn(__fsqrt_rn(__fmul_rn(v2, a.c2)), a.eps));
        w = __fsub_rn(w, __fmul_rn(a.lr_w[p], uw));
        d = __fsub_rn(d, __fmul_rn(a.lr_d[p], ud));
    }
    // NaN delays stay NaN (the forward's rounding counts them and uses slot 0)
    d = (d < a.d_min) ? a.d_min : (d > a.d_max) ? a.d_max : d;
    a.W[p][k] = w;
    a.D[p][k] = d;
}

}  // namespace

hipError_t launch_optimizer(const OptArgs& a, hipStream_t s) {
    if (a.nparams <= 0) return hipSuccess;
    hipLaunchKernelGGL(optimizer_kernel, dim3(grid_for(a.nparams, 256)), dim3(256), 0, s, a);
    return hipGetLastError();
}
