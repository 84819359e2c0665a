// Host side of the streamed density kernel k_djs (soap_device.h): variants,
// on-chip plan and launch.  Its own translation unit, so that its variants
// compile beside the other kernels.
#include "soap_device.h"

namespace soap {
using namespace dev;

// variants: QT (radial pair, lm) tasks per thread; GTO with NA >= n_max
// exponentials per l, the polynomial quadrature from k_radial's factors
template <typename T, typename ST, int RBF, int NA>
static const void *djs_kernel_q(int qt) {
    switch (qt) {
    case 1: return (const void *)k_djs<T, ST, 1, NA, RBF>;
    case 2: return (const void *)k_djs<T, ST, 2, NA, RBF>;
    case 3: return (const void *)k_djs<T, ST, 3, NA, RBF>;
    case 4: return (const void *)k_djs<T, ST, 4, NA, RBF>;
    default: return nullptr;
    }
}
template <typename T, typename ST>
static const void *djs_kernel_t(int rbf, int qt, int na) {
    if (rbf == 1) return djs_kernel_q<T, ST, 1, 8>(qt);
    if (rbf == 0 && na == 8) return djs_kernel_q<T, ST, 0, 8>(qt);
    if (rbf == 0 && na == 16) return djs_kernel_q<T, ST, 0, 16>(qt);
    return nullptr;
}
static const void *djs_kernel(bool f64, bool ar64, int rbf, int qt, int na) {
    if (f64) return djs_kernel_t<double, double>(rbf, qt, na);
    return ar64 ? djs_kernel_t<float, double>(rbf, qt, na) : djs_kernel_t<float, float>(rbf, qt, na);
}

bool djs_shape(const Params &P, int *qt, int *na) {
    if (P.rbf != 0 && P.rbf != 1) return false;
    if (P.rbf == 0 && P.n > 16) return false;
    const int t = djs_tasks(P);
    if (t > 4) return false;
    *qt = t < 1 ? 1 : t;
    *na = P.n <= 8 ? 8 : 16;
    return djs_kernel(false, false, P.rbf, *qt, *na) != nullptr;
}

size_t djs_lds_bytes(const Params &P, int W, bool st64) { return 8 * djs_lds_doubles(P, W, st64 ? 8 : 4); }

int djs_blocks_per_cu(bool f64, bool ar64, int rbf, int qt, int na, size_t lds) {
    int nb = 0;
    const void *k = djs_kernel(f64, ar64, rbf, qt, na);
    if (!k) return 0;
    const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k, BSC, lds);
    return (e == hipSuccess && nb > 0) ? nb : 0;
}

// dynamic LDS above the default limit for every variant (set_lds_limits)
hipError_t djs_set_lds_limit(int lim) {
    hipError_t e = hipSuccess;
    for (int f64 = 0; f64 < 2; ++f64)
        for (int ar64 = 0; ar64 < 2; ++ar64)
            for (int rbf = 0; rbf < 2; ++rbf)
                for (int qt = 1; qt <= 4; ++qt)
                    for (int na : {8, 16}) {
                        const void *k = djs_kernel(f64 != 0, ar64 != 0, rbf, qt, na);
                        if (k && e == hipSuccess)
                            e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, lim);
                    }
    return e;
}

hipError_t launch_djs(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, const DjsLaunch &cfg,
                      void *c_scratch, hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    Params Pk = P;
    Rows Rk = R;
    int W = cfg.W;
    void *args[] = {&Pk, &Rk, &pos, &W, &c_scratch};
    // persistent: as many workgroups as stay resident, each striding over the centers
    const int64_t blocks = std::min<int64_t>(R.nc, (int64_t)cfg.blocks);
    return hipLaunchKernel(djs_kernel(f64, ar64, P.rbf, cfg.qt, cfg.na), dim3((unsigned)blocks), dim3(BSC), args,
                           cfg.lds, st);
}

} // namespace soap
