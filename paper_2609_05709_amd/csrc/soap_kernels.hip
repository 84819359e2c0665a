// Host side of the SOAP kernels: launch configuration and launches.  The
// device code is in soap_device.h.
#include "soap_device.h"

namespace soap {
using namespace dev;

size_t density_lds_bytes(const Params &P, int jac, int lg0, int lg1, int W, bool st64) {
    const size_t Lg = (size_t)(lg1 * lg1 - lg0 * lg0);
    const size_t SnL = (size_t)P.S * P.n * Lg;
    const int RBk = row_block(NWD * W);
    size_t d = table_doubles(P, lg1 - lg0) + even(SnL * (jac ? 4 : 1)) + even(4 * (size_t)RBk) + even((RBk + 1) / 2) +
               even((size_t)P.n) + NWD * dens_wave_doubles(P, jac, lg0, lg1, W, st64 ? 8 : 4);
    return d * 8;
}

// the density kernel of a precision (positions and outputs T, staging ST),
// mode, radial basis and occupancy variant
template <typename T, typename ST, int RBF, bool HI>
static const void *density_kernel_r(int mode) {
    return mode == 0 ? (const void *)dev::k_density<T, T, 0, RBF, false, ST>
                     : mode == 1 ? (const void *)dev::k_density<T, T, 1, RBF, HI && dev::dens_has_high(1, RBF), ST>
                                 : (const void *)dev::k_density<T, T, 2, RBF, HI, ST>;
}
template <typename T, typename ST, int RBF>
static const void *density_kernel_h(int mode, bool hi) {
    return hi ? density_kernel_r<T, ST, RBF, true>(mode) : density_kernel_r<T, ST, RBF, false>(mode);
}
template <typename T, typename ST>
static const void *density_kernel_t(int mode, int rbf, bool hi) {
    if (rbf == 3) { // the compensated GTO exists for float64 only
        if constexpr (sizeof(T) == 8) return density_kernel_h<T, ST, 3>(mode, hi);
        return nullptr;
    }
    return rbf == 0 ? density_kernel_h<T, ST, 0>(mode, hi)
                    : (rbf == 1 ? density_kernel_h<T, ST, 1>(mode, hi) : density_kernel_h<T, ST, 2>(mode, hi));
}
// ar64: float64 staging with float32 outputs (ignored for float64 outputs)
static const void *density_kernel(bool f64, bool ar64, int mode, int rbf, bool hi) {
    if (f64) return density_kernel_t<double, double>(mode, rbf, hi);
    return ar64 ? density_kernel_t<float, double>(mode, rbf, hi) : density_kernel_t<float, float>(mode, rbf, hi);
}

// k_desc variants: QT (lm, pair of radial indices) tasks per thread, NA >=
// n_max, SR >= S species slots (groups of 4 radial indices measured 27% slower
// at 10^6 atoms: two waves then do the projection while the other two wait)
constexpr int DESC_AG = 2;
template <typename T, typename ST, int SR>
static const void *desc_kernel_s(int qt, int na) {
    if (qt == 1 && na == 8) return (const void *)dev::k_desc<T, T, ST, 1, DESC_AG, 8, SR>;
    if (qt == 1 && na == 16) return (const void *)dev::k_desc<T, T, ST, 1, DESC_AG, 16, SR>;
    if (qt == 2 && na == 8) return (const void *)dev::k_desc<T, T, ST, 2, DESC_AG, 8, SR>;
    if (qt == 2 && na == 16) return (const void *)dev::k_desc<T, T, ST, 2, DESC_AG, 16, SR>;
    if (qt == 4 && na == 16) return (const void *)dev::k_desc<T, T, ST, 4, DESC_AG, 16, SR>;
    return nullptr;
}
template <typename T, typename ST>
static const void *desc_kernel_t(int qt, int na, int sr) {
    return sr == 2 ? desc_kernel_s<T, ST, 2>(qt, na) : (sr == 4 ? desc_kernel_s<T, ST, 4>(qt, na) : nullptr);
}
static const void *desc_kernel(bool f64, bool ar64, int qt, int na, int sr) {
    if (f64) return desc_kernel_t<double, double>(qt, na, sr);
    return ar64 ? desc_kernel_t<float, double>(qt, na, sr) : desc_kernel_t<float, float>(qt, na, sr);
}

// k_djac variants: QT (lm, pair) tasks per thread, NA >= n_max, SR >= S species slots
template <typename T, typename ST, int SR>
static const void *djac_kernel_s(int qt, int na) {
    if (qt == 1 && na == 8) return (const void *)dev::k_djac<T, T, ST, 1, 8, SR>;
    if (qt == 1 && na == 16) return (const void *)dev::k_djac<T, T, ST, 1, 16, SR>;
    if (qt == 2 && na == 8) return (const void *)dev::k_djac<T, T, ST, 2, 8, SR>;
    if (qt == 2 && na == 16) return (const void *)dev::k_djac<T, T, ST, 2, 16, SR>;
    return nullptr;
}
template <typename T, typename ST>
static const void *djac_kernel_t(int qt, int na, int sr) {
    return sr == 2 ? djac_kernel_s<T, ST, 2>(qt, na) : (sr == 4 ? djac_kernel_s<T, ST, 4>(qt, na) : nullptr);
}
static const void *djac_kernel(bool f64, bool ar64, int qt, int na, int sr) {
    if (f64) return djac_kernel_t<double, double>(qt, na, sr);
    return ar64 ? djac_kernel_t<float, double>(qt, na, sr) : djac_kernel_t<float, float>(qt, na, sr);
}

// k_radial variants: NA >= n_max radial indices per lane
template <typename T> static const void *radial_kernel_t(int na) {
    if (na == 4) return (const void *)dev::k_radial<T, 4>;
    if (na == 8) return (const void *)dev::k_radial<T, 8>;
    if (na == 12) return (const void *)dev::k_radial<T, 12>;
    if (na == 16) return (const void *)dev::k_radial<T, 16>;
    return nullptr;
}
static const void *radial_kernel(bool f64, int na) { return f64 ? radial_kernel_t<double>(na) : radial_kernel_t<float>(na); }
static int radial_na(int n) { return n <= 4 ? 4 : (n <= 8 ? 8 : (n <= 12 ? 12 : 16)); }

size_t radial_bytes_per_edge(const Params &P) { return 16 * (size_t)P.n * (P.lmax + 1); }

hipError_t launch_radial(const Params &P, const Rows &R, const void *pos, bool f64, int64_t e_base, void *out,
                         hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    const int na = radial_na(P.n);
    const void *k = radial_kernel(f64, na);
    const size_t lds = 8 * dev::radial_lds_doubles(P, na);
    int ncu = 256, dev_id = 0, per = 0;
    (void)hipGetDevice(&dev_id);
    (void)hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev_id);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, k, BSR, lds) != hipSuccess || per < 1) per = 1;
    // blocks of cb centers: about 16 workgroups per CU of work, at most
    // RAD_CB_MAX centers a block, the blocks striding over the centers
    int cb = (int)std::min<int64_t>(RAD_CB_MAX, std::max<int64_t>(1, R.nc / (16 * (int64_t)ncu)));
    const int64_t need = (R.nc + cb - 1) / cb;
    const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>(need, (int64_t)ncu * per * 64));
    Params Pk = P;
    Rows Rk = R;
    void *args[] = {&Pk, &Rk, &pos, &e_base, &cb, &out};
    return hipLaunchKernel(k, dim3(blocks), dim3(BSR), args, lds, st);
}

bool density_has_high(int mode, int rbf) { return dev::dens_has_high(mode, rbf); }

int density_blocks_per_cu(bool f64, bool ar64, int mode, int rbf, bool hi, size_t lds) {
    int nb = 0;
    const hipError_t e =
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, density_kernel(f64, ar64, mode, rbf, hi), BSD, lds);
    return (e == hipSuccess && nb > 0) ? nb : 1;
}

size_t jacobian_lds_bytes(const Params &P, int W, bool at64) {
    const int ab = at64 ? 8 : 4;
    const size_t L = (size_t)P.L, Sn = (size_t)P.S * P.n;
    const int RBk = row_block(NWJ * W);
    size_t d = table_doubles(P, P.lmax + 1) + even((Sn * L * ab + 7) / 8) + even(4 * (size_t)RBk) + even((RBk + 1) / 2) +
               even(((size_t)P.tri_lw + 1) / 2) + NWJ * jac_wave_doubles(P, W, ab);
    return d * 8;
}

// Fewest contiguous l-groups whose LDS (c and one component of D for the
// group, plus the group's part of an output row) stays within 80 KB, two
// workgroups per CU; a single l above the budget may use up to the hard limit.
int plan_outputs(const Params &P, bool f64, bool st64, bool allow_rows, OutPlan *O) {
    const int lw = P.lmax + 1, ob = f64 ? 8 : 4;
    const size_t hard = 159 * 1024;
    // whole rows (k_outputs_rows) where c, one component of D and a row fit
    const size_t rows_lds = 8 * outputs_rows_doubles(P, ob, st64 ? 8 : 4);
    O->st64 = st64;
    O->rows = allow_rows && rows_lds <= hard && (size_t)P.L * P.S * P.n <= (size_t)OUT_PF * BSO2;
    if (O->rows) {
        O->n_groups = 1;
        O->lgrp[0] = 0;
        O->lgrp[1] = lw;
        O->lds = rows_lds;
        return 0;
    }
    // l-groups of up to 52 KB (three workgroups per CU); a single l may use up to the hard limit
    const size_t budget = 52 * 1024;
    int G = 0, l = 0;
    size_t worst = 0;
    O->lgrp[0] = 0;
    while (l < lw) {
        int e = l + 1;
        if (8 * outputs_group_doubles(P, l, e, ob) > hard) return -1;
        while (e < lw && 8 * outputs_group_doubles(P, l, e + 1, ob) <= budget) ++e;
        worst = std::max(worst, 8 * outputs_group_doubles(P, l, e, ob));
        O->lgrp[++G] = e;
        l = e;
    }
    O->n_groups = G;
    O->lds = worst;
    return 0;
}

hipError_t launch_outputs(const Params &P, const OutPlan &O, int64_t nc, bool f64, const void *scratch, void *desc,
                          void *jself, hipStream_t st) {
    if (nc <= 0) return hipSuccess;
    if (O.rows) {
        if (f64)
            hipLaunchKernelGGL((k_outputs_rows<double, double>), dim3((unsigned)nc), dim3(BSO2), O.lds, st, P,
                               (const double *)scratch,
                               (double *)desc, (double *)jself);
        else if (O.st64)
            hipLaunchKernelGGL((k_outputs_rows<float, double>), dim3((unsigned)nc), dim3(BSO2), O.lds, st, P,
                               (const double *)scratch,
                               (float *)desc, (float *)jself);
        else
            hipLaunchKernelGGL((k_outputs_rows<float, float>), dim3((unsigned)nc), dim3(BSO2), O.lds, st, P,
                               (const float *)scratch,
                               (float *)desc, (float *)jself);
        return hipGetLastError();
    }
    dim3 grid((unsigned)nc), block(BSO);
    if (f64)
        hipLaunchKernelGGL((k_outputs<double, double>), grid, block, O.lds, st, P, O, (const double *)scratch,
                           (double *)desc, (double *)jself);
    else if (O.st64)
        hipLaunchKernelGGL((k_outputs<float, double>), grid, block, O.lds, st, P, O, (const double *)scratch,
                           (float *)desc, (float *)jself);
    else
        hipLaunchKernelGGL((k_outputs<float, float>), grid, block, O.lds, st, P, O, (const float *)scratch,
                           (float *)desc, (float *)jself);
    return hipGetLastError();
}

int jacobian_max_w() { return JAC_MAX_W; }

// The float32 Jacobian kernel is also compiled for fixed (n_max, l_max + 1)
// pairs (jacobian_fixed.hip); the generic kernel covers every other basis and
// float64.
const void *jacobian_kernel(bool f64, bool ar64, int rbf, int n, int lw) {
    if (f64)
        return rbf == 3 ? reinterpret_cast<const void *>(&k_jacobian<double, double, 0, 0, 3>)
                        : reinterpret_cast<const void *>(&k_jacobian<double, double, 0, 0>);
    if (rbf == 3) return nullptr; // float64 only
    if (ar64) return reinterpret_cast<const void *>(&k_jacobian<float, float, 0, 0, -1, double>);
    const void *k = jacobian_fixed_0(n, lw);
    if (!k) k = jacobian_fixed_1(n, lw);
    if (!k) k = jacobian_fixed_2(n, lw);
    return k ? k : reinterpret_cast<const void *>(&k_jacobian<float, float, 0, 0>);
}

int jacobian_blocks_per_cu(bool f64, bool ar64, int rbf, int n, int lw, size_t lds) {
    int nb = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, jacobian_kernel(f64, ar64, rbf, n, lw), BSJ, lds);
    return (e == hipSuccess && nb > 0) ? nb : 0;
}

hipError_t set_lds_limits() {
    const int lim = 159 * 1024; // the kernels' static LDS uses part of the 160 KB
    hipError_t e = hipSuccess;
#define SOAP_SET(K)                                                                                          \
    if (e == hipSuccess) e = hipFuncSetAttribute((const void *)(K), hipFuncAttributeMaxDynamicSharedMemorySize, lim);
    for (int f64 = 0; f64 < 2; ++f64)
        for (int ar64 = 0; ar64 < 2; ++ar64)
            for (int mode = 0; mode < 3; ++mode)
                for (int rbf = 0; rbf < (f64 ? 4 : 3); ++rbf)
                    for (int hi = 0; hi < 2; ++hi) SOAP_SET(density_kernel(f64 != 0, ar64 != 0, mode, rbf, hi != 0));
    for (int f64 = 0; f64 < 2; ++f64)
        for (int ar64 = 0; ar64 < 2; ++ar64)
            for (int qt : {1, 2, 4})
                for (int na : {8, 16})
                    for (int sr : {2, 4})
                        if (desc_kernel(f64 != 0, ar64 != 0, qt, na, sr))
                            SOAP_SET(desc_kernel(f64 != 0, ar64 != 0, qt, na, sr));
    for (int f64 = 0; f64 < 2; ++f64)
        for (int ar64 = 0; ar64 < 2; ++ar64)
            for (int qt : {1, 2})
                for (int na : {8, 16})
                    for (int sr : {2, 4}) SOAP_SET(djac_kernel(f64 != 0, ar64 != 0, qt, na, sr));
    for (int f64 = 0; f64 < 2; ++f64)
        for (int na : {4, 8, 12, 16}) SOAP_SET(radial_kernel(f64 != 0, na));
    SOAP_SET((k_outputs<float, float>));
    SOAP_SET((k_outputs<float, double>));
    SOAP_SET((k_outputs_rows<float, float>));
    SOAP_SET((k_outputs_rows<float, double>));
    SOAP_SET((k_outputs_rows<double, double>));
    SOAP_SET((k_outputs<double, double>));
    SOAP_SET(k_power_single<float>);
    SOAP_SET(k_power_single<double>);
    SOAP_SET((k_jacobian<float, float, 0, 0>));
    SOAP_SET((k_jacobian<double, double, 0, 0>));
    SOAP_SET((k_jacobian<double, double, 0, 0, 3>));
    SOAP_SET((k_jacobian<float, float, 0, 0, -1, double>));
    for (int n = 1; n <= NMAX; ++n)
        for (int lw = 1; lw <= LMAX + 1; ++lw) {
            const void *k = jacobian_kernel(false, false, 0, n, lw);
            if (k != reinterpret_cast<const void *>(&k_jacobian<float, float, 0, 0>)) SOAP_SET(k);
        }
#undef SOAP_SET
    if (e == hipSuccess) e = djs_set_lds_limit(lim);
    return e;
}

hipError_t launch_density(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, int mode,
                          const DensityLaunch &cfg, unsigned long long *work, WorkBase *epoch, void *desc, void *c_out,
                          void *jself, void *c_scratch, void *jc_edge, hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    const int64_t per_group = std::min<int64_t>(R.nc, (int64_t)cfg.blocks);
    WorkBase b = *epoch;
    Params Pk = P;
    Rows Rk = R;
    int W = cfg.W;
    void *args[] = {&Pk, &Rk, &pos, &W, &work, &b, &desc, &c_out, &jself, &c_scratch, &jc_edge};
    const void *k = density_kernel(f64, ar64, mode, P.rbf, cfg.hi);
    const hipError_t e =
        hipLaunchKernel(k, dim3((unsigned)(per_group * P.n_groups)), dim3(BSD), args, cfg.lds, st);
    // each group's counter is taken for every center but the per_group
    // static ones, plus one final, empty fetch per workgroup: n_c increments
    // for every group this launch runs, none for the others
    if (e == hipSuccess)
        for (int g = 0; g < P.n_groups; ++g) epoch->b[g] += (uint64_t)R.nc;
    return e;
}

bool desc_shape(const Params &P, int *qt, int *na, int *sr) {
    if (P.rbf != 0 || P.S > 4) return false;
    const int t = dev::desc_tasks(P, DESC_AG);
    *qt = t <= 1 ? 1 : (t <= 2 ? 2 : 4);
    *na = P.n <= 8 ? 8 : 16;
    *sr = P.S <= 2 ? 2 : 4;
    return t <= 4 && desc_kernel(false, false, *qt, *na, *sr) != nullptr;
}

size_t desc_lds_bytes(const Params &P, int W, bool st64) { return 8 * dev::desc_lds_doubles(P, W, st64 ? 8 : 4); }

int desc_blocks_per_cu(bool f64, bool ar64, int ql, int na, int sr, size_t lds) {
    int nb = 0;
    const hipError_t e =
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, desc_kernel(f64, ar64, ql, na, sr), BSC, lds);
    return (e == hipSuccess && nb > 0) ? nb : 0;
}

hipError_t launch_desc(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, const DescLaunch &cfg,
                       void *desc, void *c_out, hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    Params Pk = P;
    Rows Rk = R;
    int W = cfg.W;
    void *args[] = {&Pk, &Rk, &pos, &W, &desc, &c_out};
    // persistent: as many workgroups as stay resident, each striding over the centers
    const int64_t blocks = std::min<int64_t>(R.nc, (int64_t)cfg.blocks);
    return hipLaunchKernel(desc_kernel(f64, ar64, cfg.ql, cfg.na, cfg.sr), dim3((unsigned)blocks), dim3(BSC), args,
                           cfg.lds, st);
}

bool djac_shape(const Params &P, int *qt, int *na, int *sr) {
    if (P.rbf != 0 || P.S > 4) return false;
    const int t = (P.L * ((P.n + 1) / 2) + BSC - 1) / BSC;
    if (t > 2) return false;
    *qt = t <= 1 ? 1 : 2;
    *na = P.n <= 8 ? 8 : 16;
    *sr = P.S <= 2 ? 2 : 4;
    return djac_kernel(false, false, *qt, *na, *sr) != nullptr;
}

size_t djac_lds_bytes(const Params &P, int W, bool st64) { return 8 * dev::djac_lds_doubles(P, W, st64 ? 8 : 4); }

int djac_blocks_per_cu(bool f64, bool ar64, int qt, int na, int sr, size_t lds) {
    int nb = 0;
    const hipError_t e =
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, djac_kernel(f64, ar64, qt, na, sr), BSC, lds);
    return (e == hipSuccess && nb > 0) ? nb : 0;
}

hipError_t launch_djac(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, const DjacLaunch &cfg,
                       void *desc, void *jself, void *c_scratch, hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    Params Pk = P;
    Rows Rk = R;
    int W = cfg.W;
    void *args[] = {&Pk, &Rk, &pos, &W, &desc, &jself, &c_scratch};
    const int64_t blocks = std::min<int64_t>(R.nc, (int64_t)cfg.blocks);
    return hipLaunchKernel(djac_kernel(f64, ar64, cfg.qt, cfg.na, cfg.sr), dim3((unsigned)blocks), dim3(BSC), args,
                           cfg.lds, st);
}

hipError_t launch_jacobian(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, const JacLaunch &cfg,
                           const void *c_scratch, void *jedge, hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    Params Pk = P;
    Rows Rk = R;
    int W = cfg.W;
    // float64: 16-byte vector stores when every section of an edge block is
    // a whole number of vectors and the output is 16-byte aligned
    const int nnl = P.n * P.n * (P.lmax + 1);
    int vec = (f64 && nnl % 2 == 0 && P.tri_lw % 2 == 0 && ((uintptr_t)jedge & 15) == 0) ? 1 : 0;
    void *args[] = {&Pk, &Rk, &pos, &W, &vec, &c_scratch, &jedge};
    return hipLaunchKernel(jacobian_kernel(f64, ar64, P.rbf, P.n, P.lmax + 1), dim3((unsigned)R.nc), dim3(BSJ), args,
                           cfg.lds, st);
}

hipError_t launch_column_mean(const void *in, bool f64, int64_t rows, int64_t cols, double *part, void *out,
                              double *mean, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const int nchunk = (int)std::min<int64_t>(rows, AVG_CHUNKS);
    const int64_t chunk_rows = (rows + nchunk - 1) / nchunk;
    const unsigned cb = (unsigned)((cols + 255) / 256);
    if (f64) {
        hipLaunchKernelGGL(k_colsum_partial<double>, dim3(cb, (unsigned)nchunk), dim3(256), 0, st, (const double *)in,
                           rows, cols, chunk_rows, part);
        hipLaunchKernelGGL(k_colmean_finish<double>, dim3(cb), dim3(256), 0, st, part, nchunk, cols, rows,
                           (double *)out, mean);
    } else {
        hipLaunchKernelGGL(k_colsum_partial<float>, dim3(cb, (unsigned)nchunk), dim3(256), 0, st, (const float *)in,
                           rows, cols, chunk_rows, part);
        hipLaunchKernelGGL(k_colmean_finish<float>, dim3(cb), dim3(256), 0, st, part, nchunk, cols, rows,
                           (float *)out, mean);
    }
    return hipGetLastError();
}

hipError_t launch_power_single(const Params &P, bool f64, const double *c, void *out, hipStream_t st) {
    const size_t lds = 8 * (size_t)P.S * P.n * P.L;
    if (f64)
        hipLaunchKernelGGL(k_power_single<double>, dim3(1), dim3(256), lds, st, P, c, (double *)out);
    else
        hipLaunchKernelGGL(k_power_single<float>, dim3(1), dim3(256), lds, st, P, c, (float *)out);
    return hipGetLastError();
}

hipError_t launch_scatter_dense(const Params &P, const Rows &R, bool f64, const void *jedge, const void *jself,
                                const int32_t *fmap, const int32_t *atom_of, void *dense, hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    if (f64)
        hipLaunchKernelGGL(dev::k_scatter_dense<double>, dim3((unsigned)R.nc), dim3(256), 0, st, P, R,
                           (const double *)jedge, (const double *)jself, fmap, atom_of, (double *)dense);
    else
        hipLaunchKernelGGL(dev::k_scatter_dense<float>, dim3((unsigned)R.nc), dim3(256), 0, st, P, R,
                           (const float *)jedge, (const float *)jself, fmap, atom_of, (float *)dense);
    return hipGetLastError();
}

} // namespace soap
