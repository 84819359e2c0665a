// C ABI of the SOAP library (declared in include/soap.h).
#include "../../include/soap.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "basis.h"
#include "soap_internal.h"

using namespace soap;

namespace {

// grow-only device buffer
struct DevBuf {
    void *p = nullptr;
    size_t cap = 0;
    hipError_t ensure(size_t bytes) {
        if (bytes <= cap && p) return hipSuccess;
        if (p) {
            hipError_t e = hipFree(p);
            p = nullptr;
            cap = 0;
            if (e != hipSuccess) return e;
        }
        size_t b = bytes < 256 ? 256 : bytes;
        hipError_t e = hipMalloc(&p, b);
        if (e == hipSuccess) cap = b;
        return e;
    }
    void release() {
        if (p) (void)hipFree(p);
        p = nullptr;
        cap = 0;
    }
    template <typename T> T *as() const { return static_cast<T *>(p); }
};

constexpr size_t LDS_HARD_LIMIT = 159 * 1024; // leaves room for static LDS

thread_local std::string g_create_error = "";

// Coefficient scratch of soap_derivatives_batch_noalloc: a fixed device array
// that every device the library runs on holds until the process ends.  Host
// code never uses the array's name as an address (on the host it is only a
// stand-in for the symbol): soap_create resolves each device's own address
// once, with that device current, and the entry point passes that address
// to the kernels.
static __device__ __align__(256) unsigned char scratch[SOAP_STATIC_SCRATCH_BYTES];
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[MAX_DEVICES] = {};
hipError_t g_scratch_err[MAX_DEVICES] = {};
bool g_scratch_done[MAX_DEVICES] = {};

// the static scratch of `device` (the current device), resolved on first use
hipError_t static_scratch(int device, void **out) {
    *out = nullptr;
    if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_done[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch_err[device] = e;
        g_scratch_ptr[device] = e == hipSuccess ? p : nullptr;
        g_scratch_done[device] = true;
    }
    *out = g_scratch_ptr[device];
    return g_scratch_err[device];
}

} // namespace

struct soap_ctx {
    int device = 0;
    std::vector<int32_t> Z; // sorted
    double r_cut = 0, sigma = 0;
    int n = 0, lmax = 0, rbf = 0, Q = 64, dtype = SOAP_FP32, arith = SOAP_ARITH_MIXED;
    int64_t F = 0, Fe = 0;
    int nq_full = 0;
    std::vector<uint32_t> fq;
    std::vector<uint32_t> dtab;   // [tri lw] diagonal-pair slots of the Jacobian kernel
    std::vector<int32_t> fmap;    // [S][Fe]
    Params P{};
    // device constants
    DevBuf d_const, d_dtab, d_fmap, d_lut;
    // neighbour workspace
    NbrWork nw{};
    DevBuf b_zero, b_bstart, b_acell, b_srec, b_sspec, b_deg, b_slots, b_scan, b_spec, b_row, b_cols, b_cscratch;
    DevBuf b_avg, b_avg_part; // averaged modes: per-center rows, column partial sums and means
    DevBuf b_radial;          // polynomial quadrature: radial factors of a call's edges
    std::vector<int64_t> h_row; // polynomial quadrature: host copy of the CSR row offsets
    // periodic cell (soap_set_cell) and the extended structure of the last build
    bool periodic = false, built_periodic = false;
    PeriodicCell cell{};
    int64_t n_ext = 0;
    DevBuf b_img_lohi, b_img_cnt, b_img_start, b_pos_ext, b_Z_ext, b_map_atom, b_map_img, b_iota;
    WorkBase work_epoch{}; // per l-group: density work-counter increments since the counters were zeroed
    int32_t *h_flags = nullptr; // pinned: [0..3] flags, int64 E at byte 16, int64 image count at byte 32
    // pinned coherent record that the neighbour search's degree scan writes
    // (error bits | largest degree << 32, rows above TCAP, E, sequence number)
    int64_t *h_rec = nullptr, *d_rec = nullptr;
    int64_t rec_seq = 0;
    int64_t *h_rowp = nullptr; // pinned staging of the row offsets (polynomial quadrature)
    size_t h_rowp_cap = 0;     // entries
    // state of the last neighbour build
    bool have_rows = false;
    int64_t n_atoms = 0, nc = 0, E = 0;
    const void *pos = nullptr;
    const int32_t *Zdev = nullptr, *centers = nullptr;
    bool built_f64 = false;
    bool ar64 = false; // float64 staging and assembly with float32 outputs (option "arith")
    // launch configuration
    DensityLaunch dens_cfg[3]{};  // [density kernel mode: descriptor, Jacobian, coefficient Jacobian]
    // whether each kernel's on-chip plan fits this basis: a basis too large for
    // one path still serves the others (the descriptor path is required)
    bool dens_ok[3] = {false, false, false}, out_ok = false, jac_ok = false;
    JacLaunch jac_cfg{};
    DescLaunch desc_cfg{};
    DjacLaunch djac_cfg{};
    int djac_tile = 0; // option "djac_tile": 0 auto (default), -1 never k_djac, else the widest chunk
    DjsLaunch djs_cfg{};
    int djs_tile = 0; // option "djs_tile": 0 auto (default), -1 never k_djs, else the widest chunk
    // pipelined derivatives: the density kernel of center chunk k + 1 on the
    // caller's stream beside the Jacobian kernel of chunk k on a second one
    int pipe_chunks = 1;         // option "pipeline": chunks per call (1 = one stream)
    int64_t batch_centers = 0;   // option "batch_centers": soap_derivatives in center batches of at most
                                 // this many (0 = one batch), the scratch sized for one batch
    int pipe_density_wg = 0;     // option "pipeline_density_wg": density workgroups per CU (0 = as planned)
    hipStream_t aux = nullptr;   // the second stream (default priority)
    std::vector<hipEvent_t> pipe_ev;
    int desc_tile = 0; // option "desc_tile": 0 auto, -1 never k_desc, else edges per chunk
    int jac_tile = 0;  // option "jac_tile": 0 auto, else edges per matrix-core tile of k_jacobian
    OutPlan out_plan{};
    bool out_rows = true; // option "out_rows": whole-row output kernel where it fits
    int groups[3] = {1, 1, 1};
    int lgrp[3][MAX_GROUPS + 1]{};
    // per-segment timing
    bool timing = false;
    struct Rec {
        int seg;
        hipEvent_t a, b;
    };
    std::vector<Rec> recs;
    std::vector<hipEvent_t> pool;
    void *static_scratch = nullptr; // this device's static scratch (soap_derivatives_batch_noalloc)
    std::string err;
};

namespace {

int fail(soap_ctx *c, int code, const char *fmt, ...) {
    if (c) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        c->err = buf;
    }
    return code;
}

int hip_fail(soap_ctx *c, hipError_t e, const char *where) {
    return fail(c, e == hipErrorOutOfMemory ? SOAP_ENOMEM : SOAP_EHIP, "%s: %s", where, hipGetErrorString(e));
}

// feature tables: full (mu,nu,n,n') combinations and the per-species edge terms
void build_feature_tables(soap_ctx *c) {
    const int S = (int)c->Z.size(), n = c->n, lw = c->lmax + 1;
    c->fq.clear();
    for (int mu = 0; mu < S; ++mu)
        for (int nu = mu; nu < S; ++nu)
            for (int a = 0; a < n; ++a)
                for (int b = (mu == nu ? a : 0); b < n; ++b)
                    c->fq.push_back((uint32_t)mu | (uint32_t)nu << 8 | (uint32_t)a << 16 | (uint32_t)b << 24);
    c->nq_full = (int)c->fq.size();
    c->F = (int64_t)c->nq_full * lw;
    c->Fe = (int64_t)lw * (n * (n + 1) / 2 + (S - 1) * n * n);
    c->fmap.assign((size_t)S * c->Fe, 0);
    // fmap[s][k]: feature index of slot k of a species-s neighbour block
    for (int s = 0; s < S; ++s) {
        int64_t k = 0;
        for (int q = 0; q < c->nq_full; ++q) {
            const uint32_t f = c->fq[q];
            const int mu = f & 0xff, nu = (f >> 8) & 0xff;
            if (mu != s && nu != s) continue;
            for (int l = 0; l < lw; ++l, ++k) c->fmap[(size_t)s * c->Fe + k] = q * lw + l;
        }
    }
    // diagonal-pair slots in feature order: (n, n' >= n, l) -> (n lw + l) | (n' lw + l) << 16
    c->dtab.clear();
    for (int a = 0; a < n; ++a)
        for (int b = a; b < n; ++b)
            for (int l = 0; l < lw; ++l) c->dtab.push_back((uint32_t)(a * lw + l) | (uint32_t)(b * lw + l) << 16);
}

// Split l = 0..lmax into contiguous groups such that each group's
// coefficient entries fit the density kernel's registers (n * Lg <= 512) and
// its LDS fits the budget (the LDS share of a workgroup at the occupancy the
// kernel's registers allow); W = edges per wave iteration, the widest that
// fits.
int plan_groups(const Params &P, int jac, bool st64, size_t budget, int *lgrp, int *ngroups, int *W_out,
                size_t *lds_out) {
    const int lw = P.lmax + 1;
    for (int G = 1; G <= lw; ++G) {
        // contiguous groups balancing sum over l of (2l+1): cut k at the l with
        // l^2 closest above k L / G, kept strictly increasing and leaving one l
        // for every later group
        int bounds[MAX_GROUPS + 1];
        bounds[0] = 0;
        for (int k = 1; k < G; ++k) {
            int b = (int)std::ceil(std::sqrt((double)k * lw * lw / G) - 1e-9);
            b = std::max(b, bounds[k - 1] + 1);
            b = std::min(b, lw - (G - k));
            bounds[k] = b;
        }
        bounds[G] = lw;
        bool ok = true;
        for (int k = 0; k < G; ++k)
            if (P.n * (bounds[k + 1] * bounds[k + 1] - bounds[k] * bounds[k]) > 64 * DENSITY_KE) ok = false;
        if (!ok) continue;
        for (int W : {8, 4, 2, 1}) {
            size_t worst = 0;
            for (int k = 0; k < G; ++k)
                worst = std::max(worst, density_lds_bytes(P, jac, bounds[k], bounds[k + 1], W, st64));
            if (worst <= budget || (W == 1 && worst <= LDS_HARD_LIMIT)) {
                for (int k = 0; k <= G; ++k) lgrp[k] = bounds[k];
                *ngroups = G;
                *W_out = W;
                *lds_out = worst;
                return 0;
            }
        }
    }
    return -1;
}

// The radial basis the kernels evaluate: the user's, except that GTO in
// float64 from n_max = 10 on takes the compensated evaluation (Params.rbf 3):
// the Loewdin coefficients amplify the rounding of sum_k beta e^{-a' r^2} by
// a factor growing from ~1e5 at n_max 10 to ~5e8 at 16.
constexpr int GTO_COMPENSATED_MIN_N = 10;
int kernel_basis(const soap_ctx *c) {
    if (c->rbf == SOAP_RBF_GTO && c->dtype == SOAP_FP64 && c->n >= GTO_COMPENSATED_MIN_N) return 3;
    return c->rbf;
}

int plan_launches(soap_ctx *c) {
    Params &P = c->P;
    P.rbf = kernel_basis(c);
    int Wd;
    size_t lds;
    int ncu = 256;
    (void)hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, c->device);
    const bool f64d = c->dtype == SOAP_FP64;
    c->ar64 = !f64d && c->arith == SOAP_ARITH_FP64;
    const bool ar64 = c->ar64, st64 = f64d || ar64;
    for (int mode = 0; mode < 3; ++mode) {
        const int jac = mode != 0; // modes 1 and 2 stage gradients
        int *lgrp = c->lgrp[mode], *G = &c->groups[mode];
        // workgroups per CU the registers allow (no LDS), and the LDS share of each
        auto plan = [&](bool hi, int *lg, int *g, int *w, size_t *ld) {
            const int by_regs = std::max(1, density_blocks_per_cu(f64d, ar64, mode, P.rbf, hi, 0));
            const size_t budget = std::min(LDS_HARD_LIMIT, (size_t)(159 * 1024) / (size_t)by_regs);
            return plan_groups(P, jac, st64, budget, lg, g, w, ld) == 0;
        };
        c->dens_ok[mode] = plan(false, lgrp, G, &Wd, &lds);
        if (!c->dens_ok[mode]) {
            if (mode == 0) return fail(c, SOAP_EINVAL, "basis too large for the density kernel's on-chip memory");
            continue;
        }
        bool hi = false;
        if (density_has_high(mode, P.rbf)) {
            // more workgroups per CU hide more latency, but split the LDS
            // further.  The Jacobian path takes three waves per SIMD only if
            // the plan keeps its l-groups and at least two edges per tile
            // (measured: 3% faster at n_max 8, l_max 6; up to twice as slow
            // where the tiles shrink).  "cc" takes two waves whenever they
            // plan (faster in 3 of 4 measured bases, by 13-29%; 13% slower at
            // n_max 12, l_max 12, where no simple rule on the plan told apart)
            int lg3[MAX_GROUPS + 1], G3 = 0, W3 = 0;
            size_t lds3 = 0;
            if (plan(true, lg3, &G3, &W3, &lds3) && (mode == 2 || (G3 == *G && W3 >= 2))) {
                hi = true;
                std::copy(lg3, lg3 + G3 + 1, lgrp);
                Wd = W3;
                lds = lds3;
            }
        }
        c->dens_cfg[mode].W = Wd;
        c->dens_cfg[mode].lds = lds;
        c->dens_cfg[mode].hi = hi;
        const int per_cu = density_blocks_per_cu(f64d, ar64, mode, P.rbf, hi, lds);
        c->dens_cfg[mode].blocks = std::max(1, ncu * per_cu / *G);
    }
    c->out_ok = plan_outputs(P, c->dtype == SOAP_FP64, st64, c->out_rows, &c->out_plan) == 0;
    // Jacobian kernel: W edges per wave tile.  The most resident waves per CU
    // first (latency hiding for its LDS-bound staging), then the widest tile;
    // a one-edge tile fills a quarter of the matrix-core rows, so at two or
    // more workgroups per CU a wider tile counts double (measured: two
    // workgroups of two-edge tiles beat three of one-edge tiles, GTO n4 l12
    // 0.76 against 1.05 ms per Jacobian launch; one workgroup of two-edge
    // tiles loses to two of one-edge tiles, CHNO 0.91 against 0.81 ms)
    const bool f64 = c->dtype == SOAP_FP64;
    int bestW = 0, bestB = 0;
    for (int W = jacobian_max_w(); W >= 1; --W) {
        if (c->jac_tile > 0 && W != c->jac_tile) continue;
        const size_t lds = jacobian_lds_bytes(P, W, st64);
        if (lds > LDS_HARD_LIMIT) continue;
        int b = jacobian_blocks_per_cu(f64, ar64, P.rbf, P.n, P.lmax + 1, lds);
        if (W >= 2 && b >= 2) b *= 2;
        if (b > bestB) {
            bestB = b;
            bestW = W;
        }
    }
    // descriptor kernel: the widest chunk of edges that keeps at least two
    // workgroups (of four waves) resident per CU; an explicit "desc_tile" is
    // the widest chunk tried, and any chunk that fits at all is taken
    c->desc_cfg = DescLaunch{};
    int ql = 0, na = 0, dsr = 0;
    if (c->desc_tile >= 0 && desc_shape(P, &ql, &na, &dsr)) {
        const int cand[3] = {64, 32, 16};
        for (int W : cand) {
            if (c->desc_tile > 0 && W > c->desc_tile) continue;
            const size_t lds = desc_lds_bytes(P, W, st64);
            if (lds > LDS_HARD_LIMIT) continue;
            const int b = desc_blocks_per_cu(f64, ar64, ql, na, dsr, lds);
            if (b >= (c->desc_tile > 0 ? 1 : 2)) {
                c->desc_cfg = DescLaunch{W, ql, na, dsr, lds, ncu * b};
                break;
            }
        }
    }
    // density step of the Jacobian path (GTO): the widest chunk of edges that
    // keeps at least two workgroups resident per CU
    c->djac_cfg = DjacLaunch{};
    int qt = 0, na2 = 0, sr = 0;
    if (c->djac_tile >= 0 && djac_shape(P, &qt, &na2, &sr)) {
        for (int W : {64, 32}) {
            if (c->djac_tile > 0 && W > c->djac_tile) continue;
            const size_t lds = djac_lds_bytes(P, W, st64);
            if (lds > LDS_HARD_LIMIT) continue;
            const int b = djac_blocks_per_cu(f64, ar64, qt, na2, sr, lds);
            if (b >= (c->djac_tile > 0 ? 1 : 2)) {
                c->djac_cfg = DjacLaunch{W, qt, na2, sr, lds, ncu * b};
                break;
            }
        }
    }
    // density step of the Jacobian path for the other GTO and polynomial
    // quadrature bases: coefficients streamed to the scratch, outputs by the
    // output kernel.  The widest chunk of edges that keeps at least two
    // workgroups resident per CU.
    c->djs_cfg = DjsLaunch{};
    int qs = 0, nas = 0;
    if (c->djac_cfg.W == 0 && c->djs_tile >= 0 && c->out_ok && djs_shape(P, &qs, &nas)) {
        for (int W : {64, 32, 16}) {
            if (c->djs_tile > 0 && W > c->djs_tile) continue;
            const size_t lds = djs_lds_bytes(P, W, st64);
            if (lds > LDS_HARD_LIMIT) continue;
            const int b = djs_blocks_per_cu(f64d, ar64, P.rbf, qs, nas, lds);
            if (b >= (c->djs_tile > 0 ? 1 : 2)) {
                c->djs_cfg = DjsLaunch{W, qs, nas, lds, ncu * b};
                break;
            }
        }
    }
    c->jac_ok = bestW > 0;
    c->jac_cfg.W = bestW;
    c->jac_cfg.lds = bestW > 0 ? jacobian_lds_bytes(P, bestW, st64) : 0;
    return SOAP_OK;
}

int upload_constants(soap_ctx *c) {
    const int n = c->n, lw = c->lmax + 1, S = (int)c->Z.size();
    char msg[256] = {0};
    const int ldN = lw + 1; // harmonics tables cover l <= l_max + 1
    std::vector<double> betaC, betaCa, aprime, betaC_lo, aprime_lo, G, rq, WN, c0(n), Nlm((size_t)ldN * ldN);
    if (c->rbf == SOAP_RBF_GTO) {
        betaC.resize((size_t)lw * n * n);
        betaCa.resize((size_t)lw * n * n);
        aprime.resize((size_t)lw * n);
        betaC_lo.resize(betaC.size());
        aprime_lo.resize(aprime.size());
        if (soap_basis_gto(c->r_cut, n, c->lmax, c->sigma, betaC.data(), betaCa.data(), aprime.data(), c0.data(),
                           msg, sizeof msg, betaC_lo.data(), nullptr, aprime_lo.data()) != 0)
            return fail(c, SOAP_EINVAL, "%s", msg);
    } else {
        G.resize((size_t)n * c->Q);
        rq.resize(c->Q);
        if (soap_basis_poly(c->r_cut, n, c->sigma, c->Q, G.data(), rq.data(), c0.data(), msg, sizeof msg) != 0)
            return fail(c, SOAP_EINVAL, "%s", msg);
        if (c->rbf == SOAP_RBF_POLYNOMIAL_LAPLACE) {
            WN.resize((size_t)n * (n + 3) * 4);
            if (soap_basis_poly_laplace(c->r_cut, n, c->sigma, WN.data(), msg, sizeof msg) != 0)
                return fail(c, SOAP_EINVAL, "%s", msg);
        }
    }
    soap_basis_sh_norms(c->lmax + 1, Nlm.data());
    // gradient identities of the harmonics per (l, m >= 0): with the degree
    // l-1 harmonics S', grad S_l,+-m takes S'_{m+1} with cA, S'_{m-1} with
    // cB and S'_m with cC (the combinations are written out in the kernels)
    std::vector<double> gcoef;
    for (int l = 0; l <= c->lmax; ++l)
        for (int m = 0; m <= l; ++m) {
            const long double N = Nlm[(size_t)l * ldN + m];
            auto Np = [&](int k) { return (long double)Nlm[(size_t)(l - 1) * ldN + k]; };
            long double cA = 0, cB = 0, cC = 0;
            if (l >= 1) {
                if (m + 1 <= l - 1) cA = (m == 0 ? N : N / 2) / Np(m + 1);
                if (m >= 1) cB = N * (long double)((l + m) * (l + m - 1)) / (2 * Np(m - 1));
                if (m <= l - 1) cC = N * (long double)(l + m) / Np(m);
            }
            gcoef.push_back((double)cA);
            gcoef.push_back((double)cB);
            gcoef.push_back((double)cC);
            gcoef.push_back((double)(l | m << 8));
        }
    // normalisation of the division-free harmonic recurrence: N_lm (2m-1)!! / (l-m)!
    std::vector<double> Nt((size_t)ldN * ldN, 0.0);
    for (int l = 0; l < ldN; ++l)
        for (int m = 0; m <= l; ++m) {
            long double v = Nlm[(size_t)l * ldN + m];
            for (int k = 1; k <= m; ++k) v *= (long double)(2 * k - 1);
            for (int k = 2; k <= l - m; ++k) v /= (long double)k;
            Nt[(size_t)l * ldN + m] = (double)v;
        }
    // one constant buffer: betaC | betaCa | aprime | remainders of betaC, aprime | G | rq | WN | c0 | Nt | gcoef |
    // exp2 table
    std::vector<double> all;
    size_t o_bc = all.size(); all.insert(all.end(), betaC.begin(), betaC.end());
    size_t o_ba = all.size(); all.insert(all.end(), betaCa.begin(), betaCa.end());
    size_t o_ap = all.size(); all.insert(all.end(), aprime.begin(), aprime.end());
    size_t o_bcl = all.size(); all.insert(all.end(), betaC_lo.begin(), betaC_lo.end());
    size_t o_apl = all.size(); all.insert(all.end(), aprime_lo.begin(), aprime_lo.end());
    size_t o_G = all.size(); all.insert(all.end(), G.begin(), G.end());
    size_t o_rq = all.size(); all.insert(all.end(), rq.begin(), rq.end());
    size_t o_wn = all.size(); all.insert(all.end(), WN.begin(), WN.end());
    size_t o_c0 = all.size(); all.insert(all.end(), c0.begin(), c0.end());
    size_t o_Nt = all.size(); all.insert(all.end(), Nt.begin(), Nt.end());
    size_t o_gc = all.size(); all.insert(all.end(), gcoef.begin(), gcoef.end());
    double e2t[128];
    soap_exp2_table64(e2t);
    while (all.size() % 2) all.push_back(0.0); // 16-byte aligned pairs
    size_t o_e2 = all.size(); all.insert(all.end(), e2t, e2t + 128);
    hipError_t e;
    if ((e = c->d_const.ensure(all.size() * 8)) != hipSuccess) return hip_fail(c, e, "hipMalloc(constants)");
    if ((e = hipMemcpy(c->d_const.p, all.data(), all.size() * 8, hipMemcpyHostToDevice)) != hipSuccess)
        return hip_fail(c, e, "hipMemcpy(constants)");
    double *d = c->d_const.as<double>();
    build_feature_tables(c);
    if ((e = c->d_dtab.ensure(c->dtab.size() * 4)) != hipSuccess) return hip_fail(c, e, "hipMalloc(dtab)");
    if ((e = hipMemcpy(c->d_dtab.p, c->dtab.data(), c->dtab.size() * 4, hipMemcpyHostToDevice)) != hipSuccess)
        return hip_fail(c, e, "hipMemcpy(dtab)");
    if ((e = c->d_fmap.ensure(c->fmap.size() * 4)) != hipSuccess) return hip_fail(c, e, "hipMalloc(fmap)");
    if ((e = hipMemcpy(c->d_fmap.p, c->fmap.data(), c->fmap.size() * 4, hipMemcpyHostToDevice)) != hipSuccess)
        return hip_fail(c, e, "hipMemcpy(fmap)");
    int8_t lut[128];
    std::memset(lut, -1, sizeof lut);
    for (int s = 0; s < S; ++s) lut[c->Z[s]] = (int8_t)s;
    if ((e = c->d_lut.ensure(128)) != hipSuccess) return hip_fail(c, e, "hipMalloc(lut)");
    if ((e = hipMemcpy(c->d_lut.p, lut, 128, hipMemcpyHostToDevice)) != hipSuccess) return hip_fail(c, e, "hipMemcpy(lut)");

    Params &P = c->P;
    P.S = S;
    P.n = n;
    P.lmax = c->lmax;
    P.L = lw * lw;
    P.rbf = c->rbf;
    P.Q = c->Q;
    P.F = (int)c->F;
    P.Fe = (int)c->Fe;
    P.nq_full = c->nq_full;
    P.sigma = c->sigma;
    P.inv_s2 = 1.0 / (c->sigma * c->sigma);
    P.rc = c->r_cut;
    P.inv_rc2 = 2.0 / c->r_cut;
    P.s2 = c->sigma * c->sigma;
    P.hs2 = 0.5 * P.s2;
    P.betaC = d + o_bc;
    P.betaCa = d + o_ba;
    P.aprime = d + o_ap;
    P.betaC_lo = d + o_bcl;
    P.aprime_lo = d + o_apl;
    P.G = d + o_G;
    P.rq = d + o_rq;
    P.WN = d + o_wn;
    P.c0 = d + o_c0;
    P.Nt = d + o_Nt;
    P.gcoef = d + o_gc;
    P.e2t = d + o_e2;
    P.dtab = c->d_dtab.as<uint32_t>();
    P.tri_lw = (int)c->dtab.size();
    return plan_launches(c);
}

hipStream_t to_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

hipEvent_t take_event(soap_ctx *c) {
    if (!c->pool.empty()) {
        hipEvent_t e = c->pool.back();
        c->pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// RAII bracket of one timed segment on a stream
struct SegTimer {
    soap_ctx *c;
    int seg;
    hipStream_t st;
    hipEvent_t a = nullptr;
    SegTimer(soap_ctx *c_, int seg_, hipStream_t st_, bool on = true) : c(c_), seg(seg_), st(st_) {
        if (on && c->timing && (a = take_event(c)) != nullptr) (void)hipEventRecord(a, st);
    }
    void done() {
        if (!a) return;
        hipEvent_t b = take_event(c);
        if (b && hipEventRecord(b, st) == hipSuccess) c->recs.push_back({seg, a, b});
        else c->pool.push_back(a);
        a = nullptr;
    }
};

int check_ctx_device(soap_ctx *c) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(c, e, "hipGetDevice");
    if (dev != c->device) return fail(c, SOAP_EINVAL, "current device %d differs from the context's device %d", dev, c->device);
    return SOAP_OK;
}

// the rows of centers [first, first + count) of the neighbour list
Rows rows_of(const soap_ctx *c, int64_t first, int64_t count) {
    Rows R;
    R.n_atoms = c->n_atoms;
    R.nc = count;
    R.c_base = first;
    R.centers = c->centers ? c->centers + first : nullptr;
    R.spec = c->b_spec.as<uint8_t>();
    R.row_ptr = c->b_row.as<int64_t>() + first;
    R.cols = c->b_cols.as<int32_t>();
    R.e_origin = R.row_ptr;
    return R;
}
// centers [cf, cf + cn) of the output batch that starts at center `first`
Rows rows_part(const soap_ctx *c, int64_t first, int64_t cf, int64_t cn) {
    Rows R = rows_of(c, cf, cn);
    R.e_origin = c->b_row.as<int64_t>() + first;
    return R;
}
Rows rows_of(const soap_ctx *c) { return rows_of(c, 0, c->nc); }

// bytes of the coefficient scratch the Jacobian path keeps per center:
// (c, Dx, Dy, Dz) at the staging precision: float32 in the mixed mode (every
// reader of the scratch rounds it to float32), else float64
size_t scratch_bytes_per_center(const soap_ctx *c) {
    const size_t elt = (c->dtype == SOAP_FP64 || c->ar64) ? 8 : 4;
    return elt * 4 * (size_t)c->P.S * c->P.n * c->P.L;
}

// the radial pass (polynomial quadrature): bytes for the edges of centers [first, first + count)
size_t radial_bytes(const soap_ctx *c, int64_t first, int64_t count) {
    if (c->P.rbf != 1 || count == 0 || c->h_row.size() != (size_t)c->nc + 1) return 0;
    return radial_bytes_per_edge(c->P) * (size_t)(c->h_row[first + count] - c->h_row[first]);
}
size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

Params params_for(const soap_ctx *c, int mode) {
    Params P = c->P;
    const int G = c->groups[mode];
    P.n_groups = G;
    for (int k = 0; k <= G; ++k) P.lgrp[k] = c->lgrp[mode][k];
    return P;
}

} // namespace

extern "C" {

int soap_create(const int32_t *species_Z, int32_t n_species, double r_cut, int32_t n_max, int32_t l_max, double sigma,
                int32_t rbf, soap_ctx **out) {
    g_create_error.clear();
    auto bad = [](const char *msg) {
        g_create_error = msg;
        return SOAP_EINVAL;
    };
    if (!out) return bad("out is NULL");
    *out = nullptr;
    if (!species_Z || n_species < 1 || n_species > 64) return bad("n_species must be in 1..64");
    if (n_max < 1 || n_max > NMAX) return bad("n_max must be in 1..16");
    if (l_max < 0 || l_max > LMAX) return bad("l_max must be in 0..14");
    if (!(sigma > 0) || !(r_cut > 0)) return bad("sigma and r_cut must be positive");
    if (rbf != SOAP_RBF_GTO && rbf != SOAP_RBF_POLYNOMIAL && rbf != SOAP_RBF_POLYNOMIAL_LAPLACE)
        return bad("unknown rbf");
    if (rbf == SOAP_RBF_GTO && !(r_cut > 1.0)) return bad("the GTO basis needs r_cut > 1");
    if (n_species * n_max > 255) return bad("n_species * n_max must not exceed 255");
    std::vector<int32_t> Z(species_Z, species_Z + n_species);
    std::sort(Z.begin(), Z.end());
    for (int k = 0; k < n_species; ++k)
        if (Z[k] < 1 || Z[k] > 127 || (k > 0 && Z[k] == Z[k - 1]))
            return bad("atomic numbers must be distinct and in 1..127");
    soap_ctx *c = new (std::nothrow) soap_ctx();
    if (!c) return SOAP_ENOMEM;
    c->Z = Z;
    c->r_cut = r_cut;
    c->sigma = sigma;
    c->n = n_max;
    c->lmax = l_max;
    c->rbf = rbf;
    int rc;
    hipError_t e = hipGetDevice(&c->device);
    if (e == hipSuccess) e = set_lds_limits();
    if (e == hipSuccess) e = hipHostMalloc((void **)&c->h_flags, 64, hipHostMallocDefault);
    if (e == hipSuccess) e = hipHostMalloc((void **)&c->h_rec, 64, hipHostMallocCoherent);
    if (e == hipSuccess) {
        std::memset(c->h_rec, 0, 64);
        e = hipHostGetDevicePointer((void **)&c->d_rec, c->h_rec, 0);
    }
    if (e == hipSuccess) e = static_scratch(c->device, &c->static_scratch);
    if (e != hipSuccess) {
        g_create_error = std::string("HIP setup failed: ") + hipGetErrorString(e);
        delete c;
        return e == hipErrorOutOfMemory ? SOAP_ENOMEM : SOAP_EHIP;
    }
    if ((rc = upload_constants(c)) != SOAP_OK) {
        g_create_error = c->err;
        soap_destroy(c);
        return rc;
    }
    *out = c;
    return SOAP_OK;
}

int soap_set_option(soap_ctx *c, const char *key, int64_t value) {
    if (!c || !key) return SOAP_EINVAL;
    if (!std::strcmp(key, "dtype")) {
        if (value != SOAP_FP32 && value != SOAP_FP64) return fail(c, SOAP_EINVAL, "dtype must be SOAP_FP32 or SOAP_FP64");
        if (value == c->dtype) return SOAP_OK;
        c->have_rows = false;
        c->dtype = (int)value;
        return plan_launches(c); // occupancy of the float64 kernels
    }
    if (!std::strcmp(key, "arith")) {
        if (value != SOAP_ARITH_MIXED && value != SOAP_ARITH_FP64)
            return fail(c, SOAP_EINVAL, "arith must be SOAP_ARITH_MIXED or SOAP_ARITH_FP64");
        if (value == c->arith) return SOAP_OK;
        c->arith = (int)value;
        return plan_launches(c); // staging sizes and occupancy of the kernels
    }
    if (!std::strcmp(key, "batch_centers")) {
        if (value < 0) return fail(c, SOAP_EINVAL, "batch_centers must be >= 0");
        c->batch_centers = value;
        return SOAP_OK;
    }
    if (!std::strcmp(key, "pipeline")) {
        if (value < 1 || value > 16) return fail(c, SOAP_EINVAL, "pipeline must be in 1..16");
        c->pipe_chunks = (int)value;
        return SOAP_OK;
    }
    if (!std::strcmp(key, "pipeline_density_wg")) {
        if (value < 0 || value > 16) return fail(c, SOAP_EINVAL, "pipeline_density_wg must be in 0..16");
        c->pipe_density_wg = (int)value;
        return SOAP_OK;
    }
    if (!std::strcmp(key, "djac_tile")) {
        if (value != 0 && value != -1 && value != 32 && value != 64)
            return fail(c, SOAP_EINVAL, "djac_tile must be 0, -1, 32 or 64");
        c->djac_tile = (int)value;
        return plan_launches(c);
    }
    if (!std::strcmp(key, "djs_tile")) {
        if (value != 0 && value != -1 && value != 16 && value != 32 && value != 64)
            return fail(c, SOAP_EINVAL, "djs_tile must be 0, -1, 16, 32 or 64");
        c->djs_tile = (int)value;
        return plan_launches(c);
    }
    if (!std::strcmp(key, "desc_tile")) {
        if (value != 0 && value != -1 && value != 16 && value != 32 && value != 64)
            return fail(c, SOAP_EINVAL, "desc_tile must be 0, -1, 16, 32 or 64");
        c->desc_tile = (int)value;
        return plan_launches(c);
    }
    if (!std::strcmp(key, "jac_tile")) {
        if (value < 0 || value > jacobian_max_w())
            return fail(c, SOAP_EINVAL, "jac_tile must be in 0..%d", jacobian_max_w());
        c->jac_tile = (int)value;
        return plan_launches(c);
    }
    if (!std::strcmp(key, "out_rows")) {
        if (value != 0 && value != 1) return fail(c, SOAP_EINVAL, "out_rows must be 0 or 1");
        c->out_rows = value == 1;
        return plan_launches(c);
    }
    if (!std::strcmp(key, "timing")) {
        if (value != 0 && value != 1) return fail(c, SOAP_EINVAL, "timing must be 0 or 1");
        c->timing = value == 1;
        return SOAP_OK;
    }
    if (!std::strcmp(key, "quad_n")) {
        if (value < 8 || value > 256) return fail(c, SOAP_EINVAL, "quad_n must be in 8..256");
        if ((int)value == c->Q) return SOAP_OK;
        c->Q = (int)value;
        return upload_constants(c);
    }
    return fail(c, SOAP_EINVAL, "unknown option '%s'", key);
}

int soap_get_option(const soap_ctx *c, const char *key, int64_t *value) {
    if (!c || !key || !value) return SOAP_EINVAL;
    const struct {
        const char *k;
        int64_t v;
    } tab[] = {{"dtype", c->dtype},
               {"arith", c->arith},
               {"quad_n", c->Q},
               {"timing", c->timing ? 1 : 0},
               {"desc_tile", c->desc_tile},
               {"jac_tile", c->jac_tile},
               {"djac_tile", c->djac_tile},
               {"djs_tile", c->djs_tile},
               {"pipeline", c->pipe_chunks},
               {"batch_centers", c->batch_centers},
               {"device", c->device},
               {"pipeline_density_wg", c->pipe_density_wg},
               {"out_rows", c->out_rows ? 1 : 0},
               {"output_kernel_rows", c->out_plan.rows ? 1 : 0},
               {"jacobian_l_groups", c->groups[1]},
               {"jacobian_density_tile",
                c->djac_cfg.W > 0 ? c->djac_cfg.W : (c->djs_cfg.W > 0 ? c->djs_cfg.W : c->dens_cfg[1].W)},
               {"jacobian_density_lds", (int64_t)(c->djac_cfg.W > 0 ? c->djac_cfg.lds
                                                                    : (c->djs_cfg.W > 0 ? c->djs_cfg.lds
                                                                                        : c->dens_cfg[1].lds))},
               {"jacobian_tile", c->jac_cfg.W},
               {"jacobian_lds", (int64_t)c->jac_cfg.lds},
               {"output_lds", (int64_t)c->out_plan.lds},
               {"descriptor_kernel", c->desc_cfg.W > 0 ? 1 : 0},
               // 0 k_density, 1 k_djac, 2 k_djs (then the output kernel)
               {"jacobian_density_kernel", c->djac_cfg.W > 0 ? 1 : (c->djs_cfg.W > 0 ? 2 : 0)}};
    for (const auto &t : tab)
        if (!std::strcmp(key, t.k)) {
            *value = t.v;
            return SOAP_OK;
        }
    return SOAP_EINVAL;
}

int64_t soap_num_features(const soap_ctx *c) { return c ? c->F : -1; }
int64_t soap_num_edge_features(const soap_ctx *c) { return c ? c->Fe : -1; }

int soap_feature_labels(const soap_ctx *c, int32_t *out) {
    if (!c || !out) return SOAP_EINVAL;
    const int lw = c->lmax + 1;
    for (int q = 0; q < c->nq_full; ++q) {
        const uint32_t f = c->fq[q];
        for (int l = 0; l < lw; ++l) {
            int32_t *o = out + 5 * ((int64_t)q * lw + l);
            o[0] = f & 0xff;
            o[1] = (f >> 8) & 0xff;
            o[2] = (f >> 16) & 0xff;
            o[3] = f >> 24;
            o[4] = l;
        }
    }
    return SOAP_OK;
}

int soap_feature_map(const soap_ctx *c, int32_t s, int32_t *out) {
    if (!c || !out || s < 0 || s >= (int32_t)c->Z.size()) return SOAP_EINVAL;
    std::memcpy(out, c->fmap.data() + (size_t)s * c->Fe, sizeof(int32_t) * c->Fe);
    return SOAP_OK;
}

// The rows over n_atoms atoms (an extended structure for periodic cells, whose
// first center_bound atoms are the real ones).
static int build_rows(soap_ctx *c, int64_t n_atoms, int64_t center_bound, const void *pos_dev, const int32_t *Z_dev,
                      int64_t n_centers, const int32_t *centers_dev, int64_t *E_out, hipStream_t st) {
    const bool f64 = c->dtype == SOAP_FP64;
    int64_t H = 1024;
    while (H < 2 * n_atoms) H <<= 1;
    const int64_t tiles = (std::max(H, n_centers) + 2047) / 2048 + 2;
    hipError_t e = hipSuccess;
    auto need = [&](DevBuf &b, size_t bytes) {
        if (e == hipSuccess) e = b.ensure(bytes);
    };
    need(c->b_zero, nbr_zero_bytes(H));
    need(c->b_bstart, 4 * (H + 1));
    need(c->b_acell, 16 * n_atoms);
    need(c->b_srec, (f64 ? 32 : 16) * n_atoms);
    need(c->b_sspec, n_atoms);
    need(c->b_spec, n_atoms);
    need(c->b_deg, 4 * n_centers);
    need(c->b_slots, 4 * (size_t)TCAP * n_centers);
    need(c->b_scan, 8 * tiles);
    need(c->b_row, 8 * (n_centers + 1));
    if (e != hipSuccess) return hip_fail(c, e, "hipMalloc(neighbour workspace)");
    NbrWork &w = c->nw;
    w.H = H;
    w.zero = c->b_zero.p;
    w.zero_bytes = nbr_zero_bytes(H);
    char *z = (char *)c->b_zero.p;
    w.flags = (int32_t *)z;
    w.work = (unsigned long long *)(z + NBR_FLAGS_BYTES);
    w.bucket_count = (int32_t *)(z + NBR_FLAGS_BYTES + NBR_WORK_BYTES);
    w.bucket_fill = w.bucket_count + H;
    w.bucket_start = c->b_bstart.as<int32_t>();
    w.atom_cell = c->b_acell.as<int4>();
    w.sorted_rec = c->b_srec.p;
    w.sorted_spec = c->b_sspec.as<uint8_t>();
    w.deg = c->b_deg.as<int32_t>();
    w.slots = c->b_slots.as<int32_t>();
    w.scan_tmp = c->b_scan.as<int64_t>();
    int64_t *row = c->b_row.as<int64_t>();
    const int64_t seq = ++c->rec_seq;
    bool rec_written = false;
    e = nbr_phase1(w, n_atoms, center_bound, pos_dev, f64, Z_dev, c->d_lut.as<int8_t>(), c->b_spec.as<uint8_t>(),
                   n_centers, centers_dev, c->r_cut, row, st, c->d_rec, seq, &rec_written);
    if (e != hipSuccess) return hip_fail(c, e, "neighbour search");
    c->work_epoch = WorkBase{}; // the density work counters were zeroed with the flags
    // With a rows buffer from an earlier build, the short rows are packed
    // before the host reads the total: the GPU works through the round trip.
    // k_pack writes nothing if the total exceeds the buffer; it runs again
    // below once the buffer has grown.
    const int64_t cap0 = c->b_cols.p ? (int64_t)(c->b_cols.cap / 4) : 0;
    if (cap0 > 0 && (e = nbr_pack(w, n_centers, row, c->b_cols.as<int32_t>(), cap0, st)) != hipSuccess)
        return hip_fail(c, e, "neighbour rows");
    // The polynomial quadrature's radial pass places each call's edges from a
    // host copy of the row offsets: copied with the flags, one synchronisation.
    c->h_row.clear();
    const bool rows_to_host = c->rbf == SOAP_RBF_POLYNOMIAL;
    if (rows_to_host) {
        const size_t m = (size_t)n_centers + 1;
        if (m > c->h_rowp_cap) {
            if (c->h_rowp) (void)hipHostFree(c->h_rowp);
            c->h_rowp = nullptr;
            c->h_rowp_cap = 0;
            if ((e = hipHostMalloc((void **)&c->h_rowp, 8 * m, hipHostMallocDefault)) != hipSuccess)
                return hip_fail(c, e, "hipHostMalloc(row offsets)");
            c->h_rowp_cap = m;
        }
        if ((e = hipMemcpyAsync(c->h_rowp, row, 8 * m, hipMemcpyDeviceToHost, st)) != hipSuccess)
            return hip_fail(c, e, "neighbour row offsets");
    }
    // The degree scan's host record when it writes one: waiting for its
    // sequence number returns as soon as the scan has ended (the short rows may
    // still be packing), where a copy and a stream synchronisation would wait
    // for a copy launch and the end of the stream.  After a bounded spin the
    // stream is synchronised instead (work queued before this call).
    bool have_rec = false;
    if (rec_written && !rows_to_host) {
        const auto t0 = std::chrono::steady_clock::now();
        for (;;) {
            if (__atomic_load_n(c->h_rec + 3, __ATOMIC_ACQUIRE) == seq) {
                have_rec = true;
                break;
            }
            if (std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(20)) {
                if ((e = hipStreamSynchronize(st)) != hipSuccess) return hip_fail(c, e, "neighbour search (sync)");
                have_rec = __atomic_load_n(c->h_rec + 3, __ATOMIC_ACQUIRE) == seq;
                break;
            }
            __builtin_ia32_pause();
        }
    }
    int32_t bad, maxdeg, n_long;
    int64_t E;
    if (have_rec) {
        const uint64_t r0 = (uint64_t)c->h_rec[0];
        bad = (int32_t)(uint32_t)r0;
        maxdeg = (int32_t)(uint32_t)(r0 >> 32);
        n_long = (int32_t)c->h_rec[1];
        E = c->h_rec[2];
    } else {
        // flags[0..3] and the total degree (int64 at flags + 4) in one copy
        if ((e = hipMemcpyAsync(c->h_flags, w.flags, 24, hipMemcpyDeviceToHost, st)) != hipSuccess ||
            (e = hipStreamSynchronize(st)) != hipSuccess)
            return hip_fail(c, e, "neighbour search (sync)");
        bad = c->h_flags[0];
        maxdeg = c->h_flags[1];
        n_long = c->h_flags[2];
        std::memcpy(&E, c->h_flags + 4, 8);
    }
    if (rows_to_host) c->h_row.assign(c->h_rowp, c->h_rowp + n_centers + 1);
    if (bad & 1) return fail(c, SOAP_ESPECIES, "an atomic number is not in the species list");
    if (bad & 2) return fail(c, SOAP_EINVAL, "a center index is out of range");
    if (maxdeg > MAX_DEGREE)
        return fail(c, SOAP_ECAPACITY, "a center has %d neighbours (limit %d)", maxdeg, MAX_DEGREE);
    const bool packed = cap0 > 0 && E <= cap0;
    if ((e = c->b_cols.ensure(4 * (size_t)std::max<int64_t>(E, 1))) != hipSuccess)
        return hip_fail(c, e, "hipMalloc(neighbour rows)");
    e = nbr_phase2(w, n_atoms, pos_dev, f64, n_centers, centers_dev, c->r_cut, row, n_long > 0, packed,
                   c->b_cols.as<int32_t>(), (int64_t)(c->b_cols.cap / 4), st);
    if (e != hipSuccess) return hip_fail(c, e, "neighbour rows");
    *E_out = E;
    return SOAP_OK;
}

// Periodic cell: the atoms plus their images that can reach an atom within
// r_cut become an extended structure (context-owned arrays); returns its size.
static int build_images(soap_ctx *c, int64_t n_atoms, const void *pos_dev, const int32_t *Z_dev, int64_t *n_ext,
                        hipStream_t st) {
    const bool f64 = c->dtype == SOAP_FP64;
    const size_t elt = f64 ? 8 : 4;
    const int64_t tiles = (n_atoms + 2047) / 2048 + 2;
    hipError_t e = hipSuccess;
    auto need = [&](DevBuf &b, size_t bytes) {
        if (e == hipSuccess) e = b.ensure(bytes);
    };
    need(c->b_img_lohi, 8 * 6);
    need(c->b_img_cnt, 4 * n_atoms);
    need(c->b_img_start, 8 * (n_atoms + 1));
    need(c->b_scan, 8 * tiles);
    if (e != hipSuccess) return hip_fail(c, e, "hipMalloc(periodic workspace)");
    double *lohi = c->b_img_lohi.as<double>();
    int64_t *start = c->b_img_start.as<int64_t>();
    if ((e = periodic_count(n_atoms, pos_dev, f64, c->cell, lohi, c->b_img_cnt.as<int32_t>(), st)) != hipSuccess ||
        (e = nbr_exclusive_scan(n_atoms, c->b_img_cnt.as<int32_t>(), start, c->b_scan.as<int64_t>(), nullptr, st)) !=
            hipSuccess ||
        (e = hipMemcpyAsync(c->h_flags + 8, start + n_atoms, 8, hipMemcpyDeviceToHost, st)) != hipSuccess ||
        (e = hipStreamSynchronize(st)) != hipSuccess)
        return hip_fail(c, e, "periodic images");
    int64_t n_img;
    std::memcpy(&n_img, c->h_flags + 8, 8);
    if (n_img < 0 || n_atoms + n_img > INT32_MAX)
        return fail(c, SOAP_ECAPACITY, "%lld periodic images exceed the supported atom count", (long long)n_img);
    const int64_t nx = n_atoms + n_img;
    need(c->b_pos_ext, elt * 3 * nx);
    need(c->b_Z_ext, 4 * nx);
    need(c->b_map_atom, 4 * nx);
    need(c->b_map_img, 12 * nx);
    if (e != hipSuccess) return hip_fail(c, e, "hipMalloc(periodic images)");
    e = periodic_fill(n_atoms, pos_dev, f64, Z_dev, c->cell, lohi, start, c->b_pos_ext.p, c->b_Z_ext.as<int32_t>(),
                      c->b_map_atom.as<int32_t>(), c->b_map_img.as<int32_t>(), st);
    if (e != hipSuccess) return hip_fail(c, e, "periodic images");
    *n_ext = nx;
    return SOAP_OK;
}

int soap_build_neighbors(soap_ctx *c, int64_t n_atoms, const void *pos_dev, const int32_t *Z_dev, int64_t n_centers,
                         const int32_t *centers_dev, int64_t *n_edges_out, void *stream) {
    if (!c) return SOAP_EINVAL;
    c->have_rows = false;
    if (n_atoms < 1 || n_atoms > INT32_MAX || !pos_dev || !Z_dev || n_centers < 1 || !n_edges_out)
        return fail(c, SOAP_EINVAL, "invalid arguments to soap_build_neighbors");
    if (!centers_dev && n_centers != n_atoms)
        return fail(c, SOAP_EINVAL, "n_centers must equal n_atoms when centers_dev is NULL");
    int rc;
    if ((rc = check_ctx_device(c)) != SOAP_OK) return rc;
    hipStream_t st = to_stream(stream);
    SegTimer timer(c, 0, st);
    int64_t E = 0, n_rows_atoms = n_atoms;
    const void *pos_rows = pos_dev;
    const int32_t *Z_rows = Z_dev, *cen_rows = centers_dev;
    if (c->periodic) {
        if ((rc = build_images(c, n_atoms, pos_dev, Z_dev, &n_rows_atoms, st)) != SOAP_OK) return rc;
        pos_rows = c->b_pos_ext.p;
        Z_rows = c->b_Z_ext.as<int32_t>();
        if (!centers_dev) { // every atom, but not the images: an explicit list
            hipError_t e = c->b_iota.ensure(4 * (size_t)n_centers);
            if (e == hipSuccess) e = fill_iota(n_centers, c->b_iota.as<int32_t>(), st);
            if (e != hipSuccess) return hip_fail(c, e, "periodic centers");
            cen_rows = c->b_iota.as<int32_t>();
        }
    }
    if ((rc = build_rows(c, n_rows_atoms, n_atoms, pos_rows, Z_rows, n_centers, cen_rows, &E, st)) != SOAP_OK)
        return rc;
    timer.done();
    c->have_rows = true;
    c->n_atoms = n_atoms;
    c->n_ext = n_rows_atoms;
    c->nc = n_centers;
    c->E = E;
    c->pos = pos_rows;
    c->Zdev = Z_rows;
    c->centers = cen_rows;
    c->built_f64 = c->dtype == SOAP_FP64;
    c->built_periodic = c->periodic;
    *n_edges_out = E;
    return SOAP_OK;
}

int soap_set_cell(soap_ctx *c, const double *cell, const int32_t *pbc) {
    if (!c) return SOAP_EINVAL;
    c->have_rows = false;
    if (!cell) {
        c->periodic = false;
        return SOAP_OK;
    }
    if (!pbc) return fail(c, SOAP_EINVAL, "pbc is NULL");
    PeriodicCell C{};
    for (int k = 0; k < 9; ++k) C.M[k] = cell[k];
    const double *a = C.M, *b = C.M + 3, *cc = C.M + 6;
    const double det = a[0] * (b[1] * cc[2] - b[2] * cc[1]) - a[1] * (b[0] * cc[2] - b[2] * cc[0]) +
                       a[2] * (b[0] * cc[1] - b[1] * cc[0]);
    if (!(std::fabs(det) > 1e-9)) return fail(c, SOAP_EINVAL, "the cell vectors are degenerate");
    // B = M^-1 (adjugate over the determinant)
    const double *m = C.M;
    C.B[0] = (m[4] * m[8] - m[5] * m[7]) / det;
    C.B[1] = (m[2] * m[7] - m[1] * m[8]) / det;
    C.B[2] = (m[1] * m[5] - m[2] * m[4]) / det;
    C.B[3] = (m[5] * m[6] - m[3] * m[8]) / det;
    C.B[4] = (m[0] * m[8] - m[2] * m[6]) / det;
    C.B[5] = (m[2] * m[3] - m[0] * m[5]) / det;
    C.B[6] = (m[3] * m[7] - m[4] * m[6]) / det;
    C.B[7] = (m[1] * m[6] - m[0] * m[7]) / det;
    C.B[8] = (m[0] * m[4] - m[1] * m[3]) / det;
    bool any = false;
    for (int k = 0; k < 3; ++k) {
        C.pbc[k] = pbc[k] != 0;
        any = any || C.pbc[k];
        if (!C.pbc[k]) continue;
        // interplanar spacing d_k = |det| / |v_{k+1} x v_{k+2}|: an image n moves by
        // at least |n_k| d_k, so fractional coordinates beyond r_cut / d_k of every
        // atom cannot reach the cutoff (padded against rounding)
        const double *u = C.M + 3 * ((k + 1) % 3), *v = C.M + 3 * ((k + 2) % 3);
        const double cx = u[1] * v[2] - u[2] * v[1], cy = u[2] * v[0] - u[0] * v[2], cz = u[0] * v[1] - u[1] * v[0];
        const double d = std::fabs(det) / std::sqrt(cx * cx + cy * cy + cz * cz);
        C.eps[k] = c->r_cut / d * (1.0 + 1e-9) + 1e-9;
    }
    c->cell = C;
    c->periodic = any;
    return SOAP_OK;
}

int soap_get_neighbor_images(soap_ctx *c, int32_t *img_dev, void *stream) {
    if (!c || !img_dev) return SOAP_EINVAL;
    if (!c->have_rows) return fail(c, SOAP_ESTATE, "no neighbour list: call soap_build_neighbors first");
    hipError_t e = map_edges(c->E, c->b_cols.as<int32_t>(), nullptr,
                             c->built_periodic ? c->b_map_img.as<int32_t>() : nullptr, nullptr, img_dev,
                             to_stream(stream));
    return e == hipSuccess ? SOAP_OK : hip_fail(c, e, "soap_get_neighbor_images");
}

int soap_get_neighbors(soap_ctx *c, int64_t *row_ptr_dev, int32_t *cols_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    if (!c->have_rows) return fail(c, SOAP_ESTATE, "no neighbour list: call soap_build_neighbors first");
    hipStream_t st = to_stream(stream);
    hipError_t e = hipSuccess;
    if (row_ptr_dev)
        e = hipMemcpyAsync(row_ptr_dev, c->b_row.p, 8 * (c->nc + 1), hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess && cols_dev && c->E > 0)
        e = c->built_periodic ? map_edges(c->E, c->b_cols.as<int32_t>(), c->b_map_atom.as<int32_t>(), nullptr,
                                          cols_dev, nullptr, st)
                              : hipMemcpyAsync(cols_dev, c->b_cols.p, 4 * c->E, hipMemcpyDeviceToDevice, st);
    return e == hipSuccess ? SOAP_OK : hip_fail(c, e, "soap_get_neighbors");
}

// whether the kernels of a density mode fit this basis (mode 1 also needs the
// edge Jacobian kernel, and the output kernel when the density kernel splits
// l into groups; the one-workgroup-per-center kernel needs neither split)
static bool jacobian_path_ok(const soap_ctx *c, int mode) {
    if (mode == 1 && c->djac_cfg.W > 0) return c->jac_ok;
    if (mode == 1 && c->djs_cfg.W > 0) return c->jac_ok && c->out_ok;
    return c->dens_ok[mode] && (mode != 1 || (c->jac_ok && (c->groups[1] == 1 || c->out_ok)));
}

// The polynomial quadrature's radial factors (B_nl, Bh_nl) of the edges of
// centers [first, first + count), evaluated once per call by k_radial into
// buf (NULL = the context's buffer, grown as needed) and read by every
// kernel of the call through P.rad.  Nothing to do for the other bases.
static int prepare_radial(soap_ctx *c, int64_t first, int64_t count, void *buf, hipStream_t st) {
    c->P.rad = nullptr;
    c->P.rad_e0 = 0;
    if (c->P.rbf != 1 || count == 0) return SOAP_OK;
    if (c->h_row.size() != (size_t)c->nc + 1) return fail(c, SOAP_ESTATE, "neighbour row offsets missing");
    if (!buf) {
        hipError_t e = c->b_radial.ensure(radial_bytes(c, first, count));
        if (e != hipSuccess) return hip_fail(c, e, "hipMalloc(radial factors)");
        buf = c->b_radial.p;
    }
    const int64_t e0 = c->h_row[first];
    hipError_t e = launch_radial(c->P, rows_of(c, first, count), c->pos, c->built_f64, e0, buf, st);
    if (e != hipSuccess) return hip_fail(c, e, "radial kernel");
    c->P.rad = (const double2 *)buf;
    c->P.rad_e0 = e0;
    return SOAP_OK;
}

// Centers [first, first + count) of the neighbour list; outputs are indexed
// from the batch's first center (and edge).
// mode as launch_density: 0 descriptor / coefficients, 1 descriptor + Jacobian,
// 2 coefficient Jacobian.  scratch: the Jacobian path's coefficient scratch
// (NULL = the context's, grown as needed).
// timed = false: no timer events (they may allocate).  wg_per_cu > 0 caps
// the persistent density kernel's workgroups per CU.
static int run_density(soap_ctx *c, int mode, int64_t first, int64_t count, void *desc, void *c_out, void *jself,
                       void *jc_edge, void *scratch, void *stream, bool timed = true, int wg_per_cu = 0,
                       bool prep_radial = true) {
    if (!c->have_rows) return fail(c, SOAP_ESTATE, "no neighbour list: call soap_build_neighbors first");
    int rc;
    if ((rc = check_ctx_device(c)) != SOAP_OK) return rc;
    if (!jacobian_path_ok(c, mode))
        return fail(c, SOAP_EINVAL, "basis too large for the on-chip memory of the %s kernels",
                    mode == 2 ? "coefficient Jacobian" : "Jacobian");
    // a caller-given scratch also holds the radial factors, after the coefficients
    void *rbuf = (scratch && mode == 1) ? (char *)scratch + align256(scratch_bytes_per_center(c) * (size_t)count)
                                        : nullptr;
    if (mode == 1 && !scratch) {
        hipError_t e = c->b_cscratch.ensure(scratch_bytes_per_center(c) * (size_t)count);
        if (e != hipSuccess) return hip_fail(c, e, "hipMalloc(coefficient scratch)");
        scratch = c->b_cscratch.p;
    }
    SegTimer timer(c, 1, to_stream(stream), timed);
    if (prep_radial && (rc = prepare_radial(c, first, count, rbuf, to_stream(stream))) != SOAP_OK) return rc;
    const Params P = params_for(c, mode);
    if (mode == 0 && c->desc_cfg.W > 0) { // one wave per center
        hipError_t e = launch_desc(P, rows_of(c, first, count), c->pos, c->built_f64, c->ar64, c->desc_cfg, desc, c_out,
                                   to_stream(stream));
        if (e != hipSuccess) return hip_fail(c, e, "descriptor kernel");
        timer.done();
        return SOAP_OK;
    }
    if (mode == 1 && c->djac_cfg.W > 0) { // one workgroup per center
        DjacLaunch dj = c->djac_cfg;
        if (wg_per_cu > 0) {
            int ncu = 256;
            (void)hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, c->device);
            dj.blocks = std::max(1, std::min(dj.blocks, ncu * wg_per_cu));
        }
        hipError_t e = launch_djac(P, rows_of(c, first, count), c->pos, c->built_f64, c->ar64, dj, desc, jself,
                                   scratch, to_stream(stream));
        if (e != hipSuccess) return hip_fail(c, e, "density kernel");
        timer.done();
        return SOAP_OK;
    }
    if (mode == 1 && c->djs_cfg.W > 0) { // one workgroup per center, then the output kernel
        DjsLaunch dj = c->djs_cfg;
        if (wg_per_cu > 0) {
            int ncu = 256;
            (void)hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, c->device);
            dj.blocks = std::max(1, std::min(dj.blocks, ncu * wg_per_cu));
        }
        hipError_t e = launch_djs(P, rows_of(c, first, count), c->pos, c->built_f64, c->ar64, dj, scratch,
                                  to_stream(stream));
        if (e != hipSuccess) return hip_fail(c, e, "density kernel");
        e = launch_outputs(P, c->out_plan, count, c->built_f64, scratch, desc, jself, to_stream(stream));
        if (e != hipSuccess) return hip_fail(c, e, "output kernel");
        timer.done();
        return SOAP_OK;
    }
    DensityLaunch cfg = c->dens_cfg[mode];
    if (wg_per_cu > 0) {
        int ncu = 256;
        (void)hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, c->device);
        cfg.blocks = std::max(1, std::min(cfg.blocks, ncu * wg_per_cu / std::max(1, P.n_groups)));
    }
    hipError_t e = launch_density(P, rows_of(c, first, count), c->pos, c->built_f64, c->ar64, mode, cfg,
                                  c->nw.work, &c->work_epoch, desc, c_out, jself, scratch, jc_edge, to_stream(stream));
    if (e != hipSuccess) return hip_fail(c, e, "density kernel");
    if (mode == 1 && P.n_groups > 1) { // with one l-group the density kernel writes desc and jself
        e = launch_outputs(P, c->out_plan, count, c->built_f64, scratch, desc, jself, to_stream(stream));
        if (e != hipSuccess) return hip_fail(c, e, "output kernel");
    }
    timer.done();
    return SOAP_OK;
}
static int run_density(soap_ctx *c, int mode, void *desc, void *c_out, void *jself, void *jc_edge, void *stream) {
    return run_density(c, mode, 0, c->nc, desc, c_out, jself, jc_edge, nullptr, stream);
}

// a batch [first, first + count) of the centers of the neighbour list
static int check_batch(soap_ctx *c, int64_t first, int64_t count) {
    if (!c->have_rows) return fail(c, SOAP_ESTATE, "no neighbour list: call soap_build_neighbors first");
    if (first < 0 || count < 0 || first > c->nc || count > c->nc - first)
        return fail(c, SOAP_EINVAL, "center batch [%lld, %lld) outside the %lld centers of the neighbour list",
                    (long long)first, (long long)(first + count), (long long)c->nc);
    return SOAP_OK;
}

int soap_compute(soap_ctx *c, void *desc_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    if (!desc_dev) return fail(c, SOAP_EINVAL, "desc_dev is NULL");
    return run_density(c, 0, desc_dev, nullptr, nullptr, nullptr, stream);
}

int soap_coefficients(soap_ctx *c, void *c_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    if (!c_dev) return fail(c, SOAP_EINVAL, "c_dev is NULL");
    return run_density(c, 0, nullptr, c_dev, nullptr, nullptr, stream);
}

int soap_coefficient_derivatives(soap_ctx *c, void *c_dev, void *jc_edge_dev, void *jc_self_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    if (!c_dev || !jc_self_dev || (!jc_edge_dev && c->E > 0)) return fail(c, SOAP_EINVAL, "output pointer is NULL");
    return run_density(c, 2, nullptr, c_dev, jc_self_dev, jc_edge_dev, stream);
}

int soap_compute_averaged(soap_ctx *c, int32_t mode, void *desc_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    if (!desc_dev) return fail(c, SOAP_EINVAL, "desc_dev is NULL");
    if (mode != SOAP_AVERAGE_INNER && mode != SOAP_AVERAGE_OUTER)
        return fail(c, SOAP_EINVAL, "averaging mode must be SOAP_AVERAGE_INNER or SOAP_AVERAGE_OUTER");
    if (!c->have_rows) return fail(c, SOAP_ESTATE, "no neighbour list: call soap_build_neighbors first");
    const size_t elt = c->built_f64 ? 8 : 4;
    const Params &P = c->P;
    const int64_t cols = mode == SOAP_AVERAGE_OUTER ? c->F : (int64_t)P.S * P.n * P.L;
    hipError_t e = c->b_avg.ensure(elt * (size_t)c->nc * cols);
    if (e == hipSuccess) e = c->b_avg_part.ensure(8 * (size_t)cols * (AVG_CHUNKS + 1));
    if (e != hipSuccess) return hip_fail(c, e, "hipMalloc(averaging scratch)");
    // per-center rows (descriptor or coefficients), then their column means
    int rc = mode == SOAP_AVERAGE_OUTER ? run_density(c, 0, c->b_avg.p, nullptr, nullptr, nullptr, stream)
                                        : run_density(c, 0, nullptr, c->b_avg.p, nullptr, nullptr, stream);
    if (rc != SOAP_OK) return rc;
    double *part = c->b_avg_part.as<double>(), *mean = part + (size_t)AVG_CHUNKS * cols;
    e = launch_column_mean(c->b_avg.p, c->built_f64, c->nc, cols, part, mode == SOAP_AVERAGE_OUTER ? desc_dev : nullptr,
                           mean, to_stream(stream));
    if (e == hipSuccess && mode == SOAP_AVERAGE_INNER)
        e = launch_power_single(P, c->built_f64, mean, desc_dev, to_stream(stream)); // Eq. powerspectrum of the mean c
    if (e != hipSuccess) return hip_fail(c, e, "averaging kernels");
    return SOAP_OK;
}

// Pipelined descriptor + Jacobian: the batch in K center chunks; the density
// kernel of each chunk on `stream`, the Jacobian kernel of the chunk on the
// context's second stream once the chunk's coefficients are in scratch, so
// that the compute-bound density kernel of chunk k + 1 runs beside the
// store-bound Jacobian kernel of chunk k; `stream` waits for the last one.
static int run_derivatives_pipelined(soap_ctx *c, int64_t first, int64_t count, int K, void *desc_dev,
                                     void *jac_edge_dev, void *jac_self_dev, void *stream) {
    hipStream_t st = to_stream(stream);
    hipError_t e = hipSuccess;
    if (!c->aux) e = hipStreamCreateWithFlags(&c->aux, hipStreamNonBlocking);
    while (e == hipSuccess && (int)c->pipe_ev.size() < K + 1) {
        hipEvent_t ev = nullptr;
        e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e == hipSuccess) c->pipe_ev.push_back(ev);
    }
    if (e == hipSuccess) e = c->b_cscratch.ensure(scratch_bytes_per_center(c) * (size_t)count);
    if (e != hipSuccess) return hip_fail(c, e, "pipelined derivatives (setup)");
    char *scratch = (char *)c->b_cscratch.p;
    { // the radial factors of every chunk at once: the chunks' Jacobian launches read them on the other stream
        SegTimer timer(c, 1, st);
        const int rc = prepare_radial(c, first, count, nullptr, st);
        if (rc != SOAP_OK) return rc;
        timer.done();
    }
    const size_t elt = c->built_f64 ? 8 : 4, pc = scratch_bytes_per_center(c);
    for (int k = 0; k < K; ++k) {
        const int64_t cf = first + count * k / K, cn = first + count * (k + 1) / K - cf;
        if (cn == 0) continue;
        const size_t o = (size_t)(cf - first);
        int rc = run_density(c, 1, cf, cn, (char *)desc_dev + o * c->F * elt, nullptr,
                             (char *)jac_self_dev + o * 3 * c->F * elt, nullptr, scratch + o * pc, stream, true,
                             c->pipe_density_wg, false);
        if (rc != SOAP_OK) return rc;
        if ((e = hipEventRecord(c->pipe_ev[k], st)) != hipSuccess ||
            (e = hipStreamWaitEvent(c->aux, c->pipe_ev[k], 0)) != hipSuccess)
            return hip_fail(c, e, "pipelined derivatives (events)");
        SegTimer timer(c, 2, c->aux);
        e = launch_jacobian(c->P, rows_part(c, first, cf, cn), c->pos, c->built_f64, c->ar64, c->jac_cfg,
                            scratch + o * pc, jac_edge_dev, c->aux);
        if (e != hipSuccess) return hip_fail(c, e, "Jacobian kernel");
        timer.done();
    }
    if ((e = hipEventRecord(c->pipe_ev[K], c->aux)) != hipSuccess ||
        (e = hipStreamWaitEvent(st, c->pipe_ev[K], 0)) != hipSuccess)
        return hip_fail(c, e, "pipelined derivatives (join)");
    return SOAP_OK;
}

// descriptor + Jacobian of the centers [first, first + count) in consecutive
// batches of at most B centers, one after another on `stream`: the density
// step and the Jacobian kernel of each batch, the coefficient scratch (and the
// polynomial radial factors) sized for one batch.  Every output is indexed
// from `first`, as in one call (the edge blocks through Rows::e_origin).
static int run_derivatives_batched(soap_ctx *c, int64_t first, int64_t count, int64_t B, void *desc_dev,
                                   void *jac_edge_dev, void *jac_self_dev, void *stream) {
    const size_t elt = c->built_f64 ? 8 : 4;
    for (int64_t cf = first; cf < first + count; cf += B) {
        const int64_t cn = std::min(B, first + count - cf), o = cf - first;
        int rc = run_density(c, 1, cf, cn, (char *)desc_dev + o * c->F * elt, nullptr,
                             (char *)jac_self_dev + o * 3 * c->F * elt, nullptr, nullptr, stream);
        if (rc != SOAP_OK) return rc;
        if (c->E == 0) continue;
        SegTimer timer(c, 2, to_stream(stream));
        hipError_t e = launch_jacobian(c->P, rows_part(c, first, cf, cn), c->pos, c->built_f64, c->ar64, c->jac_cfg,
                                       c->b_cscratch.p, jac_edge_dev, to_stream(stream));
        if (e != hipSuccess) return hip_fail(c, e, "Jacobian kernel");
        timer.done();
    }
    return SOAP_OK;
}

// descriptor + Jacobian of a center batch; scratch as run_density
static int run_derivatives(soap_ctx *c, int64_t first, int64_t count, void *desc_dev, void *jac_edge_dev,
                           void *jac_self_dev, void *scratch, void *stream, bool timed = true) {
    if (count == 0) return SOAP_OK;
    if (timed && !scratch && c->batch_centers > 0 && count > c->batch_centers) {
        int rc;
        if (!jacobian_path_ok(c, 1))
            return fail(c, SOAP_EINVAL, "basis too large for the on-chip memory of the Jacobian kernels");
        if ((rc = check_ctx_device(c)) != SOAP_OK) return rc;
        return run_derivatives_batched(c, first, count, c->batch_centers, desc_dev, jac_edge_dev, jac_self_dev,
                                       stream);
    }
    // the pipelined path needs its own stream, events and the context's
    // scratch: not for the allocation-free entry point
    if (timed && !scratch && c->pipe_chunks > 1 && c->E > 0 && count >= 2 * c->pipe_chunks) {
        int rc;
        if (!jacobian_path_ok(c, 1))
            return fail(c, SOAP_EINVAL, "basis too large for the on-chip memory of the Jacobian kernels");
        if ((rc = check_ctx_device(c)) != SOAP_OK) return rc;
        return run_derivatives_pipelined(c, first, count, c->pipe_chunks, desc_dev, jac_edge_dev, jac_self_dev,
                                         stream);
    }
    int rc = run_density(c, 1, first, count, desc_dev, nullptr, jac_self_dev, nullptr, scratch, stream, timed);
    if (rc != SOAP_OK) return rc;
    if (c->E == 0) return SOAP_OK;
    SegTimer timer(c, 2, to_stream(stream), timed);
    hipError_t e = launch_jacobian(c->P, rows_of(c, first, count), c->pos, c->built_f64, c->ar64, c->jac_cfg,
                                   scratch ? scratch : c->b_cscratch.p, jac_edge_dev, to_stream(stream));
    if (e != hipSuccess) return hip_fail(c, e, "Jacobian kernel");
    timer.done();
    return SOAP_OK;
}

int soap_derivatives(soap_ctx *c, void *desc_dev, void *jac_edge_dev, void *jac_self_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    if (!desc_dev || !jac_self_dev || (!jac_edge_dev && c->E > 0))
        return fail(c, SOAP_EINVAL, "output pointer is NULL");
    if (!c->have_rows) return fail(c, SOAP_ESTATE, "no neighbour list: call soap_build_neighbors first");
    return run_derivatives(c, 0, c->nc, desc_dev, jac_edge_dev, jac_self_dev, nullptr, stream);
}

int soap_compute_batch(soap_ctx *c, int64_t first, int64_t count, void *desc_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    int rc = check_batch(c, first, count);
    if (rc != SOAP_OK) return rc;
    if (!desc_dev && count > 0) return fail(c, SOAP_EINVAL, "desc_dev is NULL");
    if (count == 0) return SOAP_OK;
    return run_density(c, 0, first, count, desc_dev, nullptr, nullptr, nullptr, nullptr, stream);
}

int soap_derivatives_batch(soap_ctx *c, int64_t first, int64_t count, void *desc_dev, void *jac_edge_dev,
                           void *jac_self_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    int rc = check_batch(c, first, count);
    if (rc != SOAP_OK) return rc;
    if (count > 0 && (!desc_dev || !jac_self_dev)) return fail(c, SOAP_EINVAL, "output pointer is NULL");
    // a NULL jac_edge_dev is allowed only for a batch without edges
    if (!jac_edge_dev && count > 0 && c->E > 0) {
        int64_t r[2];
        hipError_t e = hipMemcpy(r, c->b_row.as<int64_t>() + first, 8, hipMemcpyDeviceToHost);
        if (e == hipSuccess) e = hipMemcpy(r + 1, c->b_row.as<int64_t>() + first + count, 8, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(c, e, "soap_derivatives_batch");
        if (r[1] > r[0]) return fail(c, SOAP_EINVAL, "jac_edge_dev is NULL for a batch with edges");
    }
    return run_derivatives(c, first, count, desc_dev, jac_edge_dev, jac_self_dev, nullptr, stream);
}

int soap_derivatives_batch_noalloc(soap_ctx *c, int64_t first, int64_t count, void *desc_dev, void *jac_edge_dev,
                                   void *jac_self_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    int rc = check_batch(c, first, count);
    if (rc != SOAP_OK) return rc;
    if (count > 0 && (!desc_dev || !jac_self_dev || !jac_edge_dev))
        return fail(c, SOAP_EINVAL, "output pointer is NULL");
    const size_t need = align256(scratch_bytes_per_center(c) * (size_t)count) + radial_bytes(c, first, count);
    if (need > (size_t)SOAP_STATIC_SCRATCH_BYTES)
        return fail(c, SOAP_ECAPACITY,
                    "%lld centers need %zu bytes of coefficient scratch%s, above the static %d bytes (at most %lld "
                    "centers per call for this basis)",
                    (long long)count, need, c->P.rbf == 1 ? " and radial factors" : "", SOAP_STATIC_SCRATCH_BYTES,
                    (long long)(SOAP_STATIC_SCRATCH_BYTES / scratch_bytes_per_center(c)));
    if (!c->static_scratch) return fail(c, SOAP_EHIP, "the static scratch of device %d is not available", c->device);
    // the density kernel writes every scratch entry the later kernels read,
    // so nothing needs clearing
    return run_derivatives(c, first, count, desc_dev, jac_edge_dev, jac_self_dev, c->static_scratch, stream,
                           false);
}

int soap_plan_batches(soap_ctx *c, int32_t what, int64_t budget_bytes, int64_t max_batches, int64_t *center_first,
                      int64_t *edge_first, int64_t *n_batches_out) {
    if (!c) return SOAP_EINVAL;
    if (!n_batches_out || budget_bytes <= 0 || (what != SOAP_BATCH_DESCRIPTOR && what != SOAP_BATCH_DERIVATIVES))
        return fail(c, SOAP_EINVAL, "invalid arguments to soap_plan_batches");
    if (!c->have_rows) return fail(c, SOAP_ESTATE, "no neighbour list: call soap_build_neighbors first");
    std::vector<int64_t> row((size_t)c->nc + 1);
    hipError_t e = hipMemcpy(row.data(), c->b_row.p, 8 * row.size(), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(c, e, "soap_plan_batches");
    const size_t elt = c->built_f64 ? 8 : 4;
    const bool jac = what == SOAP_BATCH_DERIVATIVES;
    // per center: descriptor row (+ center block and coefficient scratch);
    // per edge: its neighbour block
    const int64_t per_center = (int64_t)(elt * c->F * (jac ? 4 : 1) + (jac ? scratch_bytes_per_center(c) : 0));
    const int64_t per_edge = (jac ? (int64_t)(elt * 3 * c->Fe) : 0) + (c->P.rbf == 1 ? (int64_t)radial_bytes_per_edge(c->P) : 0);
    int64_t nb = 0, b0 = 0;
    while (b0 < c->nc) {
        int64_t b1 = b0, bytes = 0;
        while (b1 < c->nc) {
            const int64_t add = per_center + per_edge * (row[b1 + 1] - row[b1]);
            if (bytes + add > budget_bytes) break;
            bytes += add;
            ++b1;
        }
        if (b1 == b0)
            return fail(c, SOAP_ECAPACITY, "center %lld alone needs %lld bytes, above the budget of %lld", (long long)b0,
                        (long long)(per_center + per_edge * (row[b0 + 1] - row[b0])), (long long)budget_bytes);
        if (center_first && nb < max_batches) {
            center_first[nb] = b0;
            if (edge_first) edge_first[nb] = row[b0];
        }
        ++nb;
        b0 = b1;
    }
    *n_batches_out = nb;
    if (center_first) {
        if (nb > max_batches)
            return fail(c, SOAP_ECAPACITY, "%lld batches needed, room for %lld", (long long)nb, (long long)max_batches);
        center_first[nb] = c->nc;
        if (edge_first) edge_first[nb] = row[c->nc];
    }
    return SOAP_OK;
}

int soap_scatter_dense(soap_ctx *c, const void *jac_edge_dev, const void *jac_self_dev, void *dense_dev, void *stream) {
    if (!c) return SOAP_EINVAL;
    if (!c->have_rows) return fail(c, SOAP_ESTATE, "no neighbour list: call soap_build_neighbors first");
    if (!jac_self_dev || !dense_dev || (!jac_edge_dev && c->E > 0)) return fail(c, SOAP_EINVAL, "NULL pointer");
    hipStream_t st = to_stream(stream);
    const size_t elt = c->built_f64 ? 8 : 4;
    hipError_t e = hipMemsetAsync(dense_dev, 0, elt * (size_t)c->nc * c->n_atoms * 3 * c->F, st);
    if (e == hipSuccess)
        e = launch_scatter_dense(c->P, rows_of(c), c->built_f64, jac_edge_dev, jac_self_dev, c->d_fmap.as<int32_t>(),
                                 c->built_periodic ? c->b_map_atom.as<int32_t>() : nullptr, dense_dev, st);
    return e == hipSuccess ? SOAP_OK : hip_fail(c, e, "soap_scatter_dense");
}

int soap_timing(soap_ctx *c, double *ms_out, int64_t *count_out, int32_t reset) {
    if (!c || !ms_out) return SOAP_EINVAL;
    double ms[3] = {0, 0, 0};
    int64_t cnt[3] = {0, 0, 0};
    for (auto &r : c->recs) {
        hipError_t e = hipEventSynchronize(r.b);
        float t = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&t, r.a, r.b);
        if (e != hipSuccess) return hip_fail(c, e, "soap_timing");
        ms[r.seg] += t;
        cnt[r.seg] += 1;
    }
    for (int k = 0; k < 3; ++k) {
        ms_out[k] = ms[k];
        if (count_out) count_out[k] = cnt[k];
    }
    if (reset) {
        for (auto &r : c->recs) {
            c->pool.push_back(r.a);
            c->pool.push_back(r.b);
        }
        c->recs.clear();
    }
    return SOAP_OK;
}

const char *soap_last_error(const soap_ctx *c) { return c ? c->err.c_str() : g_create_error.c_str(); }

void soap_destroy(soap_ctx *c) {
    if (!c) return;
    (void)hipDeviceSynchronize();
    for (DevBuf *b : {&c->d_const, &c->d_dtab, &c->d_fmap, &c->d_lut, &c->b_zero, &c->b_bstart, &c->b_acell,
                      &c->b_srec, &c->b_sspec, &c->b_deg, &c->b_slots, &c->b_scan, &c->b_spec, &c->b_row, &c->b_cols,
                      &c->b_cscratch, &c->b_avg, &c->b_avg_part, &c->b_img_lohi, &c->b_img_cnt, &c->b_img_start,
                      &c->b_pos_ext, &c->b_Z_ext, &c->b_map_atom, &c->b_map_img, &c->b_iota})
        b->release();
    if (c->h_flags) (void)hipHostFree(c->h_flags);
    if (c->h_rec) (void)hipHostFree(c->h_rec);
    if (c->h_rowp) (void)hipHostFree(c->h_rowp);
    for (hipEvent_t e : c->pipe_ev) (void)hipEventDestroy(e);
    if (c->aux) (void)hipStreamDestroy(c->aux);
    for (auto &r : c->recs) {
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
    }
    for (hipEvent_t e : c->pool) (void)hipEventDestroy(e);
    delete c;
}

} // extern "C"
