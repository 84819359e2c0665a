// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace soap {

constexpr int NMAX = 16;       // largest n_max
constexpr int LMAX = 14;       // largest l_max
constexpr int LT_MAX = LMAX + 2;
constexpr int MAX_GROUPS = LMAX + 1;
constexpr int MAX_DEGREE = 2048;

// Everything the descriptor kernels need about the basis; passed by value.
struct Params {
    int S, n, lmax, L, rbf, Q; // L = (lmax+1)^2; rbf 0 GTO, 1 polynomial, 2 polynomial (Laplace form),
                               // 3 GTO with the compensated float64 evaluation
    int F, Fe, nq_full;        // features, edge features, (mu,nu,n,n') combinations
    double sigma, inv_s2;      // 1 / sigma^2
    double rc, inv_rc2;        // cutoff radius, 2 / rc
    double s2, hs2;            // sigma^2, sigma^2 / 2
    const double *betaC;       // GTO [l][n][k]
    const double *betaCa;      // GTO [l][n][k]
    const double *aprime;      // GTO [l][k]
    const double *betaC_lo, *aprime_lo; // GTO: rounding remainders of betaC and aprime (compensated path)
    const double *G;           // polynomial [n][Q], includes 4 pi
    const double *rq;          // polynomial [Q]
    const double *WN;          // polynomial, Laplace form [n][n+3][4]: Chebyshev series of P_n0..P_n3 on [0, rc]
    const double2 *rad;        // polynomial quadrature: radial factors (B_nl, Bh_nl) of the call's edges,
                               // [edge - rad_e0][n][l] (k_radial)
    int64_t rad_e0;            // structure index of the first edge of rad
    const double *c0;          // on-site term [n]
    const double *e2t;         // GTO: [64][2] 2^(j/64) as (value, remainder) (soap_exp2_table64)
    const double *Nt;          // [lmax+2][lmax+2] N_lm (2m-1)!! / (l-m)! (division-free recurrence)
    const double *gcoef;       // [(l, m >= 0)][4] gradient identities of the harmonics (cA, cB, cC, l | m << 8)
    const uint32_t *dtab;      // [tri_lw] diagonal-pair slots: (n lw + l) | (n' lw + l) << 16, n' >= n
    int tri_lw;                // n (n + 1) / 2 * (l_max + 1)
    int n_groups;              // l-groups of the density kernel
    int lgrp[MAX_GROUPS + 1];  // group g covers l in [lgrp[g], lgrp[g+1])
};

// Neighbour rows of the current structure, or of a range of its centers:
// the range's rows row_ptr[0..nc] are a slice of the structure's CSR
// offsets, and center ci of the range is center c_base + ci of the
// structure (its row, its atom index).  Edge outputs are indexed from the
// first edge of the output batch: edge e of the structure is entry
// e - *e_origin (a launch may cover part of a batch, its edges then land
// after the earlier part's).
struct Rows {
    int64_t n_atoms, nc;
    int64_t c_base;           // structure index of the range's first center
    const int32_t *centers;   // [nc] atom of each center of the range; NULL = c_base + ci
    const uint8_t *spec;      // species index per atom
    const int64_t *row_ptr;   // [nc+1]
    const int32_t *cols;      // [E] (indexed by structure edge)
    const int64_t *e_origin;  // row offset of the output batch's first center
};

// Density work counters: one 64-bit counter per l-group, zeroed at the
// neighbour build and never reset in between.  Every density launch advances
// the counters of the groups it runs by exactly n_c (its centers but the
// static first ones, plus one empty fetch per workgroup), so each group keeps
// its own count of the increments taken so far; a launch planning fewer
// groups leaves the other counters, and their counts, untouched.
struct WorkBase {
    uint64_t b[MAX_GROUPS];
};

// ---- neighbour search (neighbors.hip) ----
constexpr int TCAP = 128; // neighbours per center kept by the collecting pass (longer rows: second pass)

struct NbrWork {
    int64_t H;                   // hash buckets (power of two)
    void *zero;                  // zeroed at every build: flags, work counters, bucket counts and fills
    size_t zero_bytes;
    int32_t *flags;              // [4] error bits, max degree, rows above TCAP, -; then int64 total degree
    unsigned long long *work;    // [MAX_GROUPS] density work counters
    int32_t *bucket_count;       // [H]
    int32_t *bucket_fill;        // [H]
    int32_t *bucket_start;       // [H+1]
    int4 *atom_cell;             // [n_atoms] cx, cy, cz, bucket
    void *sorted_rec;            // [n_atoms] float4 / double4: position, atom index
    uint8_t *sorted_spec;        // [n_atoms]
    int32_t *deg;                // [nc]
    int32_t *slots;              // [nc][TCAP] ordered rows of up to TCAP neighbours
    int64_t *scan_tmp;           // block sums
};
// bytes of the zeroed block for H buckets, and the offsets of its parts
constexpr size_t NBR_FLAGS_BYTES = 64, NBR_WORK_BYTES = 8 * (MAX_GROUPS + 1);
inline size_t nbr_zero_bytes(int64_t H) { return NBR_FLAGS_BYTES + NBR_WORK_BYTES + 8 * (size_t)H; }

// Periodic structures: the neighbour search runs over the atoms plus the
// images of them that can lie within r_cut of an atom (an extended
// structure); the kernels then see each image as an atom.
struct PeriodicCell {
    double M[9];   // lattice vectors a, b, c as rows
    double B[9];   // M^-1: fractional coordinates f = r B (r as a row vector)
    double eps[3]; // r_cut over the interplanar spacing, padded; 0 for open directions
    int pbc[3];
};
// fractional bounds (lo[3], hi[3]) of the atoms, then per atom the number of
// its images n != 0 whose fractional coordinates stay within [lo - eps,
// hi + eps] along every periodic direction (open directions: n = 0)
hipError_t periodic_count(int64_t n, const void *pos, bool pos64, const PeriodicCell &C, double *lohi, int32_t *cnt,
                          hipStream_t st);
// extended structure: the atoms, then their images (atom-major, images in
// lexicographic (n_a, n_b, n_c) order) at r + ((n_a a + n_b b) + n_c c)
// evaluated in float64 and stored at the position precision; atom index and
// image of every entry
hipError_t periodic_fill(int64_t n, const void *pos, bool pos64, const int32_t *Z, const PeriodicCell &C,
                         const double *lohi, const int64_t *start, void *pos_ext, int32_t *Z_ext, int32_t *map_atom,
                         int32_t *map_img, hipStream_t st);
// int32 counts -> int64 exclusive offsets (out has n+1); the total also to *total_copy
hipError_t nbr_exclusive_scan(int64_t n, const int32_t *in, int64_t *out, int64_t *tmp, int64_t *total_copy,
                              hipStream_t st);
// out[k] = k
hipError_t fill_iota(int64_t n, int32_t *out, hipStream_t st);
// out[e] = map[cols[e]] (atom of each edge), and img_out[e][3] = map_img[cols[e]] if given
hipError_t map_edges(int64_t E, const int32_t *cols, const int32_t *map, const int32_t *map_img, int32_t *out,
                     int32_t *img_out, hipStream_t st);

// center_bound: centers must index atoms below it (the atoms of an extended
// periodic structure that are not images).  rec (may be NULL): device address
// of a host-visible record of four int64, error bits | largest degree << 32,
// rows above TCAP, total degree, then seq (stored last, with a system-scope
// release); *rec_written says whether this launch writes it (one-workgroup
// scan of the degrees only, n_centers <= 16384)
hipError_t nbr_phase1(const NbrWork &w, int64_t n_atoms, int64_t center_bound, const void *pos, bool pos64,
                      const int32_t *Z, const int8_t *lut, uint8_t *spec, int64_t nc, const int32_t *centers,
                      double r_cut, int64_t *row_ptr, hipStream_t st, int64_t *rec, int64_t seq,
                      bool *rec_written);
// rows of up to TCAP neighbours from their slots into cols (cap entries);
// writes nothing if the rows need more than cap, so it may run before the
// host has read the total
hipError_t nbr_pack(const NbrWork &w, int64_t nc, const int64_t *row_ptr, int32_t *cols, int64_t cap,
                    hipStream_t st);
// long_rows: some row is longer than TCAP (flags[2] > 0); packed: nbr_pack
// has already written the short rows
hipError_t nbr_phase2(const NbrWork &w, int64_t n_atoms, const void *pos, bool pos64, int64_t nc,
                      const int32_t *centers, double r_cut, const int64_t *row_ptr, bool long_rows, bool packed,
                      int32_t *cols, int64_t cap, hipStream_t st);

// ---- descriptor kernels (soap_kernels.hip) ----
struct DensityLaunch {
    int W;           // edges per wave iteration
    size_t lds;      // dynamic LDS bytes
    int blocks;      // persistent workgroups per l-group
    bool hi;         // the variant compiled for three waves per SIMD (see density_has_high)
};
struct DescLaunch {
    int W;          // edges per chunk (0: the descriptor path uses k_density)
    int ql, na, sr; // tasks per thread, radial size, species slots
    size_t lds;
    int blocks; // resident workgroups (persistent launch)
};
struct DjacLaunch {
    int W;          // edges per chunk (0: the Jacobian path uses k_density)
    int qt, na, sr; // tasks per thread, radial size, species slots
    size_t lds;
    int blocks;     // resident workgroups (persistent launch)
};
struct DjsLaunch {
    int W;          // edges per chunk (0: not used)
    int qt, na;     // tasks per thread, radial size (GTO)
    size_t lds;
    int blocks;     // resident workgroups (persistent launch)
};
struct JacLaunch {
    int W;          // edges per wave tile (at most jacobian_max_w())
    size_t lds;
};

// st64: float64 staging (float64 outputs, or float64 arithmetic with float32 outputs)
size_t density_lds_bytes(const Params &P, int jac, int lg0, int lg1, int W, bool st64);
// f64: float64 positions and outputs; ar64: float64 arithmetic with float32 outputs
int density_blocks_per_cu(bool f64, bool ar64, int mode, int rbf, bool hi, size_t lds); // mode as launch_density
bool density_has_high(int mode, int rbf); // a three-waves-per-SIMD variant exists
constexpr int DENSITY_KE = 8; // coefficient entries per lane in k_density: n * Lg <= 512
size_t jacobian_lds_bytes(const Params &P, int W, bool at64); // at64: float64 assembly
int jacobian_max_w();
// resident workgroups per CU (0 if it does not fit)
int jacobian_blocks_per_cu(bool f64, bool ar64, int rbf, int n, int lw, size_t lds);
// float32 Jacobian kernels for fixed (n_max, l_max + 1); NULL if not compiled
const void *jacobian_fixed_0(int n, int lw);
const void *jacobian_fixed_1(int n, int lw);
const void *jacobian_fixed_2(int n, int lw);
hipError_t set_lds_limits();

// desc (may be NULL; descriptor path), c_out (may be NULL, dtype), c_scratch (jac only, float64,
// [center][c, Dx, Dy, Dz][lm][species n])
// work: per-group counters (WorkBase); *epoch holds each group's count of
// the increments made since they were zeroed (advanced here for the groups
// the launch runs).
// mode 0: descriptor (desc, c_out may be NULL); 1: descriptor + Jacobian (desc,
// jself, c_scratch); 2: coefficient Jacobian (c_out, jself = [n_c][3][S][n][L],
// jc_edge = [E][3][n][L])
hipError_t launch_density(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, int mode,
                          const DensityLaunch &cfg, unsigned long long *work, WorkBase *epoch, void *desc, void *c_out,
                          void *jself, void *c_scratch, void *jc_edge, hipStream_t st);
// power spectrum and center block from the coefficient scratch (Jacobian
// path): whole rows (rows = true: c and one component of D for every l in
// LDS), else l-groups of the output kernel, each sized to its LDS budget
struct OutPlan {
    bool rows;
    bool st64; // whole rows: c and D staged in float64 (else float32, the mixed mode)
    int n_groups;
    int lgrp[MAX_GROUPS + 1];
    size_t lds;
};
// allow_rows = false keeps the l-group kernel; 0, or -1 if one l does not fit
int plan_outputs(const Params &P, bool f64, bool st64, bool allow_rows, OutPlan *O);
hipError_t launch_outputs(const Params &P, const OutPlan &O, int64_t nc, bool f64, const void *scratch, void *desc,
                          void *jself, hipStream_t st);
// one-wave-per-center descriptor kernel (GTO): the shape of its accumulators
// (false if the basis has none), LDS bytes for W edges per chunk, resident
// workgroups per CU, launch (desc and c_out may each be NULL)
bool desc_shape(const Params &P, int *ql, int *na, int *sr);
size_t desc_lds_bytes(const Params &P, int W, bool st64);
int desc_blocks_per_cu(bool f64, bool ar64, int ql, int na, int sr, size_t lds);
hipError_t launch_desc(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, const DescLaunch &cfg,
                       void *desc, void *c_out, hipStream_t st);
// one-workgroup-per-center density step of the Jacobian path (GTO): shape,
// LDS bytes, resident workgroups per CU, launch (writes desc, jself and the
// coefficients for k_jacobian)
bool djac_shape(const Params &P, int *qt, int *na, int *sr);
size_t djac_lds_bytes(const Params &P, int W, bool st64);
// the polynomial quadrature's radial pass: (B_nl, Bh_nl) of every edge of the
// rows, at out[edge - e_base][n][l]
size_t radial_bytes_per_edge(const Params &P);
hipError_t launch_radial(const Params &P, const Rows &R, const void *pos, bool f64, int64_t e_base, void *out,
                         hipStream_t st);
int djac_blocks_per_cu(bool f64, bool ar64, int qt, int na, int sr, size_t lds);
hipError_t launch_djac(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, const DjacLaunch &cfg,
                       void *desc, void *jself, void *c_scratch, hipStream_t st);
hipError_t launch_jacobian(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, const JacLaunch &cfg,
                           const void *c_scratch, void *jedge, hipStream_t st);
// density step of the Jacobian path with the coefficients streamed to the
// scratch (k_djs, density_streamed.hip): GTO and polynomial quadrature bases
// of at most four (radial pair, lm) tasks per thread
bool djs_shape(const Params &P, int *qt, int *na);
size_t djs_lds_bytes(const Params &P, int W, bool st64);
int djs_blocks_per_cu(bool f64, bool ar64, int rbf, int qt, int na, size_t lds);
hipError_t launch_djs(const Params &P, const Rows &R, const void *pos, bool f64, bool ar64, const DjsLaunch &cfg,
                      void *c_scratch, hipStream_t st);
hipError_t djs_set_lds_limit(int lim);
// column means of a row-major (rows x cols) array of the output type, in
// float64: part[AVG_CHUNKS][cols] partial sums, then mean[cols] (float64)
// and, if out is not NULL, out[cols] at the output type
constexpr int AVG_CHUNKS = 256;
hipError_t launch_column_mean(const void *in, bool f64, int64_t rows, int64_t cols, double *part, void *out,
                              double *mean, hipStream_t st);
// power spectrum of one coefficient set c[S][n][L] (float64) into out[F]
hipError_t launch_power_single(const Params &P, bool f64, const double *c, void *out, hipStream_t st);
// atom_of (may be NULL = identity): atom of every (extended) neighbour index;
// blocks of several images of one atom are summed
hipError_t launch_scatter_dense(const Params &P, const Rows &R, bool f64, const void *jedge, const void *jself,
                                const int32_t *fmap, const int32_t *atom_of, void *dense, hipStream_t st);

} // namespace soap
