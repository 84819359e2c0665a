/*
 * soap.h -- C ABI of the MI355X SOAP descriptor + analytic Jacobian library.
 *
 * What is computed (arXiv 2609.05709, Sec. 2):
 *   - species-resolved Gaussian-smeared neighbour densities, Eq. (density):
 *     every atom j != i with |r_j - r_i| < r_cut contributes an unnormalised
 *     Gaussian of width sigma to the density of its species; the center atom
 *     itself is included in its own species' density through the
 *     position-independent l = 0 on-site term (Sec. 2.2, last term of
 *     Eq. (gto-coefficients); Sec. 2.3 for the polynomial basis);
 *   - expansion coefficients c^mu_nlm, Eq. (projection), in real spherical
 *     harmonics and either the GTO radial basis (Sec. 2.2, Eqs. (gto-basis),
 *     (gto-alphas), (gto-lowdin), closed form Eq. (gto-coefficients)) or the
 *     polynomial radial basis (Sec. 2.3, Eqs. (poly-basis)-(poly-overlap),
 *     coefficients Eq. (poly-coefficients-exact) with the radial integral
 *     Eq. (poly-radial-integral) evaluated by a fixed Gauss-Legendre rule on
 *     [0, r_cut], Sec. 3.1);
 *   - the power spectrum p^{mu nu}_{n n' l}, Eq. (powerspectrum);
 *   - its Cartesian Jacobian by the product rule, Eq. (powerspectrum-derivative),
 *     with d c / d r_j from Eq. (gto-derivative) or
 *     Eq. (poly-cartesian-derivative), and the center's own block from
 *     translational invariance (end of Sec. 2.1).
 *
 * Feature order (Sec. 3.1): species pairs (mu, nu) with mu <= nu over the
 * species sorted by ascending Z, then n, then n' (n' >= n when mu == nu, all
 * n' when mu < nu), then l innermost.  F = (l_max+1) * S n (S n + 1) / 2.
 *
 * Conventions shared by all entry points:
 *   - Units: angstrom.
 *   - Device pointers ("_dev") are HIP device memory on the context's device,
 *     owned by the caller; they must stay valid until the work enqueued on
 *     `stream` has completed.  `stream` is a hipStream_t (NULL = the default
 *     stream).  All calls are asynchronous on `stream` unless stated.
 *   - dtype (option "dtype"): SOAP_FP32 (default) = float32 positions and
 *     outputs; SOAP_FP64 = float64 positions and outputs.  The float64 mode
 *     computes everything in float64.  The float32 mode forms the edge
 *     geometry, radial sums, projection sums, power spectrum, center block
 *     and the Jacobian's precontraction with float64 products and sums, but
 *     rounds operands to float32 where they are staged on chip: the
 *     harmonics and radial factors before the projection's products, the
 *     coefficients before the Jacobian's precontraction (and c, D before
 *     the output kernel's products where that kernel runs), and the
 *     precontraction results and radial factors before the Jacobian's final
 *     two-term assembly, which then runs in float32.  Option "arith" = SOAP_ARITH_FP64 keeps float64
 *     through every step in the float32 mode too and rounds only the
 *     stored outputs (the paper's choice, Sec. 3.1: float64 internal
 *     arithmetic, outputs cast at the end).
 *   - Every function returns SOAP_OK or a negative status; on error nothing
 *     is enqueued and soap_last_error() describes the cause.  No function
 *     aborts or throws across this interface.
 *   - A context is not thread-safe; use one context per host thread.
 */
#ifndef SOAP_MI355X_H
#define SOAP_MI355X_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct soap_ctx soap_ctx;

#define SOAP_OK 0
#define SOAP_EINVAL (-1)    /* argument out of range */
#define SOAP_ESPECIES (-2)  /* an atomic number is not in the species list */
#define SOAP_ENOMEM (-3)    /* device or host allocation failed */
#define SOAP_EHIP (-4)      /* a HIP runtime call failed */
#define SOAP_ECAPACITY (-5) /* a neighbour row exceeds the supported degree */
#define SOAP_ESTATE (-6)    /* call order violated (e.g. compute before build) */

#define SOAP_RBF_GTO 0
#define SOAP_RBF_POLYNOMIAL 1         /* exact radial integral, Gauss-Legendre quadrature */
#define SOAP_RBF_POLYNOMIAL_LAPLACE 2 /* same basis, Laplace (steepest-descent) form to O(sigma^2) */

#define SOAP_FP32 0
#define SOAP_FP64 1

/* averaging modes of soap_compute_averaged (Sec. 3, the density-averaged variants) */
#define SOAP_AVERAGE_INNER 1
#define SOAP_AVERAGE_OUTER 2

/* Largest neighbour count per center the neighbour builder accepts. */
#define SOAP_MAX_DEGREE 2048

/* internal arithmetic of the float32 mode (option "arith") */
#define SOAP_ARITH_MIXED 0 /* float32 staging and final assembly (default) */
#define SOAP_ARITH_FP64 1  /* float64 throughout, outputs rounded at the store */

/* bytes of the fixed device scratch of soap_derivatives_batch_noalloc */
#define SOAP_STATIC_SCRATCH_BYTES (64 * 1024 * 1024)

/* outputs a center batch plan is sized for (soap_plan_batches) */
#define SOAP_BATCH_DESCRIPTOR 0
#define SOAP_BATCH_DERIVATIVES 1

/*
 * Create a context on the current HIP device.  Arguments follow the paper's
 * problem statement (Sec. 3.1: r_cut, n_max, l_max, sigma, rbf, species).
 *   species_Z : n_species distinct atomic numbers (1..127), any order (host).
 *   r_cut     : cutoff radius; GTO requires r_cut > 1 (the widths of
 *               Eq. (gto-alphas) place the first primitive at 1 A).
 *   n_max     : 1..16 radial functions;  l_max: 0..14;  sigma > 0.
 *   rbf       : SOAP_RBF_GTO, SOAP_RBF_POLYNOMIAL (Eq. poly-coefficients-exact,
 *               the radial integral by Gauss-Legendre quadrature) or
 *               SOAP_RBF_POLYNOMIAL_LAPLACE (the same basis with the radial
 *               factors of Eqs. poly-coefficients and poly-radial-derivative,
 *               the Laplace form to first order in sigma^2: an approximation
 *               for sigma small against the distances r and r_cut - r; the
 *               on-site term of a center, and of a neighbour at distance 0,
 *               stays the quadrature's).
 * Basis constants (Loewdin coefficients, quadrature tables) are computed here
 * on the host in 113-bit floating point and uploaded once.  The kernels keep
 * a center's coefficients on chip: a basis whose descriptor path does not
 * fit is rejected here (SOAP_EINVAL); one that fits the descriptor path but
 * not a Jacobian path (large S n_max, e.g. 16 species at n_max 8, l_max 6)
 * is accepted, and soap_derivatives / soap_coefficient_derivatives then
 * return SOAP_EINVAL.
 * Errors: SOAP_EINVAL, SOAP_ENOMEM, SOAP_EHIP.  *out is NULL on error.
 */
int soap_create(const int32_t *species_Z, int32_t n_species, double r_cut, int32_t n_max, int32_t l_max,
                double sigma, int32_t rbf, soap_ctx **out);

/*
 * Set an option of the constructor (Sec. 3.1 lists the constructor's
 * arguments: the output dtype, the quadrature order of the polynomial
 * radial integral, and the per-segment profiler).  Keys:
 *   "dtype"  : SOAP_FP32 or SOAP_FP64 (default SOAP_FP32);
 *   "arith"  : SOAP_ARITH_MIXED (default) or SOAP_ARITH_FP64, the internal
 *              arithmetic of the float32 mode (see dtype above; the float64
 *              mode is float64 throughout either way);
 *   "quad_n" : Gauss-Legendre order for the polynomial basis, 8..256
 *              (default 64; Sec. 3.1, the fixed Gauss-Legendre rule on
 *              [0, r_cut]); rebuilds the quadrature table;
 *   "timing" : 1 = record HIP events around every segment of later calls
 *              (see soap_timing), 0 = off (default);
 *   "desc_tile": kernel choice of the GTO descriptor path (a tuning knob;
 *              results are identical either way up to rounding order):
 *              0 = automatic (default), -1 = the density kernel shared with
 *              the Jacobian path, 16 / 32 / 64 = the descriptor kernel
 *              whose waves each own whole centers, with at most that many
 *              edges per chunk (the widest that fits on chip);
 *   "jac_tile" : edges per matrix-core tile of the edge Jacobian kernel (a
 *              tuning knob, results identical up to rounding order): 0 =
 *              automatic (default: the most resident workgroups, then the
 *              widest tile), 1..4 = that width (a width whose LDS does not
 *              fit leaves the Jacobian path without a plan: the calls that
 *              need it return SOAP_EINVAL, as for a basis too large);
 *   "djac_tile": kernel choice of the density step of the GTO Jacobian path
 *              (a tuning knob, results identical up to rounding order):
 *              0 = automatic (default), -1 = the shared density kernel and
 *              the output kernel, 32 / 64 = the kernel that gives each
 *              center a workgroup, with at most that many edges per chunk;
 *   "djs_tile" : kernel choice of the density step of the Jacobian path for
 *              the GTO bases outside "djac_tile"'s kernel and the polynomial
 *              quadrature bases (a tuning knob, results identical up to
 *              rounding order): 0 = automatic (default), -1 = the shared
 *              density kernel, 16 / 32 / 64 = the kernel that gives each
 *              center a workgroup and streams its coefficients to the
 *              scratch, with at most that many edges per chunk (then the
 *              output kernel writes the descriptor and center blocks);
 *   "out_rows" : 1 (default) = the output kernel of the Jacobian path
 *              writes whole rows where c and one component of D fit on
 *              chip, 0 = always in l-groups (a tuning knob, results
 *              identical);
 *   "batch_centers": >= 0 (default 0 = one batch): soap_derivatives
 *              computes its centers in consecutive batches of at most that
 *              many, one after another on the stream, so that the library's
 *              scratch (the coefficients c, D of the Jacobian path:
 *              4 S n_max (l_max+1)^2 values per center, float32 in the mixed
 *              arithmetic and float64 otherwise, and the polynomial
 *              quadrature's radial factors) is sized for one batch (Sec. 3.3:
 *              center batches bound the memory of one call); the outputs are
 *              the same arrays, bit for bit, as in one batch;
 *   "pipeline" : 1..16 (default 1): soap_derivatives splits its centers
 *              into that many chunks and overlaps each chunk's edge
 *              Jacobian (a second stream) with the next chunk's density
 *              step;
 *   "pipeline_density_wg": 0..16 (default 0 = no cap), workgroups per
 *              CU of the density kernel while pipelined.
 * Options take effect for calls made after this one; changing "dtype"
 * discards the neighbour list.  Errors: SOAP_EINVAL.
 */
int soap_set_option(soap_ctx *ctx, const char *key, int64_t value);

/*
 * Read an option (any key of soap_set_option) or a planning decision of the
 * context into *value (host):
 *   "device"                  : the HIP device ordinal the context was created
 *                               on (the current device at soap_create: the
 *                               device argument of the paper's constructor,
 *                               Sec. 3.1); every call must run with it current;
 *   "descriptor_kernel"       : 1 if soap_compute / soap_coefficients run the
 *                               descriptor kernel that gives each center a
 *                               workgroup, 0 if the shared density kernel;
 *   "jacobian_density_kernel" : the density step of soap_derivatives: 1 the
 *                               kernel that gives each center a workgroup and
 *                               writes its outputs ("djac_tile"), 2 the one
 *                               that streams the coefficients to the scratch
 *                               ("djs_tile"), 0 the shared density kernel;
 *   "output_kernel_rows"      : 1 if the output kernel of the Jacobian path
 *                               (run when the shared density kernel splits
 *                               l into groups, and after the streaming
 *                               density kernel) writes whole rows, 0 if it
 *                               works in l-groups;
 *   "jacobian_l_groups"       : l-groups of the shared density kernel on the
 *                               Jacobian path (above 1, the output kernel
 *                               runs after it);
 *   "jacobian_density_tile", "jacobian_density_lds": edges per chunk and
 *                               LDS bytes per workgroup of the density step
 *                               of the Jacobian path;
 *   "jacobian_tile", "jacobian_lds": edges per wave tile and LDS bytes per
 *                               workgroup of the edge Jacobian kernel;
 *   "output_lds"              : LDS bytes per workgroup of the output kernel.
 * Errors: SOAP_EINVAL (NULL argument, unknown key).
 */
int soap_get_option(const soap_ctx *ctx, const char *key, int64_t *value);

/* Number of descriptor features F (see feature order above); -1 if ctx is NULL. */
int64_t soap_num_features(const soap_ctx *ctx);

/*
 * Number of features F_e a neighbour block can touch: the features whose
 * species pair contains the neighbour's species,
 * F_e = (l_max+1) (n(n+1)/2 + (S-1) n^2), the same for every species.
 */
int64_t soap_num_edge_features(const soap_ctx *ctx);

/*
 * Feature labels: out[5*f + {0..4}] = (mu, nu, n, n', l) for f < F (host
 * buffer of 5F int32).  Species indices refer to the sorted species list.
 */
int soap_feature_labels(const soap_ctx *ctx, int32_t *out);

/*
 * For species index s (0..S-1 in sorted order), write to host buffer out[F_e]
 * the full feature index of each compressed slot of a neighbour block.
 */
int soap_feature_map(const soap_ctx *ctx, int32_t species_index, int32_t *out);

/*
 * Build the neighbour list of a structure (the neighbour-search step of
 * Sec. 3.1, here a hashed cell list on the device):
 *   N(i) = { j != i : |r_j - r_i|^2 < r_cut^2 }, the squared distance formed
 *   in float64 as ((dx*dx + dy*dy) + dz*dz), dx = (double)x_j - (double)x_i,
 *   without fused multiply-adds.  Coincident atoms (distance 0) are kept as
 *   edges; they add their on-site term to the density and have a zero
 *   Jacobian block.
 *   n_atoms     : >= 1.
 *   pos_dev     : n_atoms x 3 positions (AoS), float32 or float64 per "dtype".
 *   Z_dev       : n_atoms atomic numbers (int32).
 *   n_centers   : number of centers (>= 1);
 *   centers_dev : n_centers atom indices (int32), or NULL for all atoms in
 *                 order (then n_centers must equal n_atoms).
 *   n_edges_out : host; receives E = sum_i |N(i)|.
 * Rows are ordered by species index (sorted Z), then by ascending atom
 * index.  The context keeps the rows and the input pointers for the calls
 * below.  This call waits once for the device (to read E and the results of
 * the device-side checks): for up to 16384 centers it waits for a record
 * that the search writes to pinned host memory as soon as E is known, so the
 * last rows may still be in flight on `stream` when it returns (work queued
 * on `stream` afterwards sees them); with more centers, or when the stream
 * has not reached the search within 20 ms, it synchronises `stream`.
 * Errors: SOAP_EINVAL, SOAP_ESPECIES (unknown Z),
 * SOAP_ECAPACITY (a row longer than SOAP_MAX_DEGREE), SOAP_ENOMEM, SOAP_EHIP.
 *
 * With a periodic cell (soap_set_cell) the edges run over periodic images:
 * (i -> j, n) for every atom j and integer image n = (n_a, n_b, n_c) along
 * the periodic directions with (j, n) != (i, 0) and the image position
 *   r_j + s(n),  s(n) = ((n_a a + n_b b) + n_c c) evaluated in float64,
 * rounded to float32 in SOAP_FP32 mode, within the cutoff of r_i by the
 * test above.  Several images of one atom, and images of the center
 * itself, are separate edges.  The images that can reach an atom are
 * copied into a context-owned extended structure (positions are not read
 * after this call); this takes one more synchronisation of `stream`.  Rows
 * are ordered by species, then atom, then image (the order of the extended
 * structure).
 */
int soap_build_neighbors(soap_ctx *ctx, int64_t n_atoms, const void *pos_dev, const int32_t *Z_dev,
                         int64_t n_centers, const int32_t *centers_dev, int64_t *n_edges_out, void *stream);

/*
 * Copy the neighbour rows of the last build: row_ptr_dev[n_centers+1]
 * (int64, CSR offsets into the edge list) and cols_dev[E] (int32 atom
 * indices).  Either pointer may be NULL.  Errors: SOAP_ESTATE, SOAP_EHIP.
 */
int soap_get_neighbors(soap_ctx *ctx, int64_t *row_ptr_dev, int32_t *cols_dev, void *stream);

/*
 * Periodic cell for the following soap_build_neighbors calls (the periodic
 * flag of the paper's constructor, Sec. 3): cell[9] (host) holds the lattice
 * vectors a, b, c as rows (angstrom), pbc[3] (host) is non-zero for each
 * periodic direction.  Positions may lie anywhere; images are generated
 * around the atoms as given.  cell = NULL returns to open boundaries (the
 * default).  Discards the neighbour list.  Errors: SOAP_EINVAL (NULL pbc,
 * degenerate cell).
 */
int soap_set_cell(soap_ctx *ctx, const double *cell, const int32_t *pbc);

/*
 * Image index n = (n_a, n_b, n_c) of every edge of the last build:
 * img_dev[E][3] (int32, device); all zero without a periodic cell.
 * Errors: SOAP_EINVAL, SOAP_ESTATE, SOAP_EHIP.
 */
int soap_get_neighbor_images(soap_ctx *ctx, int32_t *img_dev, void *stream);

/*
 * Descriptor: desc_dev[n_centers][F] (dtype), Eq. (powerspectrum).
 * Errors: SOAP_ESTATE (no neighbour list), SOAP_ENOMEM, SOAP_EHIP.
 */
int soap_compute(soap_ctx *ctx, void *desc_dev, void *stream);

/*
 * Expansion coefficients c^mu_nlm (the raw coefficients of Eq. (projection),
 * the "cc" quantity of Sec. 3.1): c_dev[n_centers][S][n_max][(l_max+1)^2]
 * (dtype), index lm = l*l + l + m; real harmonics with m > 0 ~ cos(m phi),
 * m < 0 ~ sin(|m| phi), no Condon-Shortley phase.
 */
int soap_coefficients(soap_ctx *ctx, void *c_dev, void *stream);

/*
 * Coefficients and their Jacobian (the "cc" mode of Sec. 3, whose kernel
 * stores the edge gradient of the coefficients directly):
 *   c_dev       [n_centers][S][n_max][L]  c^mu_nlm(i), as soap_coefficients
 *                                         (L = (l_max+1)^2, index l*l + l + m);
 *   jc_edge_dev [E][3][n_max][L]          d c^{species(j)}_nlm(i) / d r_j for
 *                                         the e-th edge (i, j) of the neighbour
 *                                         rows: B^_nl r S_lm + B_nl grad S_lm
 *                                         (Eqs. (gto-derivative),
 *                                         (poly-cartesian-derivative)); the
 *                                         other species blocks of c(i) do not
 *                                         depend on r_j and are not stored;
 *   jc_self_dev [n_centers][3][S][n_max][L] d c(i) / d r_i = - sum_j d c(i) / d r_j
 *                                         (translational invariance).
 * A coincident neighbour (r = 0) contributes its on-site term to c and a zero
 * gradient.  jc_edge_dev may be NULL when the neighbour list has no edges.
 * Errors: SOAP_EINVAL, SOAP_ESTATE, SOAP_ENOMEM, SOAP_EHIP.
 */
int soap_coefficient_derivatives(soap_ctx *ctx, void *c_dev, void *jc_edge_dev, void *jc_self_dev, void *stream);

/*
 * Density-averaged descriptor over the centers of the neighbour list (the
 * "inner" and "outer" modes of Sec. 3), one row desc_dev[F] (dtype):
 *   SOAP_AVERAGE_OUTER: (1/n_c) sum_i p_i, the mean power spectrum;
 *   SOAP_AVERAGE_INNER: the power spectrum, Eq. (powerspectrum), of the mean
 *                       coefficients (1/n_c) sum_i c_i.
 * Uses a context-owned device scratch of n_c rows (F or S n_max L values of
 * the dtype).  Errors: SOAP_EINVAL (bad mode, NULL pointer), SOAP_ESTATE,
 * SOAP_ENOMEM, SOAP_EHIP.
 */
int soap_compute_averaged(soap_ctx *ctx, int32_t mode, void *desc_dev, void *stream);

/*
 * Descriptor and Jacobian, Eqs. (powerspectrum), (powerspectrum-derivative):
 *   desc_dev     [n_centers][F]        p_i
 *   jac_edge_dev [E][3][F_e]           d p_i / d r_j for the e-th edge (i, j)
 *                                      of the neighbour rows, compressed to the
 *                                      F_e features that can be non-zero (the
 *                                      pairs containing species(j); the map
 *                                      is soap_feature_map(species(j)));
 *   jac_self_dev [n_centers][3][F]     d p_i / d r_i = - sum_j d p_i / d r_j.
 * All derivatives not stored are exactly zero (atoms outside the cutoff,
 * features whose pair lacks species(j)).  Any element alignment works; in
 * float64 mode a 16-byte aligned jac_edge_dev is written with 16-byte stores
 * (faster) when both section lengths n_max^2 (l_max+1) and
 * n_max (n_max+1)/2 (l_max+1) are even.  Errors: SOAP_ESTATE, SOAP_ENOMEM,
 * SOAP_EHIP.
 */
int soap_derivatives(soap_ctx *ctx, void *desc_dev, void *jac_edge_dev, void *jac_self_dev, void *stream);

/*
 * Center batches (Sec. 3.3: the work is split into batches of centers of one
 * structure, and on one device the batches bound the memory of a single
 * call, so that a structure of any size streams through the device).  The
 * neighbour rows of every center are built once per structure by
 * soap_build_neighbors (4 bytes per edge); the batch calls below compute the
 * outputs of centers [first, first + count) of that list, indexed from the
 * batch's first center and first edge:
 *   soap_compute_batch     : desc_dev[count][F], as soap_compute;
 *   soap_derivatives_batch : desc_dev[count][F], jac_edge_dev[E_b][3][F_e],
 *                            jac_self_dev[count][3][F], as soap_derivatives,
 *                            where E_b = edge_first[k+1] - edge_first[k] of
 *                            the batch (soap_plan_batches), i.e. the edges of
 *                            its centers' rows; jac_edge_dev may be NULL only
 *                            when E_b = 0.
 * Each center's outputs are bitwise identical to those of the single call
 * over all centers (the per-center sums run in a fixed order).  The
 * Jacobian's coefficient scratch (4 S n_max (l_max+1)^2 values per center:
 * float32 in the mixed arithmetic, whose readers round c and D to float32,
 * float64 with dtype float64 or arith "fp64") is sized per batch.  count = 0 enqueues nothing.  Errors:
 * SOAP_EINVAL (range outside the centers, NULL outputs), SOAP_ESTATE,
 * SOAP_ENOMEM, SOAP_EHIP.
 */
int soap_compute_batch(soap_ctx *ctx, int64_t first, int64_t count, void *desc_dev, void *stream);
int soap_derivatives_batch(soap_ctx *ctx, int64_t first, int64_t count, void *desc_dev, void *jac_edge_dev,
                           void *jac_self_dev, void *stream);

/*
 * soap_derivatives_batch for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same outputs, bitwise, with the Jacobian path's
 * coefficient scratch taken from a fixed device array of
 * SOAP_STATIC_SCRATCH_BYTES (64 MiB) that the library holds on every device
 * it runs on (resolved at soap_create) instead of the context's growable
 * buffer.  This call allocates nothing and records no timing events; the
 * neighbour list must already be built (soap_build_neighbors allocates).
 * Limit: count * 4 S n_max (l_max+1)^2 scratch values (4 bytes each in the
 * mixed arithmetic, else 8; plus the polynomial quadrature's radial factors)
 * <= SOAP_STATIC_SCRATCH_BYTES (e.g. 5349 centers of the 2-species n_max 8,
 * l_max 6 basis in the mixed arithmetic, 2674 in float64), else
 * SOAP_ECAPACITY with nothing enqueued; larger structures go through in
 * batches.  Every call on one device shares that device's array, which
 * keeps the last call's contents (every entry read is written first, so
 * nothing needs clearing): calls that overlap on one device, on different
 * streams or from different contexts or host threads, race and must be
 * serialised by the caller.  jac_edge_dev must not be NULL for count > 0.
 * Errors: SOAP_EINVAL, SOAP_ESTATE, SOAP_ECAPACITY, SOAP_EHIP.
 */
int soap_derivatives_batch_noalloc(soap_ctx *ctx, int64_t first, int64_t count, void *desc_dev, void *jac_edge_dev,
                                   void *jac_self_dev, void *stream);

/*
 * Split the centers of the neighbour list into consecutive batches whose
 * memory stays within budget_bytes: for `what` = SOAP_BATCH_DESCRIPTOR the
 * descriptor rows; for SOAP_BATCH_DERIVATIVES the descriptor rows, center
 * blocks, neighbour blocks and the library's coefficient scratch of the
 * batch.  Greedy in center order.  On return *n_batches_out = the number of
 * batches B; if center_first (host, max_batches + 1 entries) is not NULL it
 * receives the first center of each batch and center_first[B] = n_centers,
 * and edge_first (host, may be NULL, max_batches + 1 entries) the first edge
 * of each batch and edge_first[B] = E.  Pass center_first = NULL to count
 * only.  Reads the row offsets back from the device (synchronous).
 * Errors: SOAP_EINVAL, SOAP_ESTATE, SOAP_ECAPACITY (a single center exceeds
 * the budget, or B > max_batches), SOAP_EHIP.
 */
int soap_plan_batches(soap_ctx *ctx, int32_t what, int64_t budget_bytes, int64_t max_batches,
                      int64_t *center_first, int64_t *edge_first, int64_t *n_batches_out);

/*
 * Expand a soap_derivatives result into the dense layout
 * dense_dev[n_centers][n_atoms][3][F] (dtype), zeros included: the
 * derivative tensor of shape (centers, atoms, 3, features) that the paper's
 * derivatives() returns (Sec. 3, the output layout shared with DScribe; the
 * dense (center, atom) blocks of Eq. (powerspectrum-derivative)).  Intended
 * for small structures (the dense array grows as n_centers * n_atoms).  With a
 * periodic cell the blocks of all images of an atom (and of the center's
 * own images) are summed into that atom's block: the derivative by the
 * atom's position, all of its images moving with it.
 */
int soap_scatter_dense(soap_ctx *ctx, const void *jac_edge_dev, const void *jac_self_dev, void *dense_dev,
                       void *stream);

/*
 * Per-segment device times of the calls made while option "timing" was on
 * (the per-segment profiler of Sec. 3.1).  Segments: 0 = neighbour search
 * (soap_build_neighbors, including its one host synchronisation),
 * 1 = density kernel (coefficients, power spectrum, center Jacobian block),
 * 2 = edge Jacobian kernel.  ms_out[3] receives the summed milliseconds and
 * count_out[3] (may be NULL) the number of timed launches per segment.
 * Synchronises on the recorded events; reset != 0 clears the records.
 * Errors: SOAP_EHIP.
 */
int soap_timing(soap_ctx *ctx, double *ms_out, int64_t *count_out, int32_t reset);

/* Message for the last error on this context ("" if none); with ctx = NULL,
 * the reason the calling thread's last soap_create failed. */
const char *soap_last_error(const soap_ctx *ctx);

/* Free the context and its device buffers (synchronises the device). NULL ok. */
void soap_destroy(soap_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* SOAP_MI355X_H */
