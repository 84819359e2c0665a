/*
 * Seeded synthetic structures for the SOAP descriptor + Jacobian workloads.
 *
 * This file holds input generation only: no SOAP arithmetic.  Both the HIP
 * path and the CPU oracle read what it produces (through the Python module
 * paper_2609_05709_amd/workloads.py), so they see bit-identical inputs.
 *
 * Random numbers come from SplitMix64 (Steele, Lea and Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014): a 64-bit counter
 * advanced by the golden-ratio increment and passed through the published
 * mix function.  Uniform doubles use the top 53 bits; normal deviates use the
 * Box-Muller transform.
 *
 * Structures:
 *  - water cluster: oxygen sites by random sequential addition, uniform in a
 *    sphere whose radius gives 0.0334 molecules per cubic angstrom, rejecting
 *    any O-O distance below 2.6 A; each molecule is the rigid geometry
 *    O-H 0.9572 A, H-O-H 104.52 deg, rotated by a uniform random unit
 *    quaternion.  Atom order O, H, H; Z = 8, 1, 1.
 *  - multi-species sphere: points uniform in a sphere of given radius with a
 *    minimum pair distance, species multiset shuffled by Fisher-Yates.
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct { uint64_t s; } sm64;

static uint64_t sm64_next(sm64 *g) {
    uint64_t z = (g->s += 0x9E3779B97F4A7C15ULL);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* uniform in [0, 1) */
static double sm64_uniform(sm64 *g) { return (double)(sm64_next(g) >> 11) * 0x1.0p-53; }

static double sm64_normal(sm64 *g) {
    /* Box-Muller; u1 in (0, 1] so the log is finite */
    double u1 = 1.0 - sm64_uniform(g);
    double u2 = sm64_uniform(g);
    return sqrt(-2.0 * log(u1)) * cos(2.0 * M_PI * u2);
}

/* ---- hashed cell grid used only for the rejection test ------------------ */
typedef struct {
    double edge;
    int64_t nbucket;      /* power of two */
    int64_t *head;        /* bucket -> first point, -1 = empty */
    int64_t *next;        /* point -> next point in bucket */
    const double *pts;    /* accepted points, xyz */
} hgrid;

static int64_t cell_of(double v, double edge) { return (int64_t)floor(v / edge); }

static int64_t bucket_of(int64_t cx, int64_t cy, int64_t cz, int64_t nbucket) {
    uint64_t h = (uint64_t)cx * 73856093ULL ^ (uint64_t)cy * 19349663ULL ^ (uint64_t)cz * 83492791ULL;
    h ^= h >> 29;
    h *= 0xBF58476D1CE4E5B9ULL;
    h ^= h >> 32;
    return (int64_t)(h & (uint64_t)(nbucket - 1));
}

static int hgrid_clear(const hgrid *g, const double p[3], double dmin) {
    int64_t cx = cell_of(p[0], g->edge), cy = cell_of(p[1], g->edge), cz = cell_of(p[2], g->edge);
    double d2min = dmin * dmin;
    for (int dx = -1; dx <= 1; ++dx)
        for (int dy = -1; dy <= 1; ++dy)
            for (int dz = -1; dz <= 1; ++dz) {
                int64_t b = bucket_of(cx + dx, cy + dy, cz + dz, g->nbucket);
                for (int64_t q = g->head[b]; q >= 0; q = g->next[q]) {
                    const double *o = g->pts + 3 * q;
                    double ex = o[0] - p[0], ey = o[1] - p[1], ez = o[2] - p[2];
                    if (ex * ex + ey * ey + ez * ez < d2min) return 0;
                }
            }
    return 1;
}

static void hgrid_insert(hgrid *g, int64_t idx) {
    const double *p = g->pts + 3 * idx;
    int64_t b = bucket_of(cell_of(p[0], g->edge), cell_of(p[1], g->edge), cell_of(p[2], g->edge), g->nbucket);
    g->next[idx] = g->head[b];
    g->head[b] = idx;
}

static int64_t pow2_at_least(int64_t n) {
    int64_t p = 1;
    while (p < n) p <<= 1;
    return p;
}

/* Random sequential addition of n points uniform in a ball of radius R with
 * minimum separation dmin.  Returns the number of draws, or -1 on failure. */
static int64_t rsa_ball(sm64 *g, int64_t n, double R, double dmin, double *pts, int64_t max_draws) {
    hgrid grid;
    grid.edge = dmin;
    grid.nbucket = pow2_at_least(2 * n + 16);
    grid.head = (int64_t *)malloc(sizeof(int64_t) * grid.nbucket);
    grid.next = (int64_t *)malloc(sizeof(int64_t) * (n > 0 ? n : 1));
    grid.pts = pts;
    if (!grid.head || !grid.next) { free(grid.head); free(grid.next); return -1; }
    for (int64_t b = 0; b < grid.nbucket; ++b) grid.head[b] = -1;
    int64_t k = 0, draws = 0;
    while (k < n) {
        if (draws >= max_draws) { k = -1; break; }
        ++draws;
        double p[3];
        for (int d = 0; d < 3; ++d) p[d] = (2.0 * sm64_uniform(g) - 1.0) * R;
        if (p[0] * p[0] + p[1] * p[1] + p[2] * p[2] > R * R) continue;
        if (!hgrid_clear(&grid, p, dmin)) continue;
        memcpy(pts + 3 * k, p, sizeof p);
        hgrid_insert(&grid, k);
        ++k;
    }
    free(grid.head);
    free(grid.next);
    return k < 0 ? -1 : draws;
}

/* Water cluster of n_mol molecules.  pos: 9*n_mol doubles, Z: 3*n_mol ints.
 * Returns the number of oxygen draws (>0) or -1. */
int64_t soapgen_water(int64_t n_mol, uint64_t seed, double density, double oo_min,
                      double *pos, int32_t *Z, double *radius_out) {
    if (n_mol <= 0) return -1;
    sm64 g = {seed};
    double R = cbrt(3.0 * (double)n_mol / (4.0 * M_PI * density));
    *radius_out = R;
    double *O = (double *)malloc(sizeof(double) * 3 * n_mol);
    if (!O) return -1;
    int64_t draws = rsa_ball(&g, n_mol, R, oo_min, O, 4000 * n_mol + 1000000);
    if (draws < 0) { free(O); return -1; }
    const double bond = 0.9572, half = 0.5 * 104.52 * M_PI / 180.0;
    const double h1[3] = {bond * sin(half), 0.0, bond * cos(half)};
    const double h2[3] = {-bond * sin(half), 0.0, bond * cos(half)};
    for (int64_t m = 0; m < n_mol; ++m) {
        double q[4], nrm = 0.0;
        do {
            nrm = 0.0;
            for (int d = 0; d < 4; ++d) { q[d] = sm64_normal(&g); nrm += q[d] * q[d]; }
        } while (nrm < 1e-12);
        nrm = sqrt(nrm);
        double w = q[0] / nrm, x = q[1] / nrm, y = q[2] / nrm, z = q[3] / nrm;
        double Rm[3][3] = {
            {1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)},
            {2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)},
            {2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)}};
        const double *o = O + 3 * m;
        double *a = pos + 9 * m;
        for (int d = 0; d < 3; ++d) {
            a[d] = o[d];
            a[3 + d] = o[d] + Rm[d][0] * h1[0] + Rm[d][1] * h1[1] + Rm[d][2] * h1[2];
            a[6 + d] = o[d] + Rm[d][0] * h2[0] + Rm[d][1] * h2[1] + Rm[d][2] * h2[2];
        }
        Z[3 * m] = 8;
        Z[3 * m + 1] = 1;
        Z[3 * m + 2] = 1;
    }
    free(O);
    return draws;
}

/* n points in a ball of radius R, minimum pair distance dmin; species from the
 * multiset zlist[0..nz) with counts zcount[], shuffled.  Returns draws or -1. */
int64_t soapgen_multispecies(int64_t n, uint64_t seed, double R, double dmin, const int32_t *zlist,
                             const int64_t *zcount, int32_t nz, double *pos, int32_t *Z) {
    int64_t tot = 0;
    for (int32_t t = 0; t < nz; ++t) tot += zcount[t];
    if (tot != n || n <= 0) return -1;
    sm64 g = {seed};
    int64_t draws = rsa_ball(&g, n, R, dmin, pos, 4000 * n + 1000000);
    if (draws < 0) return -1;
    int64_t k = 0;
    for (int32_t t = 0; t < nz; ++t)
        for (int64_t c = 0; c < zcount[t]; ++c) Z[k++] = zlist[t];
    for (int64_t i = n - 1; i > 0; --i) { /* Fisher-Yates */
        int64_t j = (int64_t)(sm64_next(&g) % (uint64_t)(i + 1));
        int32_t t = Z[i]; Z[i] = Z[j]; Z[j] = t;
    }
    return draws;
}

/* raw stream, for tests of the generator itself */
void soapgen_splitmix_stream(uint64_t seed, int64_t n, uint64_t *out) {
    sm64 g = {seed};
    for (int64_t i = 0; i < n; ++i) out[i] = sm64_next(&g);
}
