// Neighbour search on the device: a hashed cell list.
//
// Cells are cubes of edge h slightly above r_cut, so two atoms closer than
// r_cut lie in the same or adjacent cells.  Cells are hashed into H buckets
// (no bounding box needed, any spatial extent); a bucket can hold atoms of
// several cells, so every candidate's cell coordinates are compared before
// its distance is tested, which also rules out visiting a candidate twice.
//
// Phase 1: species lookup, cell hashing, bucket counts -> bucket offsets,
//          bucket fill, per-center neighbour counts -> CSR row offsets.
// Phase 2: per center, gather the neighbour keys (species, atom) in LDS,
//          order them by rank (keys are unique), write the row.
// The cutoff test is the exact float64 one defined in soap.h.
#include "soap_internal.h"

namespace soap {
namespace {

constexpr double CELL_PAD = 1.0001;

__device__ __forceinline__ uint32_t cell_hash(int cx, int cy, int cz, uint32_t mask) {
    uint32_t h = (uint32_t)cx * 73856093u ^ (uint32_t)cy * 19349663u ^ (uint32_t)cz * 83492791u;
    h ^= h >> 15;
    h *= 0x2c1b3c6du;
    h ^= h >> 12;
    return h & mask;
}

template <typename PosT>
__device__ __forceinline__ double3 load_pos(const PosT *pos, int64_t i) {
    return make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);
}

// |r_j - r_i|^2 < r_cut^2 evaluated as ((dx*dx + dy*dy) + dz*dz), no contraction
__device__ __forceinline__ bool within_cutoff(double3 a, double3 b, double rc2) {
#pragma clang fp contract(off)
    double dx = b.x - a.x, dy = b.y - a.y, dz = b.z - a.z;
    double d2 = dx * dx + dy * dy;
    d2 = d2 + dz * dz;
    return d2 < rc2;
}

template <typename PosT>
__global__ void k_prepare(int64_t n, const PosT *__restrict__ pos, const int32_t *__restrict__ Z,
                          const int8_t *__restrict__ lut, uint8_t *__restrict__ spec, int4 *__restrict__ cell,
                          int32_t *__restrict__ count, uint32_t mask, double inv_h, int32_t *__restrict__ flags) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    int z = Z[i];
    int s = (z >= 0 && z < 128) ? (int)lut[z] : -1;
    if (s < 0) {
        atomicOr(&flags[0], 1);
        s = 0;
    }
    spec[i] = (uint8_t)s;
    double3 p = load_pos(pos, i);
    int cx = (int)floor(p.x * inv_h), cy = (int)floor(p.y * inv_h), cz = (int)floor(p.z * inv_h);
    uint32_t b = cell_hash(cx, cy, cz, mask);
    cell[i] = make_int4(cx, cy, cz, (int)b);
    atomicAdd(&count[b], 1);
}

template <typename PosT>
__global__ void k_bucket_fill(int64_t n, const PosT *__restrict__ pos, const int4 *__restrict__ cell,
                              const int32_t *__restrict__ start, int32_t *__restrict__ fill,
                              int4 *__restrict__ scell, double4 *__restrict__ spos, int32_t *__restrict__ satom) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    int4 c = cell[i];
    int slot = start[c.w] + atomicAdd(&fill[c.w], 1);
    double3 p = load_pos(pos, i);
    scell[slot] = c;
    spos[slot] = make_double4(p.x, p.y, p.z, 0.0);
    satom[slot] = (int32_t)i;
}

// Candidate enumeration shared by the count and fill passes: one 64-lane wave
// per center.  Lanes 0..26 look up one neighbouring cell each (bucket range
// and cell coordinates) into the wave's LDS slots; a prefix over the 27
// bucket sizes then lets every lane take candidates t = lane, lane + 64, ...
// of the concatenated buckets, so the loads of one center are spread over
// the whole wave instead of walking each bucket serially.
struct CellSlots {
    int off[28];   // prefix of bucket sizes
    int start[27]; // first sorted slot of each bucket
    int cx[27], cy[27], cz[27];
};

__device__ __forceinline__ int wave_prefix_cells(CellSlots &cs, int lane, int4 ci, const int32_t *__restrict__ start,
                                                 uint32_t mask) {
    int sz = 0;
    if (lane < 27) {
        const int tx = ci.x + lane % 3 - 1, ty = ci.y + (lane / 3) % 3 - 1, tz = ci.z + lane / 9 - 1;
        const uint32_t b = cell_hash(tx, ty, tz, mask);
        const int s0 = start[b];
        sz = start[b + 1] - s0;
        cs.start[lane] = s0;
        cs.cx[lane] = tx;
        cs.cy[lane] = ty;
        cs.cz[lane] = tz;
    }
    // inclusive scan of sz over lanes 0..26
    int v = sz;
    for (int d = 1; d < 32; d <<= 1) {
        const int u = __shfl_up(v, d, 64);
        if (lane >= d) v += u;
    }
    if (lane < 27) cs.off[lane + 1] = v;
    if (lane == 0) cs.off[0] = 0;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    return cs.off[27];
}

// Candidate t of the concatenated buckets: its sorted slot, or -1 if it
// belongs to another cell that shares the bucket.
__device__ __forceinline__ int candidate_slot(const CellSlots &cs, int t, const int4 *__restrict__ scell) {
    int d = 0;
    while (cs.off[d + 1] <= t) ++d;
    const int slot = cs.start[d] + (t - cs.off[d]);
    const int4 sc = scell[slot];
    return (sc.x == cs.cx[d] && sc.y == cs.cy[d] && sc.z == cs.cz[d]) ? slot : -1;
}

template <typename PosT>
__global__ __launch_bounds__(256) void k_count(int64_t n_atoms, int64_t nc, const int32_t *__restrict__ centers,
                                               const PosT *__restrict__ pos, const int4 *__restrict__ cell,
                                               const int32_t *__restrict__ start, const int4 *__restrict__ scell,
                                               const double4 *__restrict__ spos, const int32_t *__restrict__ satom,
                                               uint32_t mask, double rc2, int32_t *__restrict__ deg,
                                               int32_t *__restrict__ flags) {
    __shared__ CellSlots slots[4];
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t c = (int64_t)blockIdx.x * 4 + w;
    if (c >= nc) return;
    const int64_t i = centers ? (int64_t)centers[c] : c;
    if (i < 0 || i >= n_atoms) {
        if (lane == 0) {
            atomicOr(&flags[0], 2);
            deg[c] = 0;
        }
        return;
    }
    CellSlots &cs = slots[w];
    const int total = wave_prefix_cells(cs, lane, cell[i], start, mask);
    const double3 pi = load_pos(pos, i);
    int cnt = 0;
    for (int t = lane; t < total; t += 64) {
        const int slot = candidate_slot(cs, t, scell);
        if (slot < 0 || satom[slot] == (int32_t)i) continue;
        const double4 q = spos[slot];
        if (within_cutoff(pi, make_double3(q.x, q.y, q.z), rc2)) ++cnt;
    }
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_down(cnt, off, 64);
    if (lane == 0) {
        deg[c] = cnt;
        atomicMax(&flags[1], cnt);
    }
}

// One 64-lane workgroup per center: matching candidates are appended to the
// LDS key list (slot from a ballot prefix), keys (species << 32 | atom) are
// unique and each key's rank among the row's keys is its output position.
template <typename PosT>
__global__ __launch_bounds__(64) void k_fill_sort(int64_t nc, const int32_t *__restrict__ centers,
                                                  const PosT *__restrict__ pos, const uint8_t *__restrict__ spec,
                                                  const int4 *__restrict__ cell, const int32_t *__restrict__ start,
                                                  const int4 *__restrict__ scell, const double4 *__restrict__ spos,
                                                  const int32_t *__restrict__ satom, uint32_t mask, double rc2,
                                                  const int64_t *__restrict__ row_ptr, int32_t *__restrict__ cols) {
    __shared__ int64_t keys[MAX_DEGREE];
    __shared__ CellSlots cs;
    const int64_t c = blockIdx.x;
    const int lane = threadIdx.x;
    const int64_t r0 = row_ptr[c];
    const int deg = (int)(row_ptr[c + 1] - r0);
    if (deg == 0) return;
    const int64_t i = centers ? (int64_t)centers[c] : c;
    const int total = wave_prefix_cells(cs, lane, cell[i], start, mask);
    const double3 pi = load_pos(pos, i);
    int base = 0;
    for (int t0 = 0; t0 < total; t0 += 64) {
        const int t = t0 + lane;
        bool hit = false;
        int j = 0;
        if (t < total) {
            const int slot = candidate_slot(cs, t, scell);
            if (slot >= 0) {
                j = satom[slot];
                if (j != (int32_t)i) {
                    const double4 q = spos[slot];
                    hit = within_cutoff(pi, make_double3(q.x, q.y, q.z), rc2);
                }
            }
        }
        const uint64_t m = __ballot(hit);
        const int pre = __popcll(m & ((1ull << lane) - 1ull));
        if (hit && base + pre < MAX_DEGREE) keys[base + pre] = ((int64_t)spec[j] << 32) | (int64_t)(uint32_t)j;
        base += __popcll(m);
    }
    __syncthreads();
    for (int k = lane; k < deg; k += 64) {
        const int64_t key = keys[k];
        int rank = 0;
        for (int t = 0; t < deg; ++t) rank += keys[t] < key;
        cols[r0 + rank] = (int32_t)(key & 0xffffffff);
    }
}

// ---- exclusive scan of int32 counts into int64 offsets (out has n+1) ----
constexpr int SCAN_THREADS = 256, SCAN_ITEMS = 8, SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;

template <typename OutT>
__global__ __launch_bounds__(SCAN_THREADS) void k_scan_tile(int64_t n, const int32_t *__restrict__ in,
                                                            OutT *__restrict__ out, int64_t *__restrict__ sums) {
    __shared__ int64_t part[SCAN_THREADS];
    const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
    int64_t v[SCAN_ITEMS], s = 0;
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        v[k] = (base + k < n) ? (int64_t)in[base + k] : 0;
        s += v[k];
    }
    part[threadIdx.x] = s;
    __syncthreads();
    for (int off = 1; off < SCAN_THREADS; off <<= 1) {
        int64_t t = (threadIdx.x >= off) ? part[threadIdx.x - off] : 0;
        __syncthreads();
        part[threadIdx.x] += t;
        __syncthreads();
    }
    int64_t run = part[threadIdx.x] - s; // exclusive within the tile
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        if (base + k < n) out[base + k] = (OutT)run;
        run += v[k];
    }
    if (threadIdx.x == SCAN_THREADS - 1) sums[blockIdx.x] = part[threadIdx.x];
}

// single workgroup: exclusive scan of the tile sums in place; total -> *total
__global__ __launch_bounds__(1024) void k_scan_sums(int64_t m, int64_t *__restrict__ sums,
                                                    int64_t *__restrict__ total) {
    __shared__ int64_t part[1024];
    const int per = (int)((m + 1023) / 1024);
    const int64_t base = (int64_t)threadIdx.x * per;
    int64_t s = 0;
    for (int k = 0; k < per; ++k)
        if (base + k < m) s += sums[base + k];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        int64_t t = (threadIdx.x >= off) ? part[threadIdx.x - off] : 0;
        __syncthreads();
        part[threadIdx.x] += t;
        __syncthreads();
    }
    int64_t run = part[threadIdx.x] - s;
    for (int k = 0; k < per; ++k)
        if (base + k < m) {
            int64_t v = sums[base + k];
            sums[base + k] = run;
            run += v;
        }
    if (threadIdx.x == 1023) *total = part[1023];
}

template <typename OutT>
__global__ void k_scan_add(int64_t n, OutT *__restrict__ out, const int64_t *__restrict__ sums,
                           const int64_t *__restrict__ total) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] += (OutT)sums[i / SCAN_TILE];
    if (i == n) out[n] = (OutT)*total;
}

template <typename OutT>
hipError_t exclusive_scan(int64_t n, const int32_t *in, OutT *out, int64_t *tmp, hipStream_t st) {
    int64_t tiles = (n + SCAN_TILE - 1) / SCAN_TILE;
    if (tiles < 1) tiles = 1;
    // tmp layout: [tiles] tile sums, then [1] total
    hipLaunchKernelGGL(k_scan_tile<OutT>, dim3((unsigned)tiles), dim3(SCAN_THREADS), 0, st, n, in, out, tmp);
    hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(1024), 0, st, tiles, tmp, tmp + tiles);
    hipLaunchKernelGGL(k_scan_add<OutT>, dim3((unsigned)((n + 1 + 255) / 256)), dim3(256), 0, st, n, out, tmp,
                       tmp + tiles);
    return hipGetLastError();
}

unsigned blocks_for(int64_t n, int bs) { return (unsigned)((n + bs - 1) / bs); }

} // namespace

hipError_t nbr_phase1(const NbrWork &w, int64_t n_atoms, const void *pos, bool pos64, const int32_t *Z,
                      const int8_t *lut, uint8_t *spec, int64_t nc, const int32_t *centers, double r_cut,
                      int64_t *row_ptr, hipStream_t st) {
    const double h = r_cut * CELL_PAD, inv_h = 1.0 / h, rc2 = r_cut * r_cut;
    const uint32_t mask = (uint32_t)(w.H - 1);
    hipError_t e;
    if ((e = hipMemsetAsync(w.bucket_count, 0, sizeof(int32_t) * w.H, st)) != hipSuccess) return e;
    if ((e = hipMemsetAsync(w.bucket_fill, 0, sizeof(int32_t) * w.H, st)) != hipSuccess) return e;
    if ((e = hipMemsetAsync(w.flags, 0, sizeof(int32_t) * 4, st)) != hipSuccess) return e;
    const unsigned gb = blocks_for(n_atoms, 256);
    if (pos64)
        hipLaunchKernelGGL(k_prepare<double>, dim3(gb), dim3(256), 0, st, n_atoms, (const double *)pos, Z, lut,
                           spec, w.atom_cell, w.bucket_count, mask, inv_h, w.flags);
    else
        hipLaunchKernelGGL(k_prepare<float>, dim3(gb), dim3(256), 0, st, n_atoms, (const float *)pos, Z, lut,
                           spec, w.atom_cell, w.bucket_count, mask, inv_h, w.flags);
    if ((e = exclusive_scan<int32_t>(w.H, w.bucket_count, w.bucket_start, w.scan_tmp, st)) != hipSuccess)
        return e;
    if (pos64)
        hipLaunchKernelGGL(k_bucket_fill<double>, dim3(gb), dim3(256), 0, st, n_atoms, (const double *)pos,
                           w.atom_cell, w.bucket_start, w.bucket_fill, w.sorted_cell, w.sorted_pos, w.sorted_atom);
    else
        hipLaunchKernelGGL(k_bucket_fill<float>, dim3(gb), dim3(256), 0, st, n_atoms, (const float *)pos,
                           w.atom_cell, w.bucket_start, w.bucket_fill, w.sorted_cell, w.sorted_pos, w.sorted_atom);
    const unsigned gc = blocks_for(nc, 4);
    if (pos64)
        hipLaunchKernelGGL(k_count<double>, dim3(gc), dim3(256), 0, st, n_atoms, nc, centers, (const double *)pos,
                           w.atom_cell, w.bucket_start, w.sorted_cell, w.sorted_pos, w.sorted_atom, mask, rc2, w.deg,
                           w.flags);
    else
        hipLaunchKernelGGL(k_count<float>, dim3(gc), dim3(256), 0, st, n_atoms, nc, centers, (const float *)pos,
                           w.atom_cell, w.bucket_start, w.sorted_cell, w.sorted_pos, w.sorted_atom, mask, rc2, w.deg,
                           w.flags);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return exclusive_scan<int64_t>(nc, w.deg, row_ptr, w.scan_tmp, st);
}

hipError_t nbr_phase2(const NbrWork &w, int64_t n_atoms, const void *pos, bool pos64, const uint8_t *spec,
                      int64_t nc, const int32_t *centers, double r_cut, const int64_t *row_ptr, int32_t *cols,
                      hipStream_t st) {
    (void)n_atoms;
    const double rc2 = r_cut * r_cut;
    const uint32_t mask = (uint32_t)(w.H - 1);
    if (pos64)
        hipLaunchKernelGGL(k_fill_sort<double>, dim3((unsigned)nc), dim3(64), 0, st, nc, centers, (const double *)pos,
                           spec, w.atom_cell, w.bucket_start, w.sorted_cell, w.sorted_pos, w.sorted_atom, mask, rc2,
                           row_ptr, cols);
    else
        hipLaunchKernelGGL(k_fill_sort<float>, dim3((unsigned)nc), dim3(64), 0, st, nc, centers, (const float *)pos,
                           spec, w.atom_cell, w.bucket_start, w.sorted_cell, w.sorted_pos, w.sorted_atom, mask, rc2,
                           row_ptr, cols);
    return hipGetLastError();
}

} // namespace soap
