// Neighbour search on the device: a hashed cell list.
//
// Cells are cubes of edge h slightly above r_cut, so two atoms closer than
// r_cut lie in the same or adjacent cells.  Cells go to H = 2^k buckets by a
// spatially coherent key: the low b = floor(k / 3) bits of the three cell
// coordinates, bit-interleaved (Morton order), with a hash of the remaining
// high bits above them.  Consequences used below:
//   - neighbouring cells get neighbouring buckets, so the sorted atom order
//     is spatially local, and so are consecutive centers in that order;
//   - the 27 cells around a center fall into 27 distinct buckets (b >= 2:
//     coordinates that differ by at most 2 differ in their low b bits), so
//     no atom is visited twice;
//   - another cell sharing a bucket with one of those 27 is at least 2^b - 1
//     cells away along some axis, i.e. at least 2 h > r_cut from the center,
//     and its atoms fail the cutoff test; no cell coordinates need comparing.
// Cells whose box lies farther than r_cut from the center are skipped.
//
// Phase 1: species lookup, cell keys, bucket counts -> bucket offsets,
//          bucket fill (position + atom records), then one wave per center
//          collects its neighbour keys (species, atom) in LDS, ranks them
//          (keys are unique) and writes the ordered row to a fixed-capacity
//          slot (TCAP entries) with its degree; CSR row offsets by scan,
//          which also finds the largest degree and the rows above TCAP.
// Phase 2 (after the host has read the total): the slots are packed into
//          the CSR rows; rows longer than TCAP are collected again, with up
//          to MAX_DEGREE keys in LDS.
// The cutoff test is the exact float64 one defined in soap.h.
#include "soap_internal.h"

namespace soap {
namespace {

constexpr double CELL_PAD = 1.0001;

// spread the low 10 bits of x to every third bit
__device__ __forceinline__ uint32_t spread3(uint32_t x) {
    x &= 0x3ff;
    x = (x | (x << 16)) & 0x030000ff;
    x = (x | (x << 8)) & 0x0300f00f;
    x = (x | (x << 4)) & 0x030c30c3;
    x = (x | (x << 2)) & 0x09249249;
    return x;
}

__device__ __forceinline__ uint32_t cell_key(int cx, int cy, int cz, int b, uint32_t mask) {
    const uint32_t lo_mask = (1u << b) - 1u;
    const uint32_t m = spread3((uint32_t)cx & lo_mask) | spread3((uint32_t)cy & lo_mask) << 1 |
                       spread3((uint32_t)cz & lo_mask) << 2;
    uint32_t h = (uint32_t)(cx >> b) * 73856093u ^ (uint32_t)(cy >> b) * 19349663u ^ (uint32_t)(cz >> b) * 83492791u;
    h ^= h >> 15;
    h *= 0x2c1b3c6du;
    h ^= h >> 12;
    return (m | (3 * b < 32 ? h << (3 * b) : 0u)) & mask;
}

template <typename PosT>
__device__ __forceinline__ double3 load_pos(const PosT *pos, int64_t i) {
    return make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);
}

// sorted-atom record: position at the input precision and the atom index
template <typename PosT> struct Rec;
template <> struct Rec<float> {
    using type = float4;
    static __device__ __forceinline__ float4 make(const float *p, int32_t i) {
        return make_float4(p[0], p[1], p[2], __int_as_float(i));
    }
    static __device__ __forceinline__ int32_t atom(float4 r) { return __float_as_int(r.w); }
    static __device__ __forceinline__ double3 pos(float4 r) { return make_double3(r.x, r.y, r.z); }
};
template <> struct Rec<double> {
    using type = double4;
    static __device__ __forceinline__ double4 make(const double *p, int32_t i) {
        return make_double4(p[0], p[1], p[2], (double)i);
    }
    static __device__ __forceinline__ int32_t atom(double4 r) { return (int32_t)r.w; }
    static __device__ __forceinline__ double3 pos(double4 r) { return make_double3(r.x, r.y, r.z); }
};

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
                          int32_t *__restrict__ count, uint32_t mask, int b, double inv_h, int32_t *__restrict__ flags) {
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
    uint32_t k = cell_key(cx, cy, cz, b, mask);
    cell[i] = make_int4(cx, cy, cz, (int)k);
    atomicAdd(&count[k], 1);
}

template <typename PosT>
__global__ void k_bucket_fill(int64_t n, const PosT *__restrict__ pos, const uint8_t *__restrict__ spec,
                              const int4 *__restrict__ cell, const int32_t *__restrict__ start,
                              int32_t *__restrict__ fill, typename Rec<PosT>::type *__restrict__ srec,
                              uint8_t *__restrict__ sspec) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int k = cell[i].w;
    const int slot = start[k] + atomicAdd(&fill[k], 1);
    srec[slot] = Rec<PosT>::make(pos + 3 * i, (int32_t)i);
    sspec[slot] = spec[i];
}

// The candidates of one center: the atoms of the buckets of the (up to) 27
// cells around it, concatenated.  Lanes 0..26 look up one cell each and
// write the sorted-record index of each of the cell's atoms into the wave's
// candidate list (cand[t], t < total); then lane l takes candidates l,
// l + 64, ... so the loads of one center spread over the whole wave.  Lists
// longer than the LDS list (cap) are walked through the bucket offsets.
struct CellSlots {
    int off[28];   // prefix of bucket sizes
    int start[27]; // first sorted slot of each bucket
};

// cell of a position: the same expression as k_prepare's
__device__ __forceinline__ int4 cell_of(double3 p, double inv_h) {
    return make_int4((int)floor(p.x * inv_h), (int)floor(p.y * inv_h), (int)floor(p.z * inv_h), 0);
}

__device__ __forceinline__ int wave_prefix_cells(CellSlots &cs, int *cand, int cap, int lane, double3 pi,
                                                 double inv_h, double lim2, int b,
                                                 const int32_t *__restrict__ start, uint32_t mask) {
    const int4 ci = cell_of(pi, inv_h);
    int sz = 0, s0 = 0;
    if (lane < 27) {
        const int dx = lane % 3 - 1, dy = (lane / 3) % 3 - 1, dz = lane / 9 - 1;
        // gap from the center to the cell's box along each axis, in cell units
        const double ux = pi.x * inv_h, uy = pi.y * inv_h, uz = pi.z * inv_h;
        const double gx = dx < 0 ? ux - (double)ci.x : dx > 0 ? (double)(ci.x + 1) - ux : 0.0;
        const double gy = dy < 0 ? uy - (double)ci.y : dy > 0 ? (double)(ci.y + 1) - uy : 0.0;
        const double gz = dz < 0 ? uz - (double)ci.z : dz > 0 ? (double)(ci.z + 1) - uz : 0.0;
        const double g2 = fmax(gx, 0.0) * fmax(gx, 0.0) + fmax(gy, 0.0) * fmax(gy, 0.0) + fmax(gz, 0.0) * fmax(gz, 0.0);
        if (g2 <= lim2) {
            const uint32_t k = cell_key(ci.x + dx, ci.y + dy, ci.z + dz, b, mask);
            s0 = start[k];
            sz = start[k + 1] - s0;
            cs.start[lane] = s0;
        }
    }
    // inclusive scan of sz over lanes 0..26
    int v = sz;
    for (int d = 1; d < 32; d <<= 1) {
        const int u = __shfl_up(v, d, 64);
        if (lane >= d) v += u;
    }
    if (lane < 27) cs.off[lane + 1] = v;
    if (lane == 0) cs.off[0] = 0;
    const int total = __shfl(v, 26, 64);
    if (total <= cap)
        for (int k = 0; k < sz; ++k) cand[v - sz + k] = s0 + k;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    return total;
}

// Collect the neighbour keys (species << 32 | atom) of center atom i into
// keys[0..kcap) in candidate order; returns the degree (which may exceed
// kcap: the surplus keys are counted, not stored).  U candidates per lane
// are loaded together.
template <typename PosT, int U>
__device__ __forceinline__ int collect_keys(const CellSlots &cs, const int *cand, int cap, int total, int lane,
                                            int64_t i, double3 pi, double rc2,
                                            const typename Rec<PosT>::type *__restrict__ srec,
                                            const uint8_t *__restrict__ sspec, int64_t *keys, int kcap) {
    int base = 0, d = 0;
    for (int t0 = 0; t0 < total; t0 += 64 * U) {
        int slot[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int t = t0 + 64 * u + lane;
            slot[u] = -1;
            if (t < total) {
                if (total <= cap) {
                    slot[u] = cand[t];
                } else {
                    while (cs.off[d + 1] <= t) ++d; // t grows with u and t0: d only moves forward
                    slot[u] = cs.start[d] + (t - cs.off[d]);
                }
            }
        }
        typename Rec<PosT>::type r[U];
        int sp[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = slot[u] < 0 ? 0 : slot[u];
            r[u] = srec[s];
            sp[u] = sspec[s];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t j = Rec<PosT>::atom(r[u]);
            const bool hit = slot[u] >= 0 && j != (int32_t)i && within_cutoff(pi, Rec<PosT>::pos(r[u]), rc2);
            const uint64_t m = __ballot(hit);
            const int pre = __popcll(m & ((1ull << lane) - 1ull));
            if (hit && base + pre < kcap) keys[base + pre] = ((int64_t)sp[u] << 32) | (int64_t)(uint32_t)j;
            base += __popcll(m);
        }
    }
    return base;
}

// Write the deg (<= what keys holds) keys of a wave in ascending order:
// each key's rank among the row's keys is its position.
__device__ __forceinline__ void write_ranked(const int64_t *keys, int deg, int lane, int32_t *__restrict__ out) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int k = lane; k < deg; k += 64) {
        const int64_t key = keys[k];
        int r0 = 0, r1 = 0, r2 = 0, r3 = 0, t = 0;
        for (; t + 4 <= deg; t += 4) { // four independent LDS reads in flight
            r0 += keys[t] < key;
            r1 += keys[t + 1] < key;
            r2 += keys[t + 2] < key;
            r3 += keys[t + 3] < key;
        }
        for (; t < deg; ++t) r0 += keys[t] < key;
        out[r0 + r1 + r2 + r3] = (int32_t)(key & 0xffffffff);
    }
}

constexpr int NBR_WAVES = 4;   // centers per workgroup in the collecting pass
constexpr int CAND_CAP = 1024; // candidate list per wave in LDS

// One wave per center.  Without a center list the centers are taken in
// sorted-atom (cell) order, so the waves resident on a CU share cells.
template <typename PosT>
__global__ __launch_bounds__(64 * NBR_WAVES) void k_collect(
    int64_t center_bound, int64_t nc, const int32_t *__restrict__ centers, const PosT *__restrict__ pos,
    const int32_t *__restrict__ start, const typename Rec<PosT>::type *__restrict__ srec,
    const uint8_t *__restrict__ sspec, uint32_t mask, int b, double inv_h, double lim2, double rc2,
    int32_t *__restrict__ deg, int32_t *__restrict__ slots, int32_t *__restrict__ flags) {
    __shared__ CellSlots cslots[NBR_WAVES];
    __shared__ int64_t kbuf[NBR_WAVES][TCAP];
    __shared__ int cbuf[NBR_WAVES][CAND_CAP];
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * NBR_WAVES + w;
    if (t >= nc) return;
    int64_t c, i;
    double3 pi;
    if (centers) {
        c = t;
        i = centers[c];
        if (i < 0 || i >= center_bound) {
            if (lane == 0) {
                atomicOr(&flags[0], 2);
                deg[c] = 0;
            }
            return;
        }
        pi = load_pos(pos, i);
    } else {
        const typename Rec<PosT>::type r = srec[t];
        i = Rec<PosT>::atom(r);
        c = i;
        pi = Rec<PosT>::pos(r);
    }
    CellSlots &cs = cslots[w];
    const int total = wave_prefix_cells(cs, cbuf[w], CAND_CAP, lane, pi, inv_h, lim2, b, start, mask);
    int64_t *keys = kbuf[w];
    const int dg = collect_keys<PosT, 4>(cs, cbuf[w], CAND_CAP, total, lane, i, pi, rc2, srec, sspec, keys, TCAP);
    if (dg <= TCAP) write_ranked(keys, dg, lane, slots + c * TCAP);
    // (the largest degree and the rows above TCAP are counted by the scan of
    // deg: one atomic per center on a single address would serialise)
    if (lane == 0) deg[c] = dg;
}

// CSR rows from the fixed-capacity slots; rows longer than TCAP are left to
// k_collect_long.
// cap: entries of cols; nothing is written if the rows need more
__global__ __launch_bounds__(256) void k_pack(int64_t nc, const int64_t *__restrict__ row_ptr,
                                              const int32_t *__restrict__ slots, int32_t *__restrict__ cols,
                                              int64_t cap) {
    const int64_t c = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (c >= nc || row_ptr[nc] > cap) return;
    const int64_t r0 = row_ptr[c];
    const int dg = (int)(row_ptr[c + 1] - r0);
    if (dg > TCAP) return;
    for (int k = lane; k < dg; k += 64) cols[r0 + k] = slots[c * TCAP + k];
}

// Rows longer than TCAP, collected again with MAX_DEGREE keys in LDS (one
// 64-lane workgroup per center; other centers return at once).
template <typename PosT>
__global__ __launch_bounds__(64) void k_collect_long(
    int64_t nc, const int32_t *__restrict__ centers, const PosT *__restrict__ pos, const int32_t *__restrict__ start, const typename Rec<PosT>::type *__restrict__ srec,
    const uint8_t *__restrict__ sspec, uint32_t mask, int b, double inv_h, double lim2, double rc2,
    const int64_t *__restrict__ row_ptr, int32_t *__restrict__ cols) {
    __shared__ int64_t keys[MAX_DEGREE];
    __shared__ CellSlots cs;
    const int64_t c = blockIdx.x;
    const int lane = threadIdx.x;
    const int64_t r0 = row_ptr[c];
    const int dg = (int)(row_ptr[c + 1] - r0);
    if (dg <= TCAP) return;
    const int64_t i = centers ? (int64_t)centers[c] : c;
    const double3 pi = load_pos(pos, i);
    const int total = wave_prefix_cells(cs, nullptr, 0, lane, pi, inv_h, lim2, b, start, mask);
    const int got = collect_keys<PosT, 4>(cs, nullptr, 0, total, lane, i, pi, rc2, srec, sspec, keys, MAX_DEGREE);
    write_ranked(keys, got < dg ? got : dg, lane, cols + r0);
}

// ---- exclusive scan of int32 counts into offsets (out has n+1) ----
constexpr int SCAN_THREADS = 256, SCAN_ITEMS = 8, SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;
constexpr int SMALL_THREADS = 1024, SMALL_ITEMS = 16, SMALL_MAX = SMALL_THREADS * SMALL_ITEMS;

// workgroup-wide exclusive scan of one value per thread (BS threads); returns
// the exclusive prefix, *sum gets the total
// Exclusive prefix of s over the workgroup (BS threads): a shuffle scan in
// each wave, then the wave totals scanned by the first wave; two barriers.
// part holds BS / 64 entries; *sum receives the workgroup total.
template <int BS>
__device__ __forceinline__ int64_t block_exclusive(int64_t s, int64_t *part, int64_t *sum) {
    constexpr int NW = BS / 64;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int64_t x = s;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    if (lane == 63) part[w] = x;
    __syncthreads();
    if (w == 0) {
        int64_t t = lane < NW ? part[lane] : 0;
#pragma unroll
        for (int d = 1; d < NW; d <<= 1) {
            const int64_t y = __shfl_up(t, d, 64);
            if (lane >= d) t += y;
        }
        if (lane < NW) part[lane] = t;
    }
    __syncthreads();
    *sum = part[NW - 1];
    return (w > 0 ? part[w - 1] : 0) + x - s;
}

// Largest value and number of values above TCAP of the workgroup's inputs,
// folded into stats[0] (max) and stats[1] (count) with one atomic each; thread
// 0 also gets the workgroup's pair as the return value.
template <int BS>
__device__ __forceinline__ int2 block_degree_stats(int vmax, int over, int *red, int32_t *__restrict__ stats) {
    for (int off = 32; off > 0; off >>= 1) {
        vmax = max(vmax, __shfl_down(vmax, off, 64));
        over += __shfl_down(over, off, 64);
    }
    if ((threadIdx.x & 63) == 0) {
        red[2 * (threadIdx.x >> 6)] = vmax;
        red[2 * (threadIdx.x >> 6) + 1] = over;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < BS / 64; ++w) {
            vmax = max(vmax, red[2 * w]);
            over += red[2 * w + 1];
        }
        atomicMax(&stats[0], vmax);
        atomicAdd(&stats[1], over);
    }
    return make_int2(vmax, over);
}

// one workgroup for n <= SMALL_MAX; total also to *total_copy and degree
// statistics to stats if given.  Rounds of SMALL_THREADS x 4 consecutive
// items: each thread takes four in one 16-byte load (coalesced across the
// wave), then a shuffle scan of the threads' sums within the waves and of the
// wave totals.  The wave-total array alternates between rounds, so a round's
// two barriers also order the previous round's reads of it.  All loads are
// issued first; the cross-lane shuffles set the time, so rounds are few.
//
// rec (may be NULL; needs stats): a host-visible record that thread 0 writes
// last, once the scan and the statistics are final: [0] err[0] | stats[0] <<
// 32, [1] stats[1], [2] the total, then [3] = seq with a system-scope release,
// so that the host can wait for this value instead of synchronising the
// stream.
template <typename OutT>
__global__ __launch_bounds__(SMALL_THREADS) void k_scan_small(int64_t n, const int32_t *__restrict__ in,
                                                              OutT *__restrict__ out, int64_t *__restrict__ total_copy,
                                                              int32_t *__restrict__ stats,
                                                              const int32_t *__restrict__ err, int64_t *rec,
                                                              int64_t seq) {
    constexpr int NW = SMALL_THREADS / 64, VEC = 4, ROUND = SMALL_THREADS * VEC, MAXR = SMALL_MAX / ROUND;
    __shared__ int64_t part[2][NW];
    __shared__ int red[2 * NW];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int64_t carry = 0;
    int vmax = 0, over = 0;
    int32_t vr[MAXR][VEC];
#pragma unroll
    for (int r = 0; r < MAXR; ++r) {
        const int64_t b = (int64_t)r * ROUND + (int64_t)threadIdx.x * VEC;
        if (b + VEC <= n) {
            const int4 q = *(const int4 *)(in + b); // in is 16-byte aligned
            vr[r][0] = q.x;
            vr[r][1] = q.y;
            vr[r][2] = q.z;
            vr[r][3] = q.w;
        } else {
#pragma unroll
            for (int k = 0; k < VEC; ++k) vr[r][k] = b + k < n ? in[b + k] : 0;
        }
    }
    const int rounds = (int)((n + ROUND - 1) / ROUND);
#pragma unroll
    for (int r = 0; r < MAXR; ++r) {
        if (r >= rounds) break;
        const int buf = r & 1;
        const int64_t b = (int64_t)r * ROUND + (int64_t)threadIdx.x * VEC;
        int64_t v = 0;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            v += vr[r][k];
            vmax = max(vmax, vr[r][k]);
            over += vr[r][k] > TCAP;
        }
        int64_t x = v;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int64_t y = __shfl_up(x, d, 64);
            if (lane >= d) x += y;
        }
        if (lane == 63) part[buf][w] = x;
        __syncthreads();
        if (w == 0) {
            int64_t t = lane < NW ? part[buf][lane] : 0;
#pragma unroll
            for (int d = 1; d < NW; d <<= 1) {
                const int64_t y = __shfl_up(t, d, 64);
                if (lane >= d) t += y;
            }
            if (lane < NW) part[buf][lane] = t;
        }
        __syncthreads();
        int64_t run = carry + (w > 0 ? part[buf][w - 1] : 0) + x - v;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            if (b + k < n) out[b + k] = (OutT)run;
            run += vr[r][k];
        }
        carry += part[buf][NW - 1];
    }
    int2 ws = make_int2(0, 0);
    if (stats) ws = block_degree_stats<SMALL_THREADS>(vmax, over, red, stats);
    if (threadIdx.x == 0) {
        out[n] = (OutT)carry;
        if (total_copy) *total_copy = carry;
        if (rec) {
            // one workgroup, and the caller zeroed stats: the workgroup's pair
            // is the final value; err was set by earlier kernels
            const int32_t e0 = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            rec[0] = (int64_t)(uint32_t)e0 | ((int64_t)(uint32_t)ws.x << 32);
            rec[1] = ws.y;
            rec[2] = carry;
            __hip_atomic_store(rec + 3, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    }
}

template <typename OutT>
__global__ __launch_bounds__(SCAN_THREADS) void k_scan_tile(int64_t n, const int32_t *__restrict__ in,
                                                            OutT *__restrict__ out, int64_t *__restrict__ sums,
                                                            int32_t *__restrict__ stats) {
    __shared__ int64_t part[SCAN_THREADS / 64];
    __shared__ int red[2 * SCAN_THREADS / 64];
    const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
    int64_t v[SCAN_ITEMS], s = 0, total;
    int vmax = 0, over = 0;
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        v[k] = (base + k < n) ? (int64_t)in[base + k] : 0;
        s += v[k];
        vmax = max(vmax, (int)v[k]);
        over += v[k] > TCAP;
    }
    if (stats) block_degree_stats<SCAN_THREADS>(vmax, over, red, stats);
    int64_t run = block_exclusive<SCAN_THREADS>(s, part, &total); // exclusive within the tile
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        if (base + k < n) out[base + k] = (OutT)run;
        run += v[k];
    }
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// single workgroup: exclusive scan of the tile sums in place; total -> *total
__global__ __launch_bounds__(1024) void k_scan_sums(int64_t m, int64_t *__restrict__ sums,
                                                    int64_t *__restrict__ total) {
    __shared__ int64_t part[1024 / 64];
    const int per = (int)((m + 1023) / 1024);
    const int64_t base = (int64_t)threadIdx.x * per;
    int64_t s = 0, tot;
    for (int k = 0; k < per; ++k)
        if (base + k < m) s += sums[base + k];
    int64_t run = block_exclusive<1024>(s, part, &tot);
    for (int k = 0; k < per; ++k)
        if (base + k < m) {
            int64_t v = sums[base + k];
            sums[base + k] = run;
            run += v;
        }
    if (threadIdx.x == 0) *total = tot;
}

template <typename OutT>
__global__ void k_scan_add(int64_t n, OutT *__restrict__ out, const int64_t *__restrict__ sums,
                           const int64_t *__restrict__ total, int64_t *__restrict__ total_copy) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] += (OutT)sums[i / SCAN_TILE];
    if (i == n) {
        out[n] = (OutT)*total;
        if (total_copy) *total_copy = *total;
    }
}

// stats (may be NULL): [0] max of in, [1] count of in > TCAP, both folded in
// with atomics (the caller zeroes them)
// rec, err, seq: k_scan_small's host record, written only by the one-workgroup
// scan (n <= SMALL_MAX); *rec_written says whether it will be
template <typename OutT>
hipError_t exclusive_scan(int64_t n, const int32_t *in, OutT *out, int64_t *tmp, int64_t *total_copy, int32_t *stats,
                          hipStream_t st, const int32_t *err = nullptr, int64_t *rec = nullptr, int64_t seq = 0,
                          bool *rec_written = nullptr) {
    if (rec_written) *rec_written = false;
    if (n <= SMALL_MAX) {
        const bool r = rec && stats && err;
        hipLaunchKernelGGL(k_scan_small<OutT>, dim3(1), dim3(SMALL_THREADS), 0, st, n, in, out, total_copy, stats,
                           err, r ? rec : nullptr, seq);
        if (rec_written) *rec_written = r;
        return hipGetLastError();
    }
    const int64_t tiles = (n + SCAN_TILE - 1) / SCAN_TILE;
    // tmp layout: [tiles] tile sums, then [1] total
    hipLaunchKernelGGL(k_scan_tile<OutT>, dim3((unsigned)tiles), dim3(SCAN_THREADS), 0, st, n, in, out, tmp, stats);
    hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(1024), 0, st, tiles, tmp, tmp + tiles);
    hipLaunchKernelGGL(k_scan_add<OutT>, dim3((unsigned)((n + 1 + 255) / 256)), dim3(256), 0, st, n, out, tmp,
                       tmp + tiles, total_copy);
    return hipGetLastError();
}

unsigned blocks_for(int64_t n, int bs) { return (unsigned)((n + bs - 1) / bs); }

// ---- periodic images ----
template <typename PosT>
__device__ __forceinline__ void frac_of(const PosT *pos, int64_t i, const PeriodicCell &C, double *f) {
    const double r[3] = {(double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]};
    for (int k = 0; k < 3; ++k) f[k] = (r[0] * C.B[k] + r[1] * C.B[3 + k]) + r[2] * C.B[6 + k];
}

// image index range of atom i per direction: f + n within [lo - eps, hi + eps]
__device__ __forceinline__ void image_range(const double *f, const PeriodicCell &C, const double *lohi, int *nlo,
                                            int *nhi) {
    for (int k = 0; k < 3; ++k) {
        const double a = lohi[k] - C.eps[k] - f[k], b = lohi[3 + k] + C.eps[k] - f[k];
        // (a non-finite coordinate gets no images; the range is capped far above any
        // count the atom limit allows, so the capped total is rejected on the host)
        if (C.pbc[k] && isfinite(a) && isfinite(b)) {
            nlo[k] = (int)fmax(ceil(a), -1e6);
            nhi[k] = (int)fmin(floor(b), 1e6);
        } else {
            nlo[k] = nhi[k] = 0;
        }
    }
}

template <typename PosT>
__global__ __launch_bounds__(1024) void k_frac_bounds(int64_t n, const PosT *__restrict__ pos, PeriodicCell C,
                                                      double *__restrict__ lohi) {
    __shared__ double red[6][1024];
    double lo[3] = {INFINITY, INFINITY, INFINITY}, hi[3] = {-INFINITY, -INFINITY, -INFINITY};
    for (int64_t i = threadIdx.x; i < n; i += 1024) {
        double f[3];
        frac_of(pos, i, C, f);
        for (int k = 0; k < 3; ++k) {
            lo[k] = fmin(lo[k], f[k]);
            hi[k] = fmax(hi[k], f[k]);
        }
    }
    for (int k = 0; k < 3; ++k) {
        red[k][threadIdx.x] = lo[k];
        red[3 + k][threadIdx.x] = hi[k];
    }
    __syncthreads();
    for (int off = 512; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off)
            for (int k = 0; k < 3; ++k) {
                red[k][threadIdx.x] = fmin(red[k][threadIdx.x], red[k][threadIdx.x + off]);
                red[3 + k][threadIdx.x] = fmax(red[3 + k][threadIdx.x], red[3 + k][threadIdx.x + off]);
            }
        __syncthreads();
    }
    if (threadIdx.x < 6) lohi[threadIdx.x] = red[threadIdx.x][0];
}

template <typename PosT>
__global__ void k_image_count(int64_t n, const PosT *__restrict__ pos, PeriodicCell C, const double *__restrict__ lohi,
                              int32_t *__restrict__ cnt) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    double f[3];
    int lo[3], hi[3];
    frac_of(pos, i, C, f);
    image_range(f, C, lohi, lo, hi);
    // n = 0 is always in range (lo <= f <= hi)
    const int64_t m = (int64_t)(hi[0] - lo[0] + 1) * (hi[1] - lo[1] + 1) * (hi[2] - lo[2] + 1) - 1;
    cnt[i] = (int32_t)(m < INT32_MAX ? m : INT32_MAX);
}

template <typename PosT>
__global__ void k_image_fill(int64_t n, const PosT *__restrict__ pos, const int32_t *__restrict__ Z, PeriodicCell C,
                             const double *__restrict__ lohi, const int64_t *__restrict__ start,
                             PosT *__restrict__ pos_ext, int32_t *__restrict__ Z_ext, int32_t *__restrict__ map_atom,
                             int32_t *__restrict__ map_img) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const double r[3] = {(double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]};
    for (int d = 0; d < 3; ++d) pos_ext[3 * i + d] = pos[3 * i + d];
    Z_ext[i] = Z[i];
    map_atom[i] = (int32_t)i;
    map_img[3 * i] = map_img[3 * i + 1] = map_img[3 * i + 2] = 0;
    double f[3];
    int lo[3], hi[3];
    frac_of(pos, i, C, f);
    image_range(f, C, lohi, lo, hi);
    int64_t x = n + start[i];
    for (int a = lo[0]; a <= hi[0]; ++a)
        for (int b = lo[1]; b <= hi[1]; ++b)
            for (int c = lo[2]; c <= hi[2]; ++c) {
                if (a == 0 && b == 0 && c == 0) continue;
                for (int d = 0; d < 3; ++d) {
                    double sft = (double)a * C.M[d];
                    sft = sft + (double)b * C.M[3 + d];
                    sft = sft + (double)c * C.M[6 + d];
                    pos_ext[3 * x + d] = (PosT)(r[d] + sft);
                }
                Z_ext[x] = Z[i];
                map_atom[x] = (int32_t)i;
                map_img[3 * x] = a;
                map_img[3 * x + 1] = b;
                map_img[3 * x + 2] = c;
                ++x;
            }
}

__global__ void k_iota(int64_t n, int32_t *__restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] = (int32_t)i;
}

__global__ void k_map_edges(int64_t E, const int32_t *__restrict__ cols, const int32_t *__restrict__ map,
                            const int32_t *__restrict__ map_img, int32_t *__restrict__ out,
                            int32_t *__restrict__ img_out) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= E) return;
    const int32_t x = cols[e];
    if (out) out[e] = map ? map[x] : x;
    if (img_out)
        for (int d = 0; d < 3; ++d) img_out[3 * e + d] = map_img ? map_img[3 * x + d] : 0;
}


struct Geometry {
    double inv_h, rc2, lim2;
    uint32_t mask;
    int b;
};

Geometry geometry(const NbrWork &w, double r_cut) {
    Geometry g;
    const double h = r_cut * CELL_PAD;
    g.inv_h = 1.0 / h;
    g.rc2 = r_cut * r_cut;
    // a cell is skipped when its box is farther than r_cut from the center,
    // tested in cell units with a relative margin far above rounding
    g.lim2 = (r_cut * g.inv_h) * (r_cut * g.inv_h) * (1.0 + 1e-6);
    g.mask = (uint32_t)(w.H - 1);
    int k = 0;
    while ((int64_t(1) << k) < w.H) ++k;
    g.b = std::min(10, k / 3);
    return g;
}

} // namespace

hipError_t nbr_phase1(const NbrWork &w, int64_t n_atoms, int64_t center_bound, const void *pos, bool pos64,
                      const int32_t *Z, const int8_t *lut, uint8_t *spec, int64_t nc, const int32_t *centers,
                      double r_cut, int64_t *row_ptr, hipStream_t st, int64_t *rec, int64_t seq,
                      bool *rec_written) {
    const Geometry g = geometry(w, r_cut);
    hipError_t e;
    // flags, density work counters and both bucket arrays are one zeroed block
    if ((e = hipMemsetAsync(w.zero, 0, w.zero_bytes, st)) != hipSuccess) return e;
    const unsigned gb = blocks_for(n_atoms, 256);
    if (pos64)
        hipLaunchKernelGGL(k_prepare<double>, dim3(gb), dim3(256), 0, st, n_atoms, (const double *)pos, Z, lut, spec,
                           w.atom_cell, w.bucket_count, g.mask, g.b, g.inv_h, w.flags);
    else
        hipLaunchKernelGGL(k_prepare<float>, dim3(gb), dim3(256), 0, st, n_atoms, (const float *)pos, Z, lut, spec,
                           w.atom_cell, w.bucket_count, g.mask, g.b, g.inv_h, w.flags);
    if ((e = exclusive_scan<int32_t>(w.H, w.bucket_count, w.bucket_start, w.scan_tmp, nullptr, nullptr, st)) !=
        hipSuccess)
        return e;
    const unsigned gc = blocks_for(nc, NBR_WAVES);
    if (pos64) {
        hipLaunchKernelGGL(k_bucket_fill<double>, dim3(gb), dim3(256), 0, st, n_atoms, (const double *)pos, spec,
                           w.atom_cell, w.bucket_start, w.bucket_fill, (double4 *)w.sorted_rec, w.sorted_spec);
        hipLaunchKernelGGL(k_collect<double>, dim3(gc), dim3(64 * NBR_WAVES), 0, st, center_bound, nc, centers,
                           (const double *)pos, w.bucket_start, (const double4 *)w.sorted_rec,
                           w.sorted_spec, g.mask, g.b, g.inv_h, g.lim2, g.rc2, w.deg, w.slots, w.flags);
    } else {
        hipLaunchKernelGGL(k_bucket_fill<float>, dim3(gb), dim3(256), 0, st, n_atoms, (const float *)pos, spec,
                           w.atom_cell, w.bucket_start, w.bucket_fill, (float4 *)w.sorted_rec, w.sorted_spec);
        hipLaunchKernelGGL(k_collect<float>, dim3(gc), dim3(64 * NBR_WAVES), 0, st, center_bound, nc, centers,
                           (const float *)pos, w.bucket_start, (const float4 *)w.sorted_rec,
                           w.sorted_spec, g.mask, g.b, g.inv_h, g.lim2, g.rc2, w.deg, w.slots, w.flags);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return exclusive_scan<int64_t>(nc, w.deg, row_ptr, w.scan_tmp, (int64_t *)(w.flags + 4), w.flags + 1, st,
                                   w.flags, rec, seq, rec_written);
}

hipError_t periodic_count(int64_t n, const void *pos, bool pos64, const PeriodicCell &C, double *lohi, int32_t *cnt,
                          hipStream_t st) {
    if (pos64) {
        hipLaunchKernelGGL(k_frac_bounds<double>, dim3(1), dim3(1024), 0, st, n, (const double *)pos, C, lohi);
        hipLaunchKernelGGL(k_image_count<double>, dim3(blocks_for(n, 256)), dim3(256), 0, st, n, (const double *)pos,
                           C, lohi, cnt);
    } else {
        hipLaunchKernelGGL(k_frac_bounds<float>, dim3(1), dim3(1024), 0, st, n, (const float *)pos, C, lohi);
        hipLaunchKernelGGL(k_image_count<float>, dim3(blocks_for(n, 256)), dim3(256), 0, st, n, (const float *)pos, C,
                           lohi, cnt);
    }
    return hipGetLastError();
}

hipError_t periodic_fill(int64_t n, const void *pos, bool pos64, const int32_t *Z, const PeriodicCell &C,
                         const double *lohi, const int64_t *start, void *pos_ext, int32_t *Z_ext, int32_t *map_atom,
                         int32_t *map_img, hipStream_t st) {
    if (pos64)
        hipLaunchKernelGGL(k_image_fill<double>, dim3(blocks_for(n, 256)), dim3(256), 0, st, n, (const double *)pos, Z,
                           C, lohi, start, (double *)pos_ext, Z_ext, map_atom, map_img);
    else
        hipLaunchKernelGGL(k_image_fill<float>, dim3(blocks_for(n, 256)), dim3(256), 0, st, n, (const float *)pos, Z,
                           C, lohi, start, (float *)pos_ext, Z_ext, map_atom, map_img);
    return hipGetLastError();
}

hipError_t nbr_exclusive_scan(int64_t n, const int32_t *in, int64_t *out, int64_t *tmp, int64_t *total_copy,
                              hipStream_t st) {
    return exclusive_scan<int64_t>(n, in, out, tmp, total_copy, nullptr, st);
}

hipError_t fill_iota(int64_t n, int32_t *out, hipStream_t st) {
    if (n > 0) hipLaunchKernelGGL(k_iota, dim3(blocks_for(n, 256)), dim3(256), 0, st, n, out);
    return hipGetLastError();
}

hipError_t map_edges(int64_t E, const int32_t *cols, const int32_t *map, const int32_t *map_img, int32_t *out,
                     int32_t *img_out, hipStream_t st) {
    if (E > 0)
        hipLaunchKernelGGL(k_map_edges, dim3(blocks_for(E, 256)), dim3(256), 0, st, E, cols, map, map_img, out, img_out);
    return hipGetLastError();
}

hipError_t nbr_pack(const NbrWork &w, int64_t nc, const int64_t *row_ptr, int32_t *cols, int64_t cap,
                    hipStream_t st) {
    if (nc <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_pack, dim3(blocks_for(nc, 4)), dim3(256), 0, st, nc, row_ptr, w.slots, cols, cap);
    return hipGetLastError();
}

hipError_t nbr_phase2(const NbrWork &w, int64_t n_atoms, const void *pos, bool pos64, int64_t nc,
                      const int32_t *centers, double r_cut, const int64_t *row_ptr, bool long_rows, bool packed,
                      int32_t *cols, int64_t cap, hipStream_t st) {
    (void)n_atoms;
    const Geometry g = geometry(w, r_cut);
    if (!packed) hipLaunchKernelGGL(k_pack, dim3(blocks_for(nc, 4)), dim3(256), 0, st, nc, row_ptr, w.slots, cols, cap);
    if (long_rows) {
        if (pos64)
            hipLaunchKernelGGL(k_collect_long<double>, dim3((unsigned)nc), dim3(64), 0, st, nc, centers,
                               (const double *)pos, w.bucket_start, (const double4 *)w.sorted_rec,
                               w.sorted_spec, g.mask, g.b, g.inv_h, g.lim2, g.rc2, row_ptr, cols);
        else
            hipLaunchKernelGGL(k_collect_long<float>, dim3((unsigned)nc), dim3(64), 0, st, nc, centers,
                               (const float *)pos, w.bucket_start, (const float4 *)w.sorted_rec,
                               w.sorted_spec, g.mask, g.b, g.inv_h, g.lim2, g.rc2, row_ptr, cols);
    }
    return hipGetLastError();
}

} // namespace soap
