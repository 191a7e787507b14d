// voxelize.hip -- sparse voxelization (Sec. 3.3, Eq. 1 and Eq. 2).
//
// 1. k_vq_quantize: every point's key floor(p / v) (Eq. 1), packed; per block the
//    per-field minima / maxima of the keys for the sort's compaction.  The same
//    launch clears the status header and the hash table and, in a block call,
//    packs the layers' weights;
// 2. the points are radix-sorted by key (radix.hip): the canonical (b, x, y, z)
//    order of the voxels and the grouping of the points by voxel in one step;
// 3. k_vq_segments: a voxel starts wherever the sorted key changes.  A scan of
//    those starts numbers the voxels; each voxel's coordinates and its first
//    point are written at its start, and every point gets its voxel index;
// 4. k_vox_mean: each voxel sums its own points (fp64) and writes its mean once
//    -- no float atomics; blocks of their own write the counts and enter each
//    voxel into the hash table (value = its index: one insert per voxel), and
//    k_vox_mean_long sums the voxels of over 32 points with a workgroup each.
// The scatter-mean onto a given voxel set (launch_voxelize_onto) finds each
// point's voxel in the set's table instead and groups the points by a counting
// sort.
#include "spv_internal.hpp"

namespace spv {

void plan_voxelize_ws(Arena& a, VoxelizeWs& w, int64_t n) {
    int64_t nn = n > 0 ? n : 1;
    uint32_t S = table_capacity(nn);
    w.table = take_table(a, S);
    plan_radix_ws(a, w.rs, nn);
    w.seg = a.take<int32_t>(nn + 1);
    w.fill = a.take<int32_t>(nn);
    w.plist = a.take<int32_t>(nn);
    w.longv = a.take<int32_t>(nn);
    w.scan_tmp = a.take<int32_t>(scan_tmp_entries(nn));
}

// Eq. 1 for point k: its packed key with the quantized (b, q), or kEmpty with
// the status flag raised for a non-finite or out-of-range point
__device__ inline uint64_t point_key(Header* h, const float* xyz, const int32_t* batch, int64_t k, float v,
                                     int (&q)[3], int& b) {
    const float p[3] = {xyz[3 * k], xyz[3 * k + 1], xyz[3 * k + 2]};
    b = batch ? batch[k] : 0;
    const bool finite = isfinite(p[0]) && isfinite(p[1]) && isfinite(p[2]);
    bool inrange = b >= 0 && b <= kBatchMax;
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        const float a = p[d] / v;  // IEEE single-precision, correctly rounded
        const float f = floorf(a);
        inrange = inrange && isfinite(a) && f >= (float)kCoordMin && f <= (float)kCoordMax;
        q[d] = inrange ? (int)f : 0;
    }
    if (!finite) {
        raise_flag(h, kFlagNonfinite);
        return kEmpty;
    }
    if (!inrange) {
        raise_flag(h, kFlagRange);
        return kEmpty;
    }
    return pack_key(b, q[0], q[1], q[2]);
}

// Eq. 1 for point k without side effects: the packed key, or kEmpty with
// *why = 1 (a non-finite coordinate) or 2 (a voxel outside the key range)
__device__ inline uint64_t point_key_of(const float* xyz, const int32_t* batch, int64_t k, float v, int& why) {
    const float p[3] = {xyz[3 * k], xyz[3 * k + 1], xyz[3 * k + 2]};
    const int b = batch ? batch[k] : 0;
    const bool finite = isfinite(p[0]) && isfinite(p[1]) && isfinite(p[2]);
    bool inrange = b >= 0 && b <= kBatchMax;
    int q[3];
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        const float a = p[d] / v;  // IEEE single-precision, correctly rounded
        const float f = floorf(a);
        inrange = inrange && isfinite(a) && f >= (float)kCoordMin && f <= (float)kCoordMax;
        q[d] = inrange ? (int)f : 0;
    }
    why = !finite ? 1 : (!inrange ? 2 : 0);
    return why ? kEmpty : pack_key(b, q[0], q[1], q[2]);
}

// What the first launch of a voxelization clears and packs besides Eq. 1.
struct VoxFirst {
    Header* h;
    Table table;      // the hash table -> empty
    uint32_t* zero;   // the sort's counters and look-back words -> 0
    int64_t nzero;
    int njobs;
    PackJob job[kMaxPackJobs];
    int npack;        // the grid's last npack blocks run the packings, the others the rest
};

// Eq. 1 per point into the sort's key buffer, with the block's record (per-field
// minima / maxima of its valid keys, its non-finite and out-of-range counts).
// Grid-stride alongside: the header, the table, the sort's scratch.  The weight
// packings run in blocks of their own at the end of the grid, so that their
// gathers' round trip does not delay the quantization.
__global__ __launch_bounds__(kRsProducerBlock) void k_vq_quantize(VoxFirst f, const float* xyz,
                                                                  const int32_t* batch, int64_t n, float v,
                                                                  uint64_t* keys, int32_t* rec) {
    const int nqb = (int)gridDim.x - f.npack;  // the quantizing blocks
    if ((int)blockIdx.x >= nqb) {
        const int64_t tp = (blockIdx.x - nqb) * (int64_t)blockDim.x + threadIdx.x;
        const int64_t sp = (int64_t)f.npack * blockDim.x;
        for (int j = 0; j < f.njobs; ++j) {
            const PackJob& q = f.job[j];
            for (int64_t t = tp; t < q.total; t += sp)
                q.wpack[t] = pack_fragment(q.W, q.Cin, q.Cout, q.ldc, q.ldcol, q.ldk, q.KCH, q.NB, t);
        }
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        f.h->status = 0;
        f.h->m = 0;
        for (int i = 0; i < 4; ++i) f.h->aux[i] = 0;
    }
    const int64_t t0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)nqb * blockDim.x;
    const int64_t nkw = (int64_t)(f.table.mask + 1) / 2;  // 16-byte runs of keys: 2 per bucket
    for (int64_t i = t0; i < nkw; i += stride)
        *(u64x2*)(f.table.keys + 8 * (i >> 1) + 2 * (i & 1)) = u64x2{kEmpty, kEmpty};
    for (int64_t i = t0; i < f.nzero; i += stride) f.zero[i] = 0u;

    int mn[4] = {0x7fffffff, 0x7fffffff, 0x7fffffff, 0x7fffffff};
    int mx[4] = {(int)0x80000000, (int)0x80000000, (int)0x80000000, (int)0x80000000};
    uint32_t nonfin = 0, range = 0;
    for (int64_t k = t0; k < n; k += stride) {  // grid-stride: one record per block, however large n
        int why = 0;
        const uint64_t key = point_key_of(xyz, batch, k, v, why);
        keys[k] = key;
        if (!why) {
            const int fl[4] = {key_b(key), key_x(key), key_y(key), key_z(key)};
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                mn[d] = min(mn[d], fl[d]);
                mx[d] = max(mx[d], fl[d]);
            }
        }
        nonfin += why == 1 ? 1u : 0u;
        range += why == 2 ? 1u : 0u;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        nonfin += __shfl_xor(nonfin, o, 64);
        range += __shfl_xor(range, o, 64);
    }
    __shared__ uint32_t bad[2];
    if (threadIdx.x < 2) bad[threadIdx.x] = 0;
    block_minmax_record(mn, mx, rec + (size_t)kRsRecWords * blockIdx.x);  // synchronizes the block
    if ((threadIdx.x & 63) == 0 && (nonfin | range)) {
        atomicAdd(&bad[0], nonfin);  // LDS
        atomicAdd(&bad[1], range);
    }
    __syncthreads();
    if (threadIdx.x < 2) rec[(size_t)kRsRecWords * blockIdx.x + 8 + threadIdx.x] = (int32_t)bad[threadIdx.x];
}

// Exclusive prefix of a tile's count over the tiles before it, by one whole
// wave: 64 predecessors' status words per round, nearest first, up to the
// nearest one holding an inclusive prefix (same protocol as the sort's passes).
__device__ inline uint32_t vq_lookback(const uint64_t* stat, int64_t tile, bool& stalled) {
    const int lane = threadIdx.x & 63;
    uint32_t excl = 0, spins = 0;
    int64_t j = tile - 1;
    while (j >= 0) {
        const uint64_t s = (j - lane >= 0)
                               ? __hip_atomic_load(stat + (j - lane), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                               : (2ull << 62);
        const uint32_t f = (uint32_t)(s >> 62);
        const uint64_t notready = __ballot(f == 0), inc = __ballot(f == 2);
        const int fi = inc ? __builtin_ctzll(inc) : 64;                // nearest inclusive prefix
        const uint64_t upto = fi < 63 ? ((2ull << fi) - 1ull) : ~0ull;  // lanes 0 .. fi
        int take;
        bool done;
        if (notready & upto) {  // consume the ready lanes before the first one not written yet
            take = __builtin_ctzll(notready & upto);
            done = false;
        } else {
            take = fi < 64 ? fi + 1 : 64;
            done = fi < 64;
        }
        uint32_t val = lane < take ? (uint32_t)s : 0u;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) val += __shfl_xor(val, o, 64);
        excl += val;
        if (done) break;
        j -= take;
        if (take == 0) {
            if (++spins > (1u << 22)) {
                stalled = true;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    return excl;
}

// Voxels from the sorted keys: position i starts a voxel when its key differs
// from position i-1's.  Tile-local ranks of the starts (position order: round,
// wave, lane) plus the look-back give every start its voxel index; there the
// voxel's coordinates and its first sorted position (seg) are written, and
// every point receives its voxel's index (invalid points, sorted last, get -1).
// The last tile writes m.  (The per-voxel kernel that follows inserts each
// voxel into the hash table: one insert per voxel, spread over the whole chip.)
__global__ __launch_bounds__(kRsThreads) void k_vq_segments(RadixWs rs, Header* h, int64_t n, int64_t ntiles,
                                                            int32_t* coords, int32_t* pt2vox, int32_t* seg,
                                                            int32_t* plist, int64_t* m_dev) {
    constexpr int I = kRsItems, NWV = kRsThreads / 64;
    __shared__ uint32_t s_tile, s_excl;
    __shared__ uint32_t wcnt[I][NWV];  // starts per (round, wave), then their exclusive prefix in the tile
    __shared__ uint32_t s_tot;
    const SortStats st = *rs.st;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) s_tile = atomicAdd(&rs.ctr[8], 1u);
    const uint64_t* K = rs_keys(rs, st);
    const uint32_t* V = rs_vals(rs, st);
    const int64_t nvalid = n - (int64_t)st.n_invalid;
    __syncthreads();
    const int64_t tile = s_tile;
    const int64_t base = tile * kRsTile;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint64_t key[I];
    uint32_t hb = 0;  // bit r: the position of round r starts a voxel
    uint32_t rk[I];   // rank of that start among its wave's starts of the round
#pragma unroll
    for (int r = 0; r < I; ++r) {
        const int64_t i = base + r * kRsThreads + tid;
        key[r] = i < nvalid ? K[i] : kEmpty;
        const uint64_t pk = (i > 0 && i - 1 < nvalid) ? K[i - 1] : kEmpty;
        const bool hd = i < nvalid && (i == 0 || key[r] != pk);
        const uint64_t bal = __ballot(hd);
        hb |= (hd ? 1u : 0u) << r;
        rk[r] = (uint32_t)__popcll(bal & lt);
        if (lane == 0) wcnt[r][wave] = (uint32_t)__popcll(bal);
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t run = 0;
        for (int r = 0; r < I; ++r)
            for (int q = 0; q < NWV; ++q) {
                const uint32_t c = wcnt[r][q];
                wcnt[r][q] = run;
                run += c;
            }
        s_tot = run;
    }
    __syncthreads();
    const uint32_t tot = s_tot;
    uint64_t* stat = rs_consumer_status(rs);
    if (tid < 64) {
        bool stalled = false;
        uint32_t excl = 0;
        if (tile == 0) {
            if (tid == 0)
                __hip_atomic_store(stat, (2ull << 62) | tot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            if (tid == 0)
                __hip_atomic_store(stat + tile, (1ull << 62) | tot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            excl = vq_lookback(stat, tile, stalled);
            if (tid == 0)
                __hip_atomic_store(stat + tile, (2ull << 62) | (uint64_t)(excl + tot), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
        if (tid == 0) {
            s_excl = excl;
            if (stalled) raise_flag(h, kFlagInternal);
            if (tile == 0) {  // invalid points (their keys were counted by the sort) make the call report
                if (st.invalid_kinds & 1u) raise_flag(h, kFlagNonfinite);
                if (st.invalid_kinds & 2u) raise_flag(h, kFlagRange);
            }
        }
    }
    __syncthreads();
    const int64_t excl = s_excl;
#pragma unroll
    for (int r = 0; r < I; ++r) {
        const int64_t i = base + r * kRsThreads + tid;
        if (i >= n) continue;
        const uint32_t k = V[i];
        plist[i] = (int32_t)k;
        if (i >= nvalid) {
            pt2vox[k] = -1;
            continue;
        }
        // the starts before this position; a start takes the next index, any
        // other position the index of its last start
        const bool hd = (hb >> r) & 1u;
        const int32_t vid = (int32_t)(excl + wcnt[r][wave] + rk[r]) - (hd ? 0 : 1);
        if (hd) {
            const uint64_t pk = rs_expand(key[r], st);
            int32_t* cv = coords + 4 * (int64_t)vid;
            cv[0] = key_b(pk);
            cv[1] = key_x(pk);
            cv[2] = key_y(pk);
            cv[3] = key_z(pk);
            seg[vid] = (int32_t)i;
        }
        pt2vox[k] = vid;
    }
    if (tile == ntiles - 1 && tid == 0) {  // the voxel count, after the last tile's look-back
        const int64_t m = excl + tot;
        seg[m] = (int32_t)nvalid;
        h->m = m;
        if (m_dev) *m_dev = m;
    }
}

// Voxel v's hash-table entry (key of coords[v], value v).  Every key is new, so
// the first compare-and-swap almost always claims its slot.
__device__ inline void vq_insert(Header* h, Table t, const int32_t* coords, int64_t v) {
    const int32_t* c = coords + 4 * v;
    uint32_t slot;
    const int r = table_insert(t, pack_key(c[0], c[1], c[2], c[3]), &slot);
    if (r > 0) *slot_val(t, slot) = (int32_t)v;
    else raise_flag(h, r < 0 ? kFlagTableFull : kFlagDuplicate);
}

// N_m = seg[v + 1] - seg[v] and the table entry when there are no features to average
__global__ void k_vq_counts(Header* h, int64_t cap, const int32_t* seg, int32_t* counts, Table t,
                            const int32_t* coords, int32_t* nbr_upper) {
    int64_t m = h->m;
    if (m > cap) m = cap;
    const int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (v >= m) return;
    counts[v] = seg[v + 1] - seg[v];
    vq_insert(h, t, coords, v);
    if (nbr_upper) clear_nbr_upper(nbr_upper, v);
}

// every point's voxel index, read at the table slot its insert found
// Runs of equal voxel ids in consecutive lanes (points of a sweep arrive in scan
// order, so a coarse voxel's points are mostly consecutive): one atomic per run,
// by its first lane, instead of one per point -- a stride-16 voxel can hold 10^3
// points.  run_of gives a lane its run's first lane and the run's length.
__device__ inline void run_of(int32_t v, int& first, int& len) {
    const int lane = threadIdx.x & 63;
    const int32_t prev = __shfl_up(v, 1, 64);
    const uint64_t heads = __ballot(lane == 0 || prev != v);
    first = 63 - __clzll(heads & (~0ull >> (63 - lane)));
    const uint64_t later = heads & ~((2ull << first) - 1ull);  // heads after the run's first lane
    len = (later ? __builtin_ctzll(later) : 64) - first;
}

__global__ void k_vox_fill(const int32_t* pt2vox, int64_t n, const int32_t* seg, int32_t* fill, int32_t* plist) {
    const int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int32_t v = k < n ? pt2vox[k] : -1;
    int first, len;
    run_of(v, first, len);
    const int lane = threadIdx.x & 63;
    int base = 0;
    if (v >= 0 && lane == first) base = atomicAdd(&fill[v], len);
    base = __shfl(base, first, 64);
    if (v >= 0) plist[seg[v] + base + (lane - first)] = (int32_t)k;
}

// Scatter-mean onto a given voxel set: each point's voxel index is found in
// the table of that set (-1 when its voxel is not in it), one probe per run of
// equal keys in the wave, and N_m is counted as in k_vox_lookup.
__global__ void k_vox_locate(Header* h, Table t, const float* xyz, const int32_t* batch, int64_t n, float v,
                             int32_t* pt2vox, int32_t* counts) {
    const int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    uint64_t key = kEmpty;
    int q[3];
    int b;
    if (k < n) key = point_key(h, xyz, batch, k, v, q, b);
    const int lane = threadIdx.x & 63;
    const uint64_t prev_key = __shfl_up(key, 1, 64);
    const bool head = key != kEmpty && (lane == 0 || prev_key != key);
    const int32_t found = head ? table_find(t, key) : -1;
    const uint64_t heads = __ballot(head) & (~0ull >> (63 - lane));
    const int src = heads ? 63 - __clzll(heads) : lane;
    const int32_t run_found = __shfl(found, src, 64);
    const int32_t vox = key == kEmpty ? -1 : run_found;
    if (k < n) pt2vox[k] = vox;
    int first, len;
    run_of(vox, first, len);
    if (vox >= 0 && lane == first) atomicAdd(&counts[vox], len);
}

__global__ void k_vox_zero(int32_t* a, int32_t* b, int64_t m) {
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i < m) {
        a[i] = 0;
        b[i] = 0;
    }
}


// Eq. 2: one thread per (voxel, VEC consecutive channels).  The points are
// summed in fp64 -- exact for 16-bit features of ordinary range, so the result
// does not depend on the order in which they were grouped -- and the mean is
// rounded once to the storage type.  A voxel of more than `run` points (a
// coarse grid near the sensor holds up to ~10^3) would keep one thread on a
// long chain of dependent loads: its first thread appends it to `longv` (count
// in h->aux[0]) and k_vox_mean_long sums it with a whole workgroup.
template <int DT, int VEC>
__device__ inline void mean_add(double (&acc)[VEC], const void* feat, int64_t row) {
    if constexpr (VEC == 8) {
        uint4 u = *(const uint4*)((const uint16_t*)feat + row);
        uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            acc[2 * j] += (double)from16<DT>(w[j] & 0xFFFF);
            acc[2 * j + 1] += (double)from16<DT>(w[j] >> 16);
        }
    } else if constexpr (VEC == 4) {
        float4 f = *(const float4*)((const float*)feat + row);
        acc[0] += (double)f.x;
        acc[1] += (double)f.y;
        acc[2] += (double)f.z;
        acc[3] += (double)f.w;
    } else {
        acc[0] += (double)ld_feat<DT>(feat, row);
    }
}

// The points lo, lo + step, ... < hi of a voxel's list into acc, in list
// order; U rows' indices, then their features, are loaded before any is
// added, so a long voxel costs 1/U of the dependent round trips.  (The
// per-voxel kernel takes U = 2: its voxels are short, and U = 4 cost it two
// waves per SIMD of occupancy.)
template <int DT, int VEC, int U>
__device__ inline void mean_add_range(double (&acc)[VEC], const void* feat, const int32_t* plist, int C, int ch,
                                      int32_t lo, int32_t hi, int32_t step) {
    int32_t p = lo;
    for (; p + (U - 1) * step < hi; p += U * step) {
        int64_t row[U];
#pragma unroll
        for (int u = 0; u < U; ++u) row[u] = (int64_t)plist[p + u * step] * C + ch;
        if constexpr (VEC == 8) {
            uint4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = *(const uint4*)((const uint16_t*)feat + row[u]);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc[2 * j] += (double)from16<DT>(w[j] & 0xFFFF);
                    acc[2 * j + 1] += (double)from16<DT>(w[j] >> 16);
                }
            }
        } else if constexpr (VEC == 4) {
            float4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = *(const float4*)((const float*)feat + row[u]);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                acc[0] += (double)v[u].x;
                acc[1] += (double)v[u].y;
                acc[2] += (double)v[u].z;
                acc[3] += (double)v[u].w;
            }
        } else {
            float v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = ld_feat<DT>(feat, row[u]);
#pragma unroll
            for (int u = 0; u < U; ++u) acc[0] += (double)v[u];
        }
    }
    for (; p < hi; p += step) mean_add<DT, VEC>(acc, feat, (int64_t)plist[p] * C + ch);
}

template <int DT, int VEC>
__device__ inline void mean_store(const double (&acc)[VEC], double N, void* vfeat, int64_t orow) {
    if (N < 1.0) N = 1.0;  // a given voxel no point falls into (scatter-mean onto a set): mean 0
    // the quotients acc / N; for N a power of two (1 for most voxels) the product
    // with 1 / N, which is exact and so the same value, without the division
    double q[VEC];
    const int ni = (int)N;
    if ((ni & (ni - 1)) == 0) {
        const double r = 1.0 / N;
#pragma unroll
        for (int j = 0; j < VEC; ++j) q[j] = acc[j] * r;
    } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) q[j] = acc[j] / N;
    }
    if constexpr (VEC == 8) {
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            w[j] = (uint32_t)to16<DT>(f64_to_f32_odd(q[2 * j])) |
                   ((uint32_t)to16<DT>(f64_to_f32_odd(q[2 * j + 1])) << 16);
        *(uint4*)((uint16_t*)vfeat + orow) = make_uint4(w[0], w[1], w[2], w[3]);
    } else if constexpr (VEC == 4) {
        *(float4*)((float*)vfeat + orow) = make_float4((float)q[0], (float)q[1], (float)q[2], (float)q[3]);
    } else {
        if constexpr (DT == SPV_F32) st_feat<DT>(vfeat, orow, (float)q[0]);
        else st_feat<DT>(vfeat, orow, f64_to_f32_odd(q[0]));
    }
}

// ins (voxelization only): the table to enter each voxel into, from coords
template <int DT, int VEC>
__global__ void k_vox_mean(Header* h, int64_t cap, const int32_t* seg, const int32_t* plist, const void* feat,
                           int C, void* vfeat, int run, int32_t* longv, int32_t* counts, Table ins,
                           const int32_t* coords, int ins_first, int32_t* nbr_upper) {
    int64_t m = h->m;
    if (m > cap) m = cap;
    const int nch = C / VEC;
    // With counts, blocks of their own count voxels and enter them into the
    // table, so that their compare-and-swap round trips overlap the averaging
    // blocks instead of holding them up: with ins_first the first nb blocks
    // (a grid that fits the chip at once), otherwise one block in every
    // nch + 1, spread evenly through a grid that runs in rounds.
    int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (counts) {
        const int64_t nb = (int64_t)gridDim.x / (nch + 1);
        int64_t grp, r;
        if (ins_first) {
            grp = blockIdx.x < nb ? blockIdx.x : (blockIdx.x - nb) / nch;
            r = blockIdx.x < nb ? 0 : (blockIdx.x - nb) - grp * nch + 1;
        } else {
            grp = blockIdx.x / (nch + 1);
            r = blockIdx.x - grp * (nch + 1);
        }
        if (r == 0) {
            const int64_t vox = grp * blockDim.x + threadIdx.x;
            if (vox >= m) return;
            counts[vox] = seg[vox + 1] - seg[vox];  // N_m
            vq_insert(h, ins, coords, vox);
            if (nbr_upper) clear_nbr_upper(nbr_upper, vox);
            return;
        }
        t = (grp * nch + r - 1) * blockDim.x + threadIdx.x;
    }
    const int64_t vox = t / nch;
    const int slot = (int)(t - vox * nch);
    if (vox >= m) return;
    int32_t lo = seg[vox], hi = seg[vox + 1];
    const int ch = slot * VEC;
    if (hi - lo > run) {
        if (ch == 0) longv[atomicAdd((unsigned long long*)&h->aux[0], 1ull)] = (int32_t)vox;
        return;
    }
    double acc[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] = 0.0;
    mean_add_range<DT, VEC, 2>(acc, feat, plist, C, ch, lo, hi, 1);
    mean_store<DT, VEC>(acc, (double)(hi - lo), vfeat, vox * C + ch);
}

// the long voxels: thread (slice, chunk) sums every slices-th point of the
// voxel for one VEC-channel chunk; the slices' partial sums are then added in
// slice order by the chunk's first thread (fixed order, and exact as above)
constexpr int kMeanLongThreads = 512;
template <int DT, int VEC>
__global__ __launch_bounds__(kMeanLongThreads) void k_vox_mean_long(const Header* h, int64_t cap, const int32_t* seg,
                                                                    const int32_t* plist, const void* feat, int C,
                                                                    void* vfeat, const int32_t* longv) {
    __shared__ double red[kMeanLongThreads][VEC];
    int64_t nl = h->aux[0];
    if (nl > cap) nl = cap;
    const int nch = C / VEC;
    const int slices = kMeanLongThreads / nch;  // >= 2: the host takes this path only then
    const int tch = threadIdx.x % nch, sl = threadIdx.x / nch;
    for (int64_t e = blockIdx.x; e < nl; e += gridDim.x) {
        const int32_t vox = longv[e];
        const int32_t lo = seg[vox], hi = seg[vox + 1];
        double acc[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) acc[j] = 0.0;
        if (sl < slices)
            mean_add_range<DT, VEC, 4>(acc, feat, plist, C, tch * VEC, lo + sl, hi, slices);
#pragma unroll
        for (int j = 0; j < VEC; ++j) red[threadIdx.x][j] = acc[j];
        __syncthreads();
        if (sl == 0) {
            for (int q = 1; q < slices; ++q)
#pragma unroll
                for (int j = 0; j < VEC; ++j) acc[j] += red[q * nch + tch][j];
            mean_store<DT, VEC>(acc, (double)(hi - lo), vfeat, (int64_t)vox * C + tch * VEC);
        }
        __syncthreads();
    }
}

constexpr int kMeanRun = 32;  // points a single thread sums
constexpr int64_t kMeanInsFirst = 1 << 18;  // up to this many points the insert blocks go first

template <int DT, int VEC>
static void launch_mean(hipStream_t s, const VoxelizeWs& w, int64_t n, const void* feat, int C, void* vfeat,
                        int32_t* counts, const int32_t* coords) {
    const int nch = C / VEC;
    // with counts: per group of nch + 1 blocks, one of inserts and nch of averaging
    const int64_t nblk = counts ? blocks_for(n, 256) * (nch + 1) : blocks_for(n * nch, 256);
    const bool split = nch <= kMeanLongThreads / 2;
    k_vox_mean<DT, VEC><<<nblk, 256, 0, s>>>(w.h, n, w.seg, w.plist, feat, C, vfeat,
                                                                 split ? kMeanRun : INT32_MAX, w.longv, counts,
                                                                 w.table, coords, n <= kMeanInsFirst ? 1 : 0,
                                                                 w.nbr_upper);
    if (split) {
        const int64_t g = n < 1024 ? (n > 0 ? n : 1) : 1024;
        k_vox_mean_long<DT, VEC><<<(unsigned)g, kMeanLongThreads, 0, s>>>(w.h, n, w.seg, w.plist, feat, C, vfeat,
                                                                          w.longv);
    }
}

// counts: written from seg, with each voxel's table entry from coords, when
// given (nullptr: the caller counted N_m and built the table already)
static void launch_mean_dt(hipStream_t s, const VoxelizeWs& w, int64_t cap, const void* feat, int C, int dt,
                           void* vfeat, int32_t* counts, const int32_t* coords) {
    const bool v16 = (dt != SPV_F32) && (C % 8 == 0), v32 = (dt == SPV_F32) && (C % 4 == 0);
    if (dt == SPV_F32) {
        if (v32) launch_mean<SPV_F32, 4>(s, w, cap, feat, C, vfeat, counts, coords);
        else launch_mean<SPV_F32, 1>(s, w, cap, feat, C, vfeat, counts, coords);
    } else if (dt == SPV_BF16) {
        if (v16) launch_mean<SPV_BF16, 8>(s, w, cap, feat, C, vfeat, counts, coords);
        else launch_mean<SPV_BF16, 1>(s, w, cap, feat, C, vfeat, counts, coords);
    } else {
        if (v16) launch_mean<SPV_F16, 8>(s, w, cap, feat, C, vfeat, counts, coords);
        else launch_mean<SPV_F16, 1>(s, w, cap, feat, C, vfeat, counts, coords);
    }
}

void launch_voxelize(hipStream_t s, const VoxelizeWs& w, const float* xyz, const int32_t* batch, int64_t n,
                     float voxel_size, const void* feat, int32_t C, int dt, int32_t* coords, void* vfeat,
                     int32_t* counts, int32_t* pt2vox, int64_t* m_dev, const PackJob* jobs, int njobs) {
    VoxFirst f;
    f.h = w.h;
    f.table = w.table;
    f.zero = w.rs.zero;  // the sort's histograms and tile counters
    f.nzero = (int64_t)radix_zero_words(n);
    f.njobs = 0;
    int64_t frags = 0;
    for (int j = 0; j < njobs && f.njobs < kMaxPackJobs; ++j)
        if (jobs[j].total > 0) {
            f.job[f.njobs++] = jobs[j];
            frags += jobs[j].total;
        }
    // about one fragment per packing thread
    f.npack = frags > 0 ? (int)blocks_for(frags, kRsProducerBlock) : 0;
    if (f.npack > 256) f.npack = 256;
    // at most kRsMaxRecords quantizing blocks: every histogram block reduces all their records
    unsigned nq = blocks_for(n, kRsProducerBlock);
    if (nq > kRsMaxRecords) nq = kRsMaxRecords;
    k_vq_quantize<<<nq + (unsigned)f.npack, kRsProducerBlock, 0, s>>>(f, xyz, batch, n, voxel_size, w.rs.ka,
                                                                      w.rs.rec);
    launch_radix_sort(s, w.rs, w.h, nullptr, n, nq);
    const int64_t nt = (int64_t)radix_tiles(n);
    k_vq_segments<<<(unsigned)nt, kRsThreads, 0, s>>>(w.rs, w.h, n, nt, coords, pt2vox, w.seg, w.plist, m_dev);
    if (feat) launch_mean_dt(s, w, n, feat, C, dt, vfeat, counts, coords);
    else k_vq_counts<<<blocks_for(n, 256), 256, 0, s>>>(w.h, n, w.seg, counts, w.table, coords, w.nbr_upper);
}

void launch_voxelize_onto(hipStream_t s, const VoxelizeWs& w, const int32_t* coords, const int64_t* m_dev,
                          int64_t m_cap, const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                          const void* feat, int32_t C, int dt, void* vfeat, int32_t* counts, int32_t* pt2vox) {
    launch_clear(s, w.h, w.table, true);
    // the set's table (value = row) and its count into h->m, which the scan and the means read
    if (m_cap > 0) launch_table_build(s, w.h, w.table, coords, m_dev, m_cap, &w.h->m);
    if (m_cap > 0) k_vox_zero<<<blocks_for(m_cap, 256), 256, 0, s>>>(counts, w.fill, m_cap);
    if (n > 0)
        k_vox_locate<<<blocks_for(n, 256), 256, 0, s>>>(w.h, w.table, xyz, batch, n, voxel_size, pt2vox, counts);
    if (!feat || m_cap == 0) return;
    launch_exclusive_scan(s, counts, w.seg, &w.h->m, m_cap, w.scan_tmp);
    if (n > 0) k_vox_fill<<<blocks_for(n, 256), 256, 0, s>>>(pt2vox, n, w.seg, w.fill, w.plist);
    launch_mean_dt(s, w, m_cap, feat, C, dt, vfeat, nullptr, nullptr);
}

}  // namespace spv
