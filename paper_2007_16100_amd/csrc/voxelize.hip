// voxelize.hip -- sparse voxelization (Sec. 3.3, Eq. 1 and Eq. 2).
//
// 1. every point's key floor(p / v) is inserted into the open-addressing hash;
//    the thread that creates an entry appends the key to the unique-key list;
// 2. the m unique keys are radix-sorted into canonical (b, x, y, z) order and the
//    table values are set to the rank, which also writes the voxel coordinates;
// 3. every point reads its voxel index (pt2vox) at the table slot its insert
//    found, and counts N_m;
// 4. a counting sort of the points by voxel (prefix sum + fill) lets each voxel
//    gather and average its own points -- no float atomics, one write per voxel.
#include "spv_internal.hpp"

namespace spv {

void plan_voxelize_ws(Arena& a, VoxelizeWs& w, int64_t n) {
    int64_t nn = n > 0 ? n : 1;
    uint32_t S = table_capacity(nn);
    w.table.keys = a.take<uint64_t>(S);
    w.table.vals = a.take<int32_t>(S);
    w.table.mask = S - 1;
    plan_sort_ws(a, w.sort, nn);
    w.pslot = a.take<uint32_t>(nn);
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

// Eq. 1 per point, then hash insert.  Invalid points get kEmpty and a status
// flag.  Consecutive returns of a sweep often share a voxel: a lane whose key
// equals the previous lane's leaves the insert to the head of its run.  The
// block appends the keys it created to the unique-key list (one counter atomic
// per block) and records their per-field min / max for the sort.
__global__ __launch_bounds__(kAppendThreads) void k_vox_insert(Header* h, Table t, SortBufs sb, uint32_t* pslot,
                                                               const float* xyz, const int32_t* batch, int64_t n,
                                                               float v) {
    const int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    bool created = false;
    uint64_t key = kEmpty;
    int q[3] = {0, 0, 0};
    int b = 0;
    if (k < n) key = point_key(h, xyz, batch, k, v, q, b);
    // runs of equal keys inside the wave: the head inserts, the others take its
    // slot (every lane between a head and a later lane of its run has its key)
    const int lane = threadIdx.x & 63;
    const uint64_t prev_key = __shfl_up(key, 1, 64);
    const bool head = key != kEmpty && (lane == 0 || prev_key != key);
    uint32_t slot = kNoSlot;
    if (head) {
        const int r = table_insert(t, key, &slot);
        created = r > 0;
        if (r < 0) {
            raise_flag(h, kFlagTableFull);
            slot = kNoSlot;
        }
    }
    const uint64_t heads = __ballot(head) & (~0ull >> (63 - lane));  // heads at lanes <= this one
    const int src = heads ? 63 - __clzll(heads) : lane;
    const uint32_t run_slot = __shfl(slot, src, 64);
    if (k < n) pslot[k] = key == kEmpty ? kNoSlot : run_slot;
    int mn[4] = {0x7fffffff, 0x7fffffff, 0x7fffffff, 0x7fffffff};
    int mx[4] = {(int)0x80000000, (int)0x80000000, (int)0x80000000, (int)0x80000000};
    if (created) {
        const int f[4] = {b, q[0], q[1], q[2]};
#pragma unroll
        for (int d = 0; d < 4; ++d) mn[d] = mx[d] = f[d];
    }
    block_append(created, key, sb.a, &h->m);
    block_minmax_record(mn, mx, sb.part + 8 * blockIdx.x);
}

// rank -> table value, voxel coordinates, zeroed counters
__global__ void k_vox_rank(const Header* h, SortBufs sb, Table t, int32_t* coords, int32_t* counts, int32_t* fill,
                           int64_t cap, int64_t* m_dev) {
    int64_t m = h->m;
    if (m > cap) m = cap;
    int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (r == 0 && m_dev) *m_dev = m;
    if (r >= m) return;
    uint64_t key = sorted_key(sb, r);
    int64_t slot = table_slot(t, key);
    if (slot >= 0) t.vals[slot] = (int32_t)r;
    coords[4 * r + 0] = key_b(key);
    coords[4 * r + 1] = key_x(key);
    coords[4 * r + 2] = key_y(key);
    coords[4 * r + 3] = key_z(key);
    counts[r] = 0;
    fill[r] = 0;
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

__global__ void k_vox_lookup(Table t, const uint32_t* pslot, int64_t n, int32_t* pt2vox, int32_t* counts) {
    const int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int32_t v = -1;
    if (k < n) {
        const uint32_t ps = pslot[k];
        v = (ps == kNoSlot) ? -1 : t.vals[ps];
        pt2vox[k] = v;
    }
    int first, len;
    run_of(v, first, len);
    if (v >= 0 && (int)(threadIdx.x & 63) == first) atomicAdd(&counts[v], len);
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

template <int DT, int VEC>
__device__ inline void mean_store(const double (&acc)[VEC], double N, void* vfeat, int64_t orow) {
    if (N < 1.0) N = 1.0;  // a given voxel no point falls into (scatter-mean onto a set): mean 0
    if constexpr (VEC == 8) {
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            w[j] = (uint32_t)to16<DT>(f64_to_f32_odd(acc[2 * j] / N)) |
                   ((uint32_t)to16<DT>(f64_to_f32_odd(acc[2 * j + 1] / N)) << 16);
        *(uint4*)((uint16_t*)vfeat + orow) = make_uint4(w[0], w[1], w[2], w[3]);
    } else if constexpr (VEC == 4) {
        *(float4*)((float*)vfeat + orow) =
            make_float4((float)(acc[0] / N), (float)(acc[1] / N), (float)(acc[2] / N), (float)(acc[3] / N));
    } else {
        if constexpr (DT == SPV_F32) st_feat<DT>(vfeat, orow, (float)(acc[0] / N));
        else st_feat<DT>(vfeat, orow, f64_to_f32_odd(acc[0] / N));
    }
}

template <int DT, int VEC>
__global__ void k_vox_mean(Header* h, int64_t cap, const int32_t* seg, const int32_t* plist, const void* feat,
                           int C, void* vfeat, int run, int32_t* longv) {
    int64_t m = h->m;
    if (m > cap) m = cap;
    const int nch = C / VEC;
    int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t vox = t / nch;
    int ch = (int)(t - vox * nch) * VEC;
    if (vox >= m) return;
    int32_t lo = seg[vox], hi = seg[vox + 1];
    if (hi - lo > run) {
        if (ch == 0) longv[atomicAdd((unsigned long long*)&h->aux[0], 1ull)] = (int32_t)vox;
        return;
    }
    double acc[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] = 0.0;
    for (int32_t p = lo; p < hi; ++p) mean_add<DT, VEC>(acc, feat, (int64_t)plist[p] * C + ch);
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
            for (int32_t p = lo + sl; p < hi; p += slices) mean_add<DT, VEC>(acc, feat, (int64_t)plist[p] * C + tch * VEC);
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

template <int DT, int VEC>
static void launch_mean(hipStream_t s, const VoxelizeWs& w, int64_t n, const void* feat, int C, void* vfeat) {
    const int64_t threads = n * (C / VEC);
    const bool split = C / VEC <= kMeanLongThreads / 2;
    k_vox_mean<DT, VEC><<<blocks_for(threads, 256), 256, 0, s>>>(w.h, n, w.seg, w.plist, feat, C, vfeat,
                                                                 split ? kMeanRun : INT32_MAX, w.longv);
    if (split) {
        const int64_t g = n < 1024 ? (n > 0 ? n : 1) : 1024;
        k_vox_mean_long<DT, VEC><<<(unsigned)g, kMeanLongThreads, 0, s>>>(w.h, n, w.seg, w.plist, feat, C, vfeat,
                                                                          w.longv);
    }
}

static void launch_mean_dt(hipStream_t s, const VoxelizeWs& w, int64_t cap, const void* feat, int C, int dt,
                           void* vfeat) {
    const bool v16 = (dt != SPV_F32) && (C % 8 == 0), v32 = (dt == SPV_F32) && (C % 4 == 0);
    if (dt == SPV_F32) {
        if (v32) launch_mean<SPV_F32, 4>(s, w, cap, feat, C, vfeat);
        else launch_mean<SPV_F32, 1>(s, w, cap, feat, C, vfeat);
    } else if (dt == SPV_BF16) {
        if (v16) launch_mean<SPV_BF16, 8>(s, w, cap, feat, C, vfeat);
        else launch_mean<SPV_BF16, 1>(s, w, cap, feat, C, vfeat);
    } else {
        if (v16) launch_mean<SPV_F16, 8>(s, w, cap, feat, C, vfeat);
        else launch_mean<SPV_F16, 1>(s, w, cap, feat, C, vfeat);
    }
}

void launch_voxelize(hipStream_t s, const VoxelizeWs& w, const float* xyz, const int32_t* batch, int64_t n,
                     float voxel_size, const void* feat, int32_t C, int dt, int32_t* coords, void* vfeat,
                     int32_t* counts, int32_t* pt2vox, int64_t* m_dev, bool table_cleared) {
    if (!table_cleared) launch_clear(s, w.h, w.table, true);
    const unsigned nins = n > 0 ? blocks_for(n, kAppendThreads) : 0u;
    if (n > 0) k_vox_insert<<<nins, kAppendThreads, 0, s>>>(w.h, w.table, w.sort, w.pslot, xyz, batch, n, voxel_size);
    launch_sort_keys(s, w.sort, &w.h->m, n, nins);
    k_vox_rank<<<blocks_for(n, 256), 256, 0, s>>>(w.h, w.sort, w.table, coords, counts, w.fill, n, m_dev);
    if (n == 0) return;
    k_vox_lookup<<<blocks_for(n, 256), 256, 0, s>>>(w.table, w.pslot, n, pt2vox, counts);
    if (!feat) return;
    launch_exclusive_scan(s, counts, w.seg, &w.h->m, n, w.scan_tmp);
    k_vox_fill<<<blocks_for(n, 256), 256, 0, s>>>(pt2vox, n, w.seg, w.fill, w.plist);
    launch_mean_dt(s, w, n, feat, C, dt, vfeat);
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
    launch_mean_dt(s, w, m_cap, feat, C, dt, vfeat);
}

}  // namespace spv
