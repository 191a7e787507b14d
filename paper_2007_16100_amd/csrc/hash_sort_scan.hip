// hash_sort_scan.hip -- the GPU voxel hash table (Sec. 3.3 "Sparse Voxelization":
// O(1) insert / lookup on the voxel coordinate) and device-count prefix sums.
// (The sort that puts voxels in canonical (b, x, y, z) order is radix.hip.)
#include "spv_internal.hpp"

namespace spv {

// ---------------------------------------------------------------------------
// table clear / build / lookup
// ---------------------------------------------------------------------------
__global__ void k_clear(Header* h, Table t, int clear_header, int64_t* zero64) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        if (clear_header) {
            h->status = 0;
            h->m = 0;
            for (int i = 0; i < 4; ++i) h->aux[i] = 0;
        }
        if (zero64) *zero64 = 0;
    }
    const uint32_t nkw = t.keys ? (t.mask + 1) / 2 : 0;  // 16-byte runs of keys: 2 per bucket
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < nkw; i += gridDim.x * blockDim.x)
        *(u64x2*)(t.keys + 8 * (size_t)(i >> 1) + 2 * (i & 1)) = u64x2{kEmpty, kEmpty};
}

void launch_clear(hipStream_t s, Header* h, Table t, bool clear_header, int64_t* zero64) {
    uint32_t n = t.mask + 1;
    unsigned g = blocks_for(n, 256 * 4);
    k_clear<<<g, 256, 0, s>>>(h, t, clear_header ? 1 : 0, zero64);
}

void launch_clear_header(hipStream_t s, Header* h) { k_clear<<<1, 64, 0, s>>>(h, Table{nullptr, 0}, 1, nullptr); }

__device__ inline bool coord_ok(const int32_t* c) {
    return c[0] >= 0 && c[0] <= kBatchMax && c[1] >= kCoordMin && c[1] <= kCoordMax && c[2] >= kCoordMin &&
           c[2] <= kCoordMax && c[3] >= kCoordMin && c[3] <= kCoordMax;
}

__global__ void k_table_build(Header* h, Table t, const int32_t* coords, const int64_t* count_dev, int64_t cap,
                              int64_t* count_out, int64_t* count_out2, int32_t* nbr_upper) {
    int64_t count = count_dev ? *count_dev : cap;
    if (count > cap) count = cap;
    if (blockIdx.x == 0 && threadIdx.x == 0) {  // the count, for kernels that take it from here
        if (count_out) *count_out = count;
        if (count_out2) *count_out2 = count;
    }
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t* c = coords + 4 * i;
        if (nbr_upper) clear_nbr_upper(nbr_upper, i);
        if (!coord_ok(c)) {
            raise_flag(h, kFlagRange);
            continue;
        }
        uint32_t slot;
        int r = table_insert(t, pack_key(c[0], c[1], c[2], c[3]), &slot);
        if (r < 0) {
            raise_flag(h, kFlagTableFull);
        } else if (r == 0) {
            raise_flag(h, kFlagDuplicate);
        } else {
            *slot_val(t, slot) = (int32_t)i;
        }
    }
}

void launch_table_build(hipStream_t s, Header* h, Table t, const int32_t* coords, const int64_t* count_dev,
                        int64_t cap, int64_t* count_out, int64_t* count_out2, int32_t* nbr_upper) {
    k_table_build<<<blocks_for(cap, 256), 256, 0, s>>>(h, t, coords, count_dev, cap, count_out, count_out2,
                                                        nbr_upper);
}

__global__ void k_table_lookup(Table t, const int32_t* q, int64_t nq, int32_t* idx) {
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i >= nq) return;
    const int32_t* c = q + 4 * i;
    // coordinates outside the key range cannot be in the table
    bool ok = c[0] >= 0 && c[0] <= kBatchMax && c[1] >= -32768 && c[1] <= 32767 && c[2] >= -32768 &&
              c[2] <= 32767 && c[3] >= -32768 && c[3] <= 32767;
    idx[i] = ok ? table_find(t, pack_key(c[0], c[1], c[2], c[3])) : -1;
}

void launch_table_lookup(hipStream_t s, Table t, const int32_t* q, int64_t nq, int32_t* idx) {
    if (nq > 0) k_table_lookup<<<blocks_for(nq, 256), 256, 0, s>>>(t, q, nq, idx);
}

__device__ inline int64_t clamp_count(const int64_t* count_dev, int64_t cap) {
    int64_t c = *count_dev;
    return c < 0 ? 0 : (c > cap ? cap : c);
}

// ---------------------------------------------------------------------------
// exclusive scan with a device-side count
// ---------------------------------------------------------------------------
constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;
constexpr unsigned kScanFusedTiles = 4096;  // up to this many tiles: two kernels, no separate scan of the sums

size_t scan_tmp_entries(int64_t cap) { return (size_t)blocks_for(cap + 1, kScanTile) + 1; }

__global__ __launch_bounds__(kScanThreads) void k_scan_tiles(const int32_t* in, int32_t* out,
                                                             const int64_t* count_dev, int64_t cap, int32_t* tmp) {
    __shared__ int lds[kScanThreads / 64 + 1];
    int64_t count = count_dev ? clamp_count(count_dev, cap) : cap;
    int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int v[kScanItems];
    int s = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        int64_t i = base + j;
        v[j] = (i < count) ? in[i] : 0;
        s += v[j];
    }
    int tot;
    int run = block_exclusive_scan(s, lds, &tot);
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        int64_t i = base + j;
        if (i <= count) out[i] = run;
        run += v[j];
    }
    if (threadIdx.x == 0) tmp[blockIdx.x] = tot;
}

__global__ __launch_bounds__(1024) void k_scan_totals(int32_t* tmp, uint32_t n) {
    __shared__ int lds[17];
    uint32_t per = (n + blockDim.x - 1) / blockDim.x;
    uint32_t lo = threadIdx.x * per, hi = min(n, lo + per);
    int s = 0;
    for (uint32_t i = lo; i < hi; ++i) s += tmp[i];
    int tot;
    int run = block_exclusive_scan(s, lds, &tot);
    for (uint32_t i = lo; i < hi; ++i) {
        int v = tmp[i];
        tmp[i] = run;
        run += v;
    }
}

__global__ void k_scan_add(int32_t* out, const int64_t* count_dev, int64_t cap, const int32_t* tmp) {
    int64_t count = count_dev ? clamp_count(count_dev, cap) : cap;
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i <= count) out[i] += tmp[i / kScanTile];
}

// tile sums only (first kernel of the two-kernel scan)
__global__ __launch_bounds__(kScanThreads) void k_scan_sums(const int32_t* in, const int64_t* count_dev, int64_t cap,
                                                            int32_t* tmp) {
    __shared__ int lds[kScanThreads / 64 + 1];
    const int64_t count = count_dev ? clamp_count(count_dev, cap) : cap;
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    int s = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        const int64_t i = base + j * kScanThreads + threadIdx.x;
        s += (i < count) ? in[i] : 0;
    }
    int tot;
    block_exclusive_scan(s, lds, &tot);
    if (threadIdx.x == 0) tmp[blockIdx.x] = tot;
}

// every tile adds up the sums of the tiles before it, then scans itself
__global__ __launch_bounds__(kScanThreads) void k_scan_apply(const int32_t* in, int32_t* out, const int64_t* count_dev,
                                                             int64_t cap, const int32_t* tmp) {
    __shared__ int lds[kScanThreads / 64 + 1];
    const int64_t count = count_dev ? clamp_count(count_dev, cap) : cap;
    int pre = 0;
    for (uint32_t b = threadIdx.x; b < blockIdx.x; b += blockDim.x) pre += tmp[b];
    int prefix;
    block_exclusive_scan(pre, lds, &prefix);
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int v[kScanItems];
    int s = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        const int64_t i = base + j;
        v[j] = (i < count) ? in[i] : 0;
        s += v[j];
    }
    int tot;
    int run = block_exclusive_scan(s, lds, &tot) + prefix;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        const int64_t i = base + j;
        if (i <= count) out[i] = run;
        run += v[j];
    }
}

void launch_exclusive_scan(hipStream_t s, const int32_t* in, int32_t* out, const int64_t* count_dev, int64_t cap,
                           int32_t* tmp) {
    unsigned nb = blocks_for(cap + 1, kScanTile);
    if (nb <= kScanFusedTiles) {
        k_scan_sums<<<nb, kScanThreads, 0, s>>>(in, count_dev, cap, tmp);
        k_scan_apply<<<nb, kScanThreads, 0, s>>>(in, out, count_dev, cap, tmp);
        return;
    }
    k_scan_tiles<<<nb, kScanThreads, 0, s>>>(in, out, count_dev, cap, tmp);
    k_scan_totals<<<1, 1024, 0, s>>>(tmp, nb);
    k_scan_add<<<blocks_for(cap + 1, 256), 256, 0, s>>>(out, count_dev, cap, tmp);
}

__global__ __launch_bounds__(1024) void k_scan_small(const uint32_t* in, uint32_t* out, uint32_t n) {
    __shared__ int lds[17];
    uint32_t per = (n + blockDim.x - 1) / blockDim.x;
    uint32_t lo = threadIdx.x * per, hi = min(n, lo + per);
    int s = 0;
    for (uint32_t i = lo; i < hi; ++i) s += (int)in[i];
    int tot;
    int run = block_exclusive_scan(s, lds, &tot);
    for (uint32_t i = lo; i < hi; ++i) {
        uint32_t v = in[i];
        out[i] = (uint32_t)run;
        run += (int)v;
    }
    if (threadIdx.x == 0) out[n] = (uint32_t)tot;
}

void launch_exclusive_scan_small(hipStream_t s, const uint32_t* in, uint32_t* out, int64_t n) {
    k_scan_small<<<1, 1024, 0, s>>>(in, out, (uint32_t)n);
}

}  // namespace spv
