// hash_sort_scan.hip -- the GPU voxel hash table (Sec. 3.3 "Sparse Voxelization":
// O(1) insert / lookup on the voxel coordinate), an LSD radix sort that puts the
// non-empty voxels in canonical (b, x, y, z) order, and device-count prefix sums.
#include "spv_internal.hpp"

namespace spv {

// ---------------------------------------------------------------------------
// table clear / build / lookup
// ---------------------------------------------------------------------------
__global__ void k_clear(Header* h, uint64_t* keys, uint32_t nslots, int clear_header) {
    if (clear_header && blockIdx.x == 0 && threadIdx.x == 0) {
        h->status = 0;
        h->m = 0;
        for (int i = 0; i < 4; ++i) h->aux[i] = 0;
    }
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < nslots; i += gridDim.x * blockDim.x) keys[i] = kEmpty;
}

void launch_clear(hipStream_t s, Header* h, Table t, bool clear_header) {
    uint32_t n = t.mask + 1;
    unsigned g = blocks_for(n, 256 * 4);
    k_clear<<<g, 256, 0, s>>>(h, t.keys, n, clear_header ? 1 : 0);
}

void launch_clear_header(hipStream_t s, Header* h) { k_clear<<<1, 64, 0, s>>>(h, nullptr, 0, 1); }

__device__ inline bool coord_ok(const int32_t* c) {
    return c[0] >= 0 && c[0] <= kBatchMax && c[1] >= kCoordMin && c[1] <= kCoordMax && c[2] >= kCoordMin &&
           c[2] <= kCoordMax && c[3] >= kCoordMin && c[3] <= kCoordMax;
}

__global__ void k_table_build(Header* h, Table t, const int32_t* coords, const int64_t* count_dev, int64_t cap) {
    int64_t count = count_dev ? *count_dev : cap;
    if (count > cap) count = cap;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t* c = coords + 4 * i;
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
            t.vals[slot] = (int32_t)i;
        }
    }
}

void launch_table_build(hipStream_t s, Header* h, Table t, const int32_t* coords, const int64_t* count_dev,
                        int64_t cap) {
    k_table_build<<<blocks_for(cap, 256), 256, 0, s>>>(h, t, coords, count_dev, cap);
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

// ---------------------------------------------------------------------------
// radix sort of packed voxel keys with a device-side count
// ---------------------------------------------------------------------------
constexpr int kSortThreads = 256;
constexpr int kSortItems = 8;
constexpr int kSortTile = kSortThreads * kSortItems;

size_t sort_hist_entries(int64_t cap) { return (size_t)256 * blocks_for(cap, kSortTile); }

void plan_sort_ws(Arena& a, SortBufs& sb, int64_t cap) {
    int64_t c = cap > 0 ? cap : 1;
    sb.a = a.take<uint64_t>(c);
    sb.b = a.take<uint64_t>(c);
    sb.hist = a.take<uint32_t>(sort_hist_entries(c));
    sb.st = a.take<SortStats>(1);
}

__global__ void k_sort_reset(SortStats* st) {
    if (threadIdx.x < 4) {
        st->fmin[threadIdx.x] = 0x7fffffff;
        st->fmax[threadIdx.x] = (int32_t)0x80000000;
        st->fbits[threadIdx.x] = 0;
    }
    if (threadIdx.x == 0) st->sort_bits = 0;
}

__device__ inline int64_t clamp_count(const int64_t* count_dev, int64_t cap) {
    int64_t c = *count_dev;
    return c < 0 ? 0 : (c > cap ? cap : c);
}

__global__ void k_sort_minmax(SortStats* h, const uint64_t* keys, const int64_t* count_dev, int64_t cap) {
    int64_t count = clamp_count(count_dev, cap);
    int mn[4] = {0x7fffffff, 0x7fffffff, 0x7fffffff, 0x7fffffff};
    int mx[4] = {(int)0x80000000, (int)0x80000000, (int)0x80000000, (int)0x80000000};
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x) {
        uint64_t k = keys[i];
        int f[4] = {key_b(k), key_x(k), key_y(k), key_z(k)};
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            mn[d] = min(mn[d], f[d]);
            mx[d] = max(mx[d], f[d]);
        }
    }
#pragma unroll
    for (int d = 0; d < 4; ++d) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            mn[d] = min(mn[d], __shfl_xor(mn[d], o, 64));
            mx[d] = max(mx[d], __shfl_xor(mx[d], o, 64));
        }
    }
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            atomicMin(&h->fmin[d], mn[d]);
            atomicMax(&h->fmax[d], mx[d]);
        }
    }
}

__device__ inline uint32_t bitwidth(uint32_t range) { return range ? 32u - __clz(range) : 0u; }

__global__ void k_sort_compact(SortStats* h, uint64_t* keys, const int64_t* count_dev, int64_t cap) {
    int64_t count = clamp_count(count_dev, cap);
    int32_t mn[4];
    uint32_t w[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        mn[d] = h->fmin[d];
        w[d] = (count > 0) ? bitwidth((uint32_t)(h->fmax[d] - h->fmin[d])) : 0u;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        for (int d = 0; d < 4; ++d) h->fbits[d] = w[d];
        h->sort_bits = w[0] + w[1] + w[2] + w[3];
    }
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x) {
        uint64_t k = keys[i];
        uint64_t ck = (uint64_t)(uint32_t)(key_b(k) - mn[0]);
        ck = (ck << w[1]) | (uint64_t)(uint32_t)(key_x(k) - mn[1]);
        ck = (ck << w[2]) | (uint64_t)(uint32_t)(key_y(k) - mn[2]);
        ck = (ck << w[3]) | (uint64_t)(uint32_t)(key_z(k) - mn[3]);
        keys[i] = ck;
    }
}

__global__ __launch_bounds__(kSortThreads) void k_radix_hist(const SortStats* h, SortBufs sb, const int64_t* count_dev,
                                                             int64_t cap, int pass) {
    const uint32_t nblk = gridDim.x;
    if ((uint32_t)(8 * pass) >= h->sort_bits) return;
    const uint64_t* src = (pass & 1) ? sb.b : sb.a;
    __shared__ uint32_t hist[256];
    hist[threadIdx.x] = 0;
    __syncthreads();
    int64_t count = clamp_count(count_dev, cap);
    int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int r = 0; r < kSortItems; ++r) {
        int64_t i = base + r * kSortThreads + threadIdx.x;
        if (i < count) atomicAdd(&hist[(src[i] >> (8 * pass)) & 0xFF], 1u);
    }
    __syncthreads();
    sb.hist[threadIdx.x * nblk + blockIdx.x] = hist[threadIdx.x];
}

// exclusive scan of the digit-major histogram by one block
__global__ __launch_bounds__(1024) void k_radix_scan(const SortStats* h, uint32_t* hist, uint32_t n, int pass) {
    if ((uint32_t)(8 * pass) >= h->sort_bits) return;
    __shared__ int lds[17];
    uint32_t per = (n + blockDim.x - 1) / blockDim.x;
    uint32_t lo = threadIdx.x * per, hi = min(n, lo + per);
    int s = 0;
    for (uint32_t i = lo; i < hi; ++i) s += (int)hist[i];
    int tot;
    int run = block_exclusive_scan(s, lds, &tot);
    for (uint32_t i = lo; i < hi; ++i) {
        uint32_t v = hist[i];
        hist[i] = (uint32_t)run;
        run += (int)v;
    }
}

__global__ __launch_bounds__(kSortThreads) void k_radix_scatter(const SortStats* h, SortBufs sb,
                                                                const int64_t* count_dev, int64_t cap, int pass) {
    const uint32_t nblk = gridDim.x;
    if ((uint32_t)(8 * pass) >= h->sort_bits) return;
    const uint64_t* src = (pass & 1) ? sb.b : sb.a;
    uint64_t* dst = (pass & 1) ? sb.a : sb.b;
    __shared__ uint32_t run[256];
    __shared__ uint32_t wcnt[kSortThreads / 64][256];
    __shared__ uint32_t woff[kSortThreads / 64][256];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    run[t] = sb.hist[t * nblk + blockIdx.x];
    for (int w = 0; w < kSortThreads / 64; ++w) wcnt[w][t] = 0;
    __syncthreads();
    int64_t count = clamp_count(count_dev, cap);
    int64_t base = (int64_t)blockIdx.x * kSortTile;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int r = 0; r < kSortItems; ++r) {
        int64_t i = base + r * kSortThreads + t;
        bool valid = i < count;
        uint64_t key = valid ? src[i] : 0;
        uint32_t d = (uint32_t)(key >> (8 * pass)) & 0xFF;
        // lanes of this wave holding the same digit
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            uint64_t bal = __ballot((d >> b) & 1);
            peers &= ((d >> b) & 1) ? bal : ~bal;
        }
        uint32_t rank = (uint32_t)__popcll(peers & lt);
        if (valid && rank == 0) wcnt[wave][d] = (uint32_t)__popcll(peers);
        __syncthreads();
        {
            uint32_t b0 = run[t];
            for (int w = 0; w < kSortThreads / 64; ++w) {
                uint32_t c = wcnt[w][t];
                woff[w][t] = b0;
                b0 += c;
                wcnt[w][t] = 0;
            }
            run[t] = b0;
        }
        __syncthreads();
        if (valid) dst[woff[wave][d] + rank] = key;
    }
}

void launch_sort_keys(hipStream_t s, SortBufs sb, const int64_t* count_dev, int64_t cap) {
    if (cap <= 0) cap = 1;
    SortStats* h = sb.st;
    k_sort_reset<<<1, 64, 0, s>>>(h);
    unsigned g = blocks_for(cap, 256 * 4);
    k_sort_minmax<<<g, 256, 0, s>>>(h, sb.a, count_dev, cap);
    k_sort_compact<<<g, 256, 0, s>>>(h, sb.a, count_dev, cap);
    unsigned nblk = blocks_for(cap, kSortTile);
    for (int pass = 0; pass < 8; ++pass) {
        k_radix_hist<<<nblk, kSortThreads, 0, s>>>(h, sb, count_dev, cap, pass);
        k_radix_scan<<<1, 1024, 0, s>>>(h, sb.hist, 256 * nblk, pass);
        k_radix_scatter<<<nblk, kSortThreads, 0, s>>>(h, sb, count_dev, cap, pass);
    }
}

// ---------------------------------------------------------------------------
// exclusive scan with a device-side count
// ---------------------------------------------------------------------------
constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

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

void launch_exclusive_scan(hipStream_t s, const int32_t* in, int32_t* out, const int64_t* count_dev, int64_t cap,
                           int32_t* tmp) {
    unsigned nb = blocks_for(cap + 1, kScanTile);
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
