// hash_sort_scan.hip -- the GPU voxel hash table (Sec. 3.3 "Sparse Voxelization":
// O(1) insert / lookup on the voxel coordinate), an LSD radix sort that puts the
// non-empty voxels in canonical (b, x, y, z) order, and device-count prefix sums.
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

// ---------------------------------------------------------------------------
// radix sort of packed voxel keys with a device-side count
// ---------------------------------------------------------------------------
constexpr int kSortThreads = 256;
constexpr int kSortItems = 4;
constexpr int kSortTile = kSortThreads * kSortItems;
constexpr int kSortParts = 256;            // partial records of the stand-alone min / max kernel
constexpr uint32_t kFusedSortBlocks = 256;  // up to this many tiles a scatter block scans the histograms itself
constexpr uint32_t kFusedStatsParts = 1024;  // up to this many min / max records the pass-0 blocks reduce them
constexpr uint64_t kFusedStatsReads = 1u << 20;  // ... if all blocks together read at most this many records

size_t sort_hist_entries(int64_t cap) { return (size_t)256 * blocks_for(cap, kSortTile) + 1; }
size_t sort_part_records(int64_t cap) {
    const size_t b = blocks_for(cap, kAppendThreads);
    return b > (size_t)kSortParts ? b : (size_t)kSortParts;
}

void plan_sort_ws(Arena& a, SortBufs& sb, int64_t cap) {
    int64_t c = cap > 0 ? cap : 1;
    sb.a = a.take<uint64_t>(c);
    sb.b = a.take<uint64_t>(c);
    sb.hist = a.take<uint32_t>(sort_hist_entries(c));
    sb.part = a.take<int32_t>(8 * sort_part_records(c));
    sb.st = a.take<SortStats>(1);
    sb.scan_tmp = a.take<int32_t>(scan_tmp_entries((int64_t)sort_hist_entries(c)));
}

__device__ inline int64_t clamp_count(const int64_t* count_dev, int64_t cap) {
    int64_t c = *count_dev;
    return c < 0 ? 0 : (c > cap ? cap : c);
}

__global__ __launch_bounds__(256) void k_sort_minmax(int32_t* part, const uint64_t* keys, const int64_t* count_dev,
                                                     int64_t cap) {
    const int64_t count = clamp_count(count_dev, cap);
    int mn[4] = {0x7fffffff, 0x7fffffff, 0x7fffffff, 0x7fffffff};
    int mx[4] = {(int)0x80000000, (int)0x80000000, (int)0x80000000, (int)0x80000000};
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t k = keys[i];
        const int f[4] = {key_b(k), key_x(k), key_y(k), key_z(k)};
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            mn[d] = min(mn[d], f[d]);
            mx[d] = max(mx[d], f[d]);
        }
    }
    block_minmax_record(mn, mx, part + 8 * blockIdx.x);
}

// reduce the partial records into the per-field minimum and bit widths
// The sort's statistics from the producers' min / max records, by one block
// (any size, a multiple of 64 threads): every thread gets them in *out.
__device__ inline void reduce_sort_stats(const int32_t* part, uint32_t nparts, const int64_t* count_dev, int64_t cap,
                                         SortStats* out) {
    int mn[4] = {0x7fffffff, 0x7fffffff, 0x7fffffff, 0x7fffffff};
    int mx[4] = {(int)0x80000000, (int)0x80000000, (int)0x80000000, (int)0x80000000};
    for (uint32_t r = threadIdx.x; r < nparts; r += blockDim.x) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            mn[d] = min(mn[d], part[8 * r + d]);
            mx[d] = max(mx[d], part[8 * r + 4 + d]);
        }
    }
    __shared__ int32_t red[8];
    __shared__ SortStats res;
    if (threadIdx.x < 8) red[threadIdx.x] = threadIdx.x < 4 ? 0x7fffffff : (int)0x80000000;
    __syncthreads();
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
            atomicMin(&red[d], mn[d]);  // LDS atomics: a few per block
            atomicMax(&red[4 + d], mx[d]);
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const bool nonempty = clamp_count(count_dev, cap) > 0;
        uint32_t bits = 0;
        for (int d = 0; d < 4; ++d) {
            const uint32_t range = nonempty ? (uint32_t)(red[4 + d] - red[d]) : 0u;
            const uint32_t w = range ? 32u - __clz(range) : 0u;
            res.fmin[d] = nonempty ? red[d] : 0;
            res.fmax[d] = nonempty ? red[4 + d] : 0;
            res.fbits[d] = w;
            bits += w;
        }
        res.sort_bits = bits;
    }
    __syncthreads();
    *out = res;
}

__global__ __launch_bounds__(256) void k_sort_stats(SortStats* st, const int32_t* part, uint32_t nparts,
                                                    const int64_t* count_dev, int64_t cap) {
    SortStats r;
    reduce_sort_stats(part, nparts, count_dev, cap, &r);
    if (threadIdx.x == 0) *st = r;
}

// lanes of this wave whose `valid` digit d equals this lane's (8 ballots)
__device__ inline uint64_t digit_peers(uint32_t d, bool valid) {
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        const uint64_t bal = __ballot((d >> b) & 1);
        peers &= ((d >> b) & 1) ? bal : ~bal;
    }
    return peers;
}

// Histogram of one 8-bit digit per tile.  Pass 0 first replaces every key by
// its compacted form (per-field minimum subtracted, fields packed into their
// bit widths) in place; it runs even when there is nothing to sort so that the
// buffer read back always holds compacted keys.  Lanes of a wave holding the
// same digit are counted by one LDS add of their leader.
// With fused_parts > 0 (pass 0 only) the block first reduces the producers'
// fused_parts min / max records itself (block 0 also stores the result for the
// later kernels), in place of a separate statistics launch.
__global__ __launch_bounds__(kSortThreads) void k_radix_hist(SortStats* st, SortBufs sb, const int64_t* count_dev,
                                                             int64_t cap, int pass, int digit_major,
                                                             uint32_t fused_parts) {
    const uint32_t nblk = gridDim.x;
    if (pass > 0 && (uint32_t)(8 * pass) >= st->sort_bits) return;
    SortStats lst;
    if (fused_parts) {
        reduce_sort_stats(sb.part, fused_parts, count_dev, cap, &lst);
        if (blockIdx.x == 0 && threadIdx.x == 0) *st = lst;
    }
    uint64_t* src = (pass & 1) ? sb.b : sb.a;
    __shared__ uint32_t hist[256];
    hist[threadIdx.x] = 0;
    const int lane = threadIdx.x & 63;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t count = clamp_count(count_dev, cap);
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    uint64_t key[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t i = base + r * kSortThreads + threadIdx.x;
        key[r] = i < count ? src[i] : 0ull;
    }
    if (pass == 0) {
        int32_t mn[4];
        uint32_t w[4];
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            mn[d] = fused_parts ? lst.fmin[d] : st->fmin[d];
            w[d] = fused_parts ? lst.fbits[d] : st->fbits[d];
        }
#pragma unroll
        for (int r = 0; r < kSortItems; ++r) {
            const int64_t i = base + r * kSortThreads + threadIdx.x;
            const uint64_t k = key[r];
            uint64_t ck = (uint64_t)(uint32_t)(key_b(k) - mn[0]);
            ck = (ck << w[1]) | (uint64_t)(uint32_t)(key_x(k) - mn[1]);
            ck = (ck << w[2]) | (uint64_t)(uint32_t)(key_y(k) - mn[2]);
            ck = (ck << w[3]) | (uint64_t)(uint32_t)(key_z(k) - mn[3]);
            key[r] = ck;
            if (i < count) src[i] = ck;
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t i = base + r * kSortThreads + threadIdx.x;
        const bool valid = i < count;
        const uint32_t d = (uint32_t)(key[r] >> (8 * pass)) & 0xFF;
        const uint64_t peers = digit_peers(d, valid);
        if (valid && (peers & lt) == 0) atomicAdd(&hist[d], (uint32_t)__popcll(peers));
    }
    __syncthreads();
    if (digit_major) sb.hist[(size_t)threadIdx.x * nblk + blockIdx.x] = hist[threadIdx.x];
    else sb.hist[(size_t)blockIdx.x * 256 + threadIdx.x] = hist[threadIdx.x];  // tile-major (coalesced)
}

// Stable scatter of one tile by one digit.  With `fused`, the block derives its
// digit offsets from the raw tile-major histograms (thread d: all tiles' counts
// of digit d, those of earlier tiles, then a scan over the digits); otherwise
// the histograms are digit-major and an exclusive scan over all of them has
// already turned them into write offsets.  Inside the tile, items are
// ranked in (round, wave, lane) order -- the index order -- from per-wave digit
// groups: counts of every (round, wave, digit) first, then one running sum per
// digit over them, then every item is written.
__global__ __launch_bounds__(kSortThreads) void k_radix_scatter(const SortStats* st, SortBufs sb,
                                                                const int64_t* count_dev, int64_t cap, int pass,
                                                                int fused) {
    constexpr int NWV = kSortThreads / 64;
    const uint32_t nblk = gridDim.x;
    if ((uint32_t)(8 * pass) >= st->sort_bits) return;
    const uint64_t* src = (pass & 1) ? sb.b : sb.a;
    uint64_t* dst = (pass & 1) ? sb.a : sb.b;
    __shared__ uint32_t cnt[kSortItems][NWV][256];  // counts, then write offsets
    __shared__ int lds[NWV + 1];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t count = clamp_count(count_dev, cap);
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    uint64_t keys[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t i = base + r * kSortThreads + t;
        keys[r] = i < count ? src[i] : 0ull;
    }
#pragma unroll
    for (int r = 0; r < kSortItems; ++r)
#pragma unroll
        for (int w = 0; w < NWV; ++w) cnt[r][w][t] = 0;
    uint32_t run;
    if (fused) {
        uint32_t tot = 0, pre = 0;
#pragma unroll 8
        for (uint32_t b = 0; b < nblk; ++b) {
            const uint32_t v = sb.hist[(size_t)b * 256 + t];  // coalesced over the digits
            tot += v;
            pre += (b < blockIdx.x) ? v : 0u;
        }
        int all;
        run = (uint32_t)block_exclusive_scan((int)tot, lds, &all) + pre;
    } else {
        run = sb.hist[(size_t)t * nblk + blockIdx.x];
        __syncthreads();
    }
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint32_t rank[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t i = base + r * kSortThreads + t;
        const bool valid = i < count;
        const uint32_t d = (uint32_t)(keys[r] >> (8 * pass)) & 0xFF;
        const uint64_t peers = digit_peers(d, valid);
        rank[r] = (uint32_t)__popcll(peers & lt);
        if (valid && rank[r] == 0) cnt[r][wave][d] = (uint32_t)__popcll(peers);
    }
    __syncthreads();
    // thread t owns digit t: running offsets over (round, wave) in index order
#pragma unroll
    for (int r = 0; r < kSortItems; ++r)
#pragma unroll
        for (int w = 0; w < NWV; ++w) {
            const uint32_t c = cnt[r][w][t];
            cnt[r][w][t] = run;
            run += c;
        }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t i = base + r * kSortThreads + t;
        if (i < count) {
            const uint32_t d = (uint32_t)(keys[r] >> (8 * pass)) & 0xFF;
            dst[cnt[r][wave][d] + rank[r]] = keys[r];
        }
    }
}

void launch_sort_keys(hipStream_t s, SortBufs sb, const int64_t* count_dev, int64_t cap, uint32_t nparts) {
    if (cap <= 0) cap = 1;
    if (nparts == 0) {
        unsigned g = blocks_for(cap, 256 * 4);
        if (g > (unsigned)kSortParts) g = kSortParts;
        k_sort_minmax<<<g, 256, 0, s>>>(sb.part, sb.a, count_dev, cap);
        nparts = g;
    }
    const unsigned nblk = blocks_for(cap, kSortTile);
    // few records: every pass-0 histogram block reduces them itself
    const uint32_t fused_parts = (nparts <= kFusedStatsParts && (uint64_t)nblk * nparts <= kFusedStatsReads) ? nparts : 0u;
    if (!fused_parts) k_sort_stats<<<1, 256, 0, s>>>(sb.st, sb.part, nparts, count_dev, cap);
    const int fused = nblk <= kFusedSortBlocks ? 1 : 0;
    // the significant bits are known on the device only: every pass a 64-bit key
    // may need is launched, and passes beyond them exit at once
    for (int pass = 0; pass < 8; ++pass) {
        k_radix_hist<<<nblk, kSortThreads, 0, s>>>(sb.st, sb, count_dev, cap, pass, !fused, pass == 0 ? fused_parts : 0u);
        if (!fused) {
            // digit-major histograms -> write offsets (a pass past the significant
            // bits scans stale counts that its scatter then ignores)
            int32_t* h = (int32_t*)sb.hist;
            launch_exclusive_scan(s, h, h, nullptr, (int64_t)256 * nblk, sb.scan_tmp);
        }
        k_radix_scatter<<<nblk, kSortThreads, 0, s>>>(sb.st, sb, count_dev, cap, pass, fused);
    }
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
