// radix.hip -- stable LSD radix sort of (64-bit key, 32-bit payload) pairs with
// one kernel per 8-bit digit: the canonical (b, x, y, z) order of the voxels of
// Sec. 3.3 (the paper leaves the order of the m voxels open; this build makes it
// ascending key order).
//
// The producer of the keys (the voxelization's quantize kernel, for instance)
// writes raw packed keys -- kEmpty for an invalid item -- and one record per
// block of per-field minima / maxima and invalid counts.  Then:
//   k_rs_hist   reduces the records into the compaction (per-field minimum
//               subtracted, fields packed into their bit widths) and counts the
//               digits of every pass over all keys at once (global histograms);
//   k_rs_pass   one launch per digit: a tile of keys ranks its items by digit
//               in index order (stable), publishes its digit counts, reads the
//               counts of the tiles before it (decoupled look-back: a tile that
//               has finished publishes its inclusive prefix, so a reader stops
//               there) and scatters its items to bucket base + prefix + rank.
// Tiles take their place in the order they start (a counter), so every tile a
// reader waits for is already running: the look-back always ends.  Passes past
// the significant bits of the compacted key exit at once.  Invalid items get
// the all-ones key, which no valid compacted key reaches; their presence makes
// the sort cover all 64 bits so that they end up last.
//
// Up to kMsMaxBlocks histogram blocks of keys, a bucket sort takes the place of
// the passes when it can (every item valid, at most 32 significant bits, and no
// bucket over kMsCap items):
//   k_rs_hist    also counts the keys of each fine bin (their top 12
//                significant bits) over all keys;
//   k_ms_scatter groups consecutive fine bins into buckets of about equal
//                item counts (order-preserving: a bucket is a range of fine
//                bins) and moves every item into its fine bin: the bin's
//                base, plus the block's share of the bin claimed with one
//                atomic per bin and block, plus its rank among the block's
//                items of that bin (index order);
//   k_ms_bucket  one workgroup per bucket sorts it in LDS by the key bits
//                below the bucket's first bin and then by the item's block
//                (an LSD sort of 8-bit digits whose passes never leave the
//                workgroup), which restores index order between blocks, and
//                writes the result in place of the keys.
// Otherwise the scatter does nothing and the bucket kernel's first workgroups
// run every pass instead (one per tile, grid barriers between the passes).
// Either way the order is the same stable ascending order.
#include "spv_internal.hpp"

namespace spv {

constexpr uint64_t kRsFlagAgg = 1ull << 62;  // status word: the tile's own count
constexpr uint64_t kRsFlagInc = 2ull << 62;  // ... the inclusive prefix (counts of this tile and all before)
constexpr uint32_t kRsSpinLimit = 1u << 22;  // polls of one status word before the sort gives up (flags an error)
constexpr int kRsHeadPasses = 4;    // passes launched one by one (enough for 32 significant bits)
constexpr unsigned kRsTailTiles = 256;  // most tiles for which those passes share one launch
constexpr int kRsBarrierCtr = 16;   // ctr[16 + pass]: arrivals at the grid barrier before pass

size_t radix_tiles(int64_t cap) { return blocks_for(cap > 0 ? cap : 1, kRsTile); }

// histogram blocks: kRhThreads threads over kRhTile keys
constexpr int kRhThreads = 256;
constexpr int kRhTile = kRhThreads * kRsItems;
constexpr unsigned kRhMaxBlocks = 1024;
// the bucket sort: at most kMsMaxBlocks histogram blocks (one tile of kRhTile
// keys each, so an item's block fits 8 bits), kMsFine fine bins, at most
// kMsMaxBuckets buckets of at most kMsCap items, each sorted by kMsThreads
// threads (two workgroups fit a CU)
constexpr unsigned kMsMaxBlocks = 256;
constexpr int kMsFineBits = 12;
constexpr int kMsFine = 1 << kMsFineBits;
constexpr int kMsMaxBuckets = 512;
constexpr int kMsThreads = 512;
constexpr int kMsRounds = 16;
constexpr int kMsCap = kMsThreads * kMsRounds;

void plan_radix_ws(Arena& a, RadixWs& w, int64_t cap) {
    const int64_t c = cap > 0 ? cap : 1;
    w.ka = a.take<uint64_t>(c);
    w.kb = a.take<uint64_t>(c);
    w.va = a.take<uint32_t>(c);
    w.vb = a.take<uint32_t>(c);
    w.rec = a.take<int32_t>((size_t)kRsRecWords * blocks_for(c, kRsProducerBlock));
    w.st = a.take<SortStats>(1);
    w.ntiles = (int64_t)radix_tiles(c);
    // zeroed by the producer: digit histograms and tile counters
    w.zero = a.take<uint32_t>(radix_zero_words(c));
    w.ghist = w.zero;
    w.ctr = w.zero + kRsPasses * kRsBins;
    w.fhist = w.ctr + 64;
    w.fcur = w.fhist + kMsFine;
    w.sb = a.take<uint32_t>(2 * (kMsMaxBuckets + 1) + 1);
    // look-back words, cleared by the sort's own kernels before each use
    w.status = a.take<uint64_t>((size_t)kRsPasses * kRsBins * w.ntiles + w.ntiles);
}

size_t radix_zero_words(int64_t) { return (size_t)kRsPasses * kRsBins + 64 + 2 * kMsFine; }

// the compacted form of a raw key (all ones for an invalid item)
__device__ inline uint64_t rs_compact(uint64_t k, const SortStats& st) {
    if (k == kEmpty) return kEmpty;
    uint64_t ck = (uint64_t)(uint32_t)(key_b(k) - st.fmin[0]);
    ck = (ck << st.fbits[1]) | (uint64_t)(uint32_t)(key_x(k) - st.fmin[1]);
    ck = (ck << st.fbits[2]) | (uint64_t)(uint32_t)(key_y(k) - st.fmin[2]);
    ck = (ck << st.fbits[3]) | (uint64_t)(uint32_t)(key_z(k) - st.fmin[3]);
    return ck;
}

// The sort's statistics from the producer's records, by one block (every
// thread receives them).  sort_bits covers all 64 bits when any item is
// invalid, so that the all-ones keys sort last.
__device__ inline void rs_reduce_stats(const int32_t* rec, uint32_t nrec, int64_t count, SortStats* out) {
    int mn[4] = {0x7fffffff, 0x7fffffff, 0x7fffffff, 0x7fffffff};
    int mx[4] = {(int)0x80000000, (int)0x80000000, (int)0x80000000, (int)0x80000000};
    uint32_t inv = 0, iflags = 0;
    for (uint32_t r = threadIdx.x; r < nrec; r += blockDim.x) {
        const int32_t* q = rec + (size_t)kRsRecWords * r;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            mn[d] = min(mn[d], q[d]);
            mx[d] = max(mx[d], q[4 + d]);
        }
        inv += (uint32_t)q[8] + (uint32_t)q[9];
        iflags |= (q[8] ? 1u : 0u) | (q[9] ? 2u : 0u);
    }
#pragma unroll
    for (int d = 0; d < 4; ++d) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            mn[d] = min(mn[d], __shfl_xor(mn[d], o, 64));
            mx[d] = max(mx[d], __shfl_xor(mx[d], o, 64));
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        inv += __shfl_xor(inv, o, 64);
        iflags |= __shfl_xor(iflags, o, 64);
    }
    __shared__ int32_t red[8];
    __shared__ uint32_t sinv, sflags;
    __shared__ SortStats res;
    if (threadIdx.x < 8) red[threadIdx.x] = threadIdx.x < 4 ? 0x7fffffff : (int)0x80000000;
    if (threadIdx.x == 0) sinv = sflags = 0;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            atomicMin(&red[d], mn[d]);  // LDS
            atomicMax(&red[4 + d], mx[d]);
        }
        atomicAdd(&sinv, inv);
        atomicOr(&sflags, iflags);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const bool any = (int64_t)sinv < count;  // at least one valid key
        uint32_t bits = 0;
        for (int d = 0; d < 4; ++d) {
            const uint32_t range = any ? (uint32_t)(red[4 + d] - red[d]) : 0u;
            const uint32_t w = range ? 32u - __clz(range) : 0u;
            res.fmin[d] = any ? red[d] : 0;
            res.fmax[d] = any ? red[4 + d] : 0;
            res.fbits[d] = w;
            bits += w;
        }
        res.n_invalid = sinv;
        res.invalid_kinds = sflags;
        res.sort_bits = sinv ? 64u : bits;
        res.msd = 0;
    }
    __syncthreads();
    *out = res;
}

__device__ inline int64_t rs_count(const int64_t* count_dev, int64_t cap) {
    if (!count_dev) return cap;
    const int64_t c = *count_dev;
    return c < 0 ? 0 : (c > cap ? cap : c);
}

// lanes of this wave whose valid digit d equals this lane's, on the digit's
// low nbits bits: one ballot per bit, and per bit the ballot or its complement
// (XNOR with the lane's bit, sign-extended) on both halves of the mask.
template <int BITS = kRsBits>
__device__ inline uint64_t rs_peers(uint32_t d, bool valid, int nbits = BITS) {
    if (nbits < BITS) d &= (1u << nbits) - 1u;  // bits above are equal in every lane
    const uint64_t v = __ballot(valid);
    int32_t m[BITS];
    uint64_t bal[BITS];
#pragma unroll
    for (int b = 0; b < BITS; ++b) {
        m[b] = (int32_t)(d << (31 - b)) >> 31;
        bal[b] = __ballot(m[b] < 0);
    }
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
#pragma unroll
    for (int b = 0; b < BITS; ++b) {
        lo &= ~((uint32_t)bal[b] ^ (uint32_t)m[b]);
        hi &= ~((uint32_t)(bal[b] >> 32) ^ (uint32_t)m[b]);
    }
    return ((uint64_t)hi << 32) | lo;
}

// Geometry of the bucket sort for a key of st.sort_bits (at most 32) bits: the
// fine bin of a compacted key is key >> shF (its top 12 bits, or all of them);
// a bucket spans at most 2^spanlog fine bins (so the key bits below its first
// bin fit 24), and A buckets share the items out by count, the bins'
// spans adding at most kMsFine >> spanlog more.
struct MsGeom {
    uint32_t shF, spanlog, A;
};
__device__ inline MsGeom ms_geom(const SortStats& st) {
    MsGeom g;
    const uint32_t F = st.sort_bits < (uint32_t)kMsFineBits ? st.sort_bits : (uint32_t)kMsFineBits;
    g.shF = st.sort_bits - F;
    g.spanlog = 24 - g.shF;
    g.A = kMsMaxBuckets - 1 - (kMsFine >> (g.spanlog < 31 ? g.spanlog : 31));
    return g;
}
// the bucket of fine bin f, whose items start at excl; sc = A / total (0 with no
// items).  A product with a rounded scale rather than a 64-bit division: still
// non-decreasing in f (a correctly rounded product is monotone), and the same
// in every block.
__device__ inline uint32_t ms_bucket_of(const MsGeom& g, uint32_t f, uint32_t excl, double sc) {
    uint32_t a = (uint32_t)((double)excl * sc);
    if (a > g.A - 1) a = g.A - 1;
    return a + (f >> g.spanlog);
}

// Statistics (block 0 stores them) and the digit histograms of every pass
// that the significant bits need, over this block's keys.
// Blocks of kRhThreads threads over kRhTile keys: four times as many blocks
// as pass tiles, so that the whole chip counts (the counting is short, and
// its time goes into waiting for loads), up to kRhMaxBlocks that stride over
// the rest.  Block b also clears the look-back words of pass 0 and of the
// consumer's scan of pass tiles b, b + grid, ...
// With `msd` (one block per kRhTile keys) each block adds its fine-bin counts
// to fhist instead of the digit counts (the bucket sort's fallback counts
// those itself).
__global__ __launch_bounds__(kRhThreads) void k_rs_hist(RadixWs w, const int64_t* count_dev, int64_t cap,
                                                         uint32_t nrec, int64_t ntiles, int msd) {
    static_assert(kRsBins == kRhThreads, "thread t clears digit t's look-back word");
    const int64_t count = rs_count(count_dev, cap);
    const int64_t base = (int64_t)blockIdx.x * kRhTile;
    uint64_t raw[kRsItems];  // loaded before the statistics are reduced (no dependence between the two)
#pragma unroll
    for (int r = 0; r < kRsItems; ++r) {
        const int64_t i = base + r * kRhThreads + threadIdx.x;
        raw[r] = i < count ? w.ka[i] : 0ull;
    }
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        w.status[(size_t)tile * kRsBins + threadIdx.x] = 0ull;
        if (threadIdx.x == 0) w.status[(size_t)kRsPasses * kRsBins * w.ntiles + tile] = 0ull;
    }
    SortStats st;
    rs_reduce_stats(w.rec, nrec, count, &st);
    if (blockIdx.x == 0 && threadIdx.x == 0) *w.st = st;
    __shared__ uint32_t hist[kRsPasses][kRsBins];
    __shared__ uint32_t fh[kMsFine];
    for (int e = threadIdx.x; e < kRsPasses * kRsBins; e += kRhThreads) (&hist[0][0])[e] = 0;
    if (msd)
        for (int e = threadIdx.x; e < kMsFine; e += kRhThreads) fh[e] = 0;
    __syncthreads();
    const int passes = rs_passes(st);
    const uint32_t shF = ms_geom(st).shF;
    // grid-stride over blocks of kRhTile keys (the first one's keys are loaded above)
    for (int64_t b0 = base; b0 < count; b0 += (int64_t)gridDim.x * kRhTile) {
        if (b0 != base) {
#pragma unroll
            for (int r = 0; r < kRsItems; ++r) {
                const int64_t i = b0 + r * kRhThreads + threadIdx.x;
                raw[r] = i < count ? w.ka[i] : 0ull;
            }
        }
#pragma unroll
        for (int r = 0; r < kRsItems; ++r) {
            const int64_t i = b0 + r * kRhThreads + threadIdx.x;
            if (i < count) {
                const uint64_t ck = rs_compact(raw[r], st);
                if (msd) {
                    if (st.sort_bits <= 32) atomicAdd(&fh[(uint32_t)(ck >> shF)], 1u);  // LDS
                } else {
                    for (int p = 0; p < passes; ++p)
                        atomicAdd(&hist[p][(uint32_t)(ck >> (kRsBits * p)) & (kRsBins - 1)], 1u);  // LDS
                }
            }
        }
    }
    __syncthreads();
    if (!msd)
        for (int e = threadIdx.x; e < passes * kRsBins; e += kRhThreads) {
            const uint32_t c = (&hist[0][0])[e];
            if (c) atomicAdd(&w.ghist[e], c);
        }
    if (msd)
        for (int e = threadIdx.x; e < kMsFine; e += kRhThreads) {
            const uint32_t c = fh[e];
            if (c) atomicAdd(&w.fhist[e], c);
        }
}

// The bucket table the scatter's block 0 publishes: starts[kMsMaxBuckets + 1]
// (positions), first fine bins[kMsMaxBuckets + 1], then the bucket count.
__device__ inline uint32_t* ms_starts(const RadixWs& w) { return w.sb; }
__device__ inline uint32_t* ms_firsts(const RadixWs& w) { return w.sb + kMsMaxBuckets + 1; }
__device__ inline uint32_t* ms_count(const RadixWs& w) { return w.sb + 2 * (kMsMaxBuckets + 1); }

// Every item into its fine bin, stable within the block: the bin's base (items
// of smaller bins), plus the block's share of the bin (claimed with one atomic
// per bin and block, in whatever order the blocks come), plus the item's rank
// among the block's items of that bin.  Wave q holds the block's keys
// [q * 256, (q + 1) * 256) in four rounds of 64, so its running count of a bin
// (in LDS, read by every lane and advanced by the bin's first lane) and the
// counts of the waves before give the rank in index order.  Every block also
// groups the fine bins into buckets from the global counts (the same table in
// every block), and takes the bucket sort only if no bucket is over kMsCap;
// block 0 publishes the table and records that the bucket sort runs (st.msd).
// An item leaves as one word: its original index above its compacted key.
__global__ __launch_bounds__(kRhThreads) void k_ms_scatter(RadixWs w, const int64_t* count_dev, int64_t cap) {
    constexpr int NWV = kRhThreads / 64;
    constexpr int BPT = kMsFine / kRhThreads;  // fine bins per thread
    static_assert(kRsItems * 64 * NWV == kRhTile, "a wave holds kRsItems rounds of 64 keys");
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const SortStats st = *w.st;
    if (st.n_invalid != 0 || st.sort_bits > 32) return;
    const MsGeom g = ms_geom(st);
    const int64_t count = rs_count(count_dev, cap);
    const int64_t base = (int64_t)blockIdx.x * kRhTile;
    uint64_t raw[kRsItems];
#pragma unroll
    for (int r = 0; r < kRsItems; ++r) {
        const int64_t i = base + wave * (kRsItems * 64) + r * 64 + lane;
        raw[r] = i < count ? w.ka[i] : 0ull;
    }
    __shared__ uint16_t wcnt[NWV][kMsFine];  // per-wave running counts, then the waves' offsets in the block's share
    __shared__ uint32_t fbase[kMsFine];      // each fine bin's first position, then the block's in it
    __shared__ uint32_t sbs[kMsMaxBuckets + 1], sbf[kMsMaxBuckets + 1];
    __shared__ int lds[NWV + 1];
    __shared__ uint32_t s_nb;
    // thread t: fine bins [t * BPT, (t + 1) * BPT) and their first positions
    uint32_t h[BPT];
    {
        const uint4* src = (const uint4*)(w.fhist + t * BPT);
#pragma unroll
        for (int q = 0; q < BPT / 4; ++q) {
            const uint4 v = src[q];
            h[4 * q] = v.x;
            h[4 * q + 1] = v.y;
            h[4 * q + 2] = v.z;
            h[4 * q + 3] = v.w;
        }
    }
    const uint32_t hprev = t > 0 ? w.fhist[t * BPT - 1] : 0u;
    uint32_t sum = 0;
#pragma unroll
    for (int j = 0; j < BPT; ++j) sum += h[j];
    int total_i;
    uint32_t e[BPT];
    e[0] = (uint32_t)block_exclusive_scan((int)sum, lds, &total_i);
#pragma unroll
    for (int j = 1; j < BPT; ++j) e[j] = e[j - 1] + h[j - 1];
    const uint32_t total = (uint32_t)total_i;
    const double sc = total ? (double)g.A / (double)total : 0.0;
    // bucket table: bucket b starts at the first fine bin whose bucket is b
    // (buckets left empty by a jump start where the next one does)
    {
        int64_t bp = -1;
        if (t > 0) bp = ms_bucket_of(g, (uint32_t)(t * BPT - 1), e[0] - hprev, sc);
#pragma unroll
        for (int j = 0; j < BPT; ++j) {
            const uint32_t f = (uint32_t)(t * BPT + j);
            const uint32_t b = ms_bucket_of(g, f, e[j], sc);
            for (int64_t q = bp + 1; q <= (int64_t)b; ++q) {
                sbs[q] = e[j];
                sbf[q] = f;
            }
            bp = b;
        }
        if (t == kRhThreads - 1) {
            sbs[bp + 1] = total;
            sbf[bp + 1] = kMsFine;
            s_nb = (uint32_t)(bp + 1);
        }
    }
    __syncthreads();
    const uint32_t nb = s_nb;
    bool over = false;
    for (uint32_t q = t; q < nb; q += kRhThreads) over |= sbs[q + 1] - sbs[q] > (uint32_t)kMsCap;
    if (__syncthreads_or(over)) return;
    if (blockIdx.x == 0) {
        for (uint32_t q = t; q <= nb; q += kRhThreads) {
            ms_starts(w)[q] = sbs[q];
            ms_firsts(w)[q] = sbf[q];
        }
        if (t == 0) {
            *ms_count(w) = nb;
            w.st->msd = 1u;
        }
    }
    if (base >= count) return;
    {
        uint4* z = (uint4*)&wcnt[0][0];
        for (int q = t; q < (int)(sizeof(wcnt) / 16); q += kRhThreads) z[q] = make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int j = 0; j < BPT; ++j) fbase[t * BPT + j] = e[j];
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint32_t ck[kRsItems], fb[kRsItems], rk[kRsItems];
#pragma unroll
    for (int r = 0; r < kRsItems; ++r) {
        const bool valid = base + wave * (kRsItems * 64) + r * 64 + lane < count;
        ck[r] = valid ? (uint32_t)rs_compact(raw[r], st) : 0u;
        fb[r] = ck[r] >> g.shF;
        const uint64_t peers = rs_peers<kMsFineBits>(fb[r], valid);
        const uint32_t lr = (uint32_t)__popcll(peers & lt);
        const uint32_t prev = wcnt[wave][fb[r]];
        rk[r] = prev + lr;
        if (valid && lr == 0) wcnt[wave][fb[r]] = (uint16_t)(prev + __popcll(peers));
    }
    __syncthreads();
    // claim the block's share of each fine bin it holds: thread t takes bins
    // t, t + 256, ... (a block's keys fill few, nearby bins: spread over the
    // threads, their atomics go out together instead of one after another)
    uint32_t claim[BPT];
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
        const int f = t + kRhThreads * j;
        uint32_t tot = 0;
#pragma unroll
        for (int q = 0; q < NWV; ++q) tot += wcnt[q][f];
        claim[j] = tot ? atomicAdd(&w.fcur[f], tot) : 0u;
    }
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
        const int f = t + kRhThreads * j;
        uint32_t run = 0;
#pragma unroll
        for (int q = 0; q < NWV; ++q) {
            const uint32_t c = wcnt[q][f];
            wcnt[q][f] = (uint16_t)run;
            run += c;
        }
        if (run) fbase[f] += claim[j];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRsItems; ++r) {
        const int64_t i = base + wave * (kRsItems * 64) + r * 64 + lane;
        if (i < count) {
            const uint32_t pos = fbase[fb[r]] + wcnt[wave][fb[r]] + rk[r];
            w.kb[pos] = ((uint64_t)(uint32_t)i << 32) | ck[r];
        }
    }
}


__device__ inline uint64_t rs_load_status(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void rs_store_status(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive prefix of this tile's count for one digit: the counts of the tiles
// before it, read WINDOW at a time from the nearest down, until a tile that
// holds its inclusive prefix.  A status word not yet written is polled again
// (the tile that writes it is running); after kRsSpinLimit polls the sort
// records an error and goes on without it, so the kernel always ends.
constexpr int kRsWindow = 32;
template <int WINDOW = kRsWindow>
__device__ inline uint32_t rs_lookback(const uint64_t* col, int64_t stride, int64_t tile, bool& stalled) {
    uint32_t excl = 0;
    int64_t j = tile - 1;
    uint32_t spins = 0;
    while (j >= 0) {
        uint64_t s[WINDOW];
#pragma unroll
        for (int q = 0; q < WINDOW; ++q) s[q] = (j - q >= 0) ? rs_load_status(col + (j - q) * stride) : kRsFlagInc;
        int q = 0;
        bool done = false;
        for (; q < WINDOW; ++q) {
            const uint64_t f = s[q] & (3ull << 62);
            if (f == 0) break;  // not written yet: read it again
            excl += (uint32_t)s[q];
            if (f == kRsFlagInc) {
                done = true;
                break;
            }
        }
        if (done) break;
        j -= q;
        if (q == 0) {
            if (++spins > kRsSpinLimit) {
                stalled = true;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    return excl;
}

// dynamic LDS of a pass: per (round, wave, digit) counts, then offsets relative
// to the tile's first item of that digit (both at most kRsTile: 16 bits)
constexpr size_t kRsPassLds = (size_t)kRsItems * (kRsThreads / 64) * kRsBins * sizeof(uint16_t);

// One tile of one pass: the tile is taken from the pass's counter (tiles get
// their place in the order they start, so every tile a reader waits for is
// already running).  Returns false, with no work done, once the pass's tiles
// are all taken.
template <bool FIRST, int WINDOW = kRsWindow>
__device__ inline bool rs_pass_tile(const RadixWs& w, Header* h, int64_t count, int64_t ntiles, int pass,
                                    unsigned char* rs_smem) {
    static_assert(kRsBins <= kRsThreads, "threads t < kRsBins own digit t");
    constexpr int NWV = kRsThreads / 64;
    uint16_t (*cnt)[NWV][kRsBins] = (uint16_t (*)[NWV][kRsBins])rs_smem;
    __shared__ uint32_t dbase[kRsBins];  // the digit's first output position for this tile
    __shared__ int lds[NWV + 1];
    __shared__ uint32_t s_tile;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if (t == 0) s_tile = atomicAdd(&w.ctr[pass], 1u);
    const bool owner = t < kRsBins;
    const uint32_t gcount = owner ? w.ghist[pass * kRsBins + t] : 0u;
    {
        uint4* z = (uint4*)rs_smem;
        for (size_t e = t; e < kRsPassLds / 16; e += kRsThreads) z[e] = make_uint4(0u, 0u, 0u, 0u);
    }
    __syncthreads();
    const int64_t tile = s_tile;
    if (tile >= ntiles) return false;
    const int64_t base = tile * kRsTile;
    const uint64_t* ksrc = (pass & 1) ? w.kb : w.ka;
    uint64_t* kdst = (pass & 1) ? w.ka : w.kb;
    const uint32_t* vsrc = (pass & 1) ? w.vb : w.va;
    uint32_t* vdst = (pass & 1) ? w.va : w.vb;
    uint64_t keys[kRsItems];
    uint32_t vals[kRsItems];
#pragma unroll
    for (int r = 0; r < kRsItems; ++r) {
        const int64_t i = base + r * kRsThreads + t;
        keys[r] = i < count ? ksrc[i] : 0ull;
        if constexpr (FIRST) vals[r] = (uint32_t)i;  // the first pass sorts the item indices
        else vals[r] = i < count ? vsrc[i] : 0u;
    }
    // the next pass's look-back words of this tile start empty (that pass starts after this one ends)
    if (owner && pass + 1 < kRsPasses) w.status[((size_t)(pass + 1) * w.ntiles + tile) * kRsBins + t] = 0ull;
    // bucket base of digit t: all keys of smaller digits
    int all;
    const uint32_t gbase = (uint32_t)block_exclusive_scan((int)gcount, lds, &all);
    if constexpr (FIRST) {
        const SortStats st = *w.st;
#pragma unroll
        for (int r = 0; r < kRsItems; ++r)
            if (base + r * kRsThreads + t < count) keys[r] = rs_compact(keys[r], st);
    }
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint32_t rank[kRsItems];
#pragma unroll
    for (int r = 0; r < kRsItems; ++r) {
        const int64_t i = base + r * kRsThreads + t;
        const bool valid = i < count;
        const uint32_t d = (uint32_t)(keys[r] >> (kRsBits * pass)) & (kRsBins - 1);
        const uint64_t peers = rs_peers(d, valid);
        rank[r] = (uint32_t)__popcll(peers & lt);
        if (valid && rank[r] == 0) cnt[r][wave][d] = (uint16_t)__popcll(peers);
    }
    __syncthreads();
    if (owner) {
        // thread t: the tile's count of digit t, published before the look-back
        uint32_t tot = 0;
#pragma unroll
        for (int r = 0; r < kRsItems; ++r)
#pragma unroll
            for (int q = 0; q < NWV; ++q) tot += (uint32_t)cnt[r][q][t];
        uint64_t* col = w.status + (size_t)pass * kRsBins * w.ntiles + t;  // status[pass][tile][digit]
        bool stalled = false;
        uint32_t excl = 0;
        if (tile == 0) {
            rs_store_status(col, kRsFlagInc | tot);
        } else {
            rs_store_status(col + tile * kRsBins, kRsFlagAgg | tot);
            excl = rs_lookback<WINDOW>(col, kRsBins, tile, stalled);
            rs_store_status(col + tile * kRsBins, kRsFlagInc | (uint64_t)(excl + tot));
        }
        if (stalled) raise_flag(h, kFlagInternal);
        // offsets over (round, wave) in index order, relative to the digit's base
        dbase[t] = gbase + excl;
        uint32_t run = 0;
#pragma unroll
        for (int r = 0; r < kRsItems; ++r)
#pragma unroll
            for (int q = 0; q < NWV; ++q) {
                const uint32_t c = cnt[r][q][t];
                cnt[r][q][t] = (uint16_t)run;
                run += c;
            }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRsItems; ++r) {
        const int64_t i = base + r * kRsThreads + t;
        if (i < count) {
            const uint32_t d = (uint32_t)(keys[r] >> (kRsBits * pass)) & (kRsBins - 1);
            const uint32_t pos = dbase[d] + cnt[r][wave][d] + rank[r];
            kdst[pos] = keys[r];
            vdst[pos] = vals[r];
        }
    }
    return true;
}

// dynamic LDS of a pass is declared by the kernels: per (round, wave, digit)
// counts, then offsets relative to the tile's first item of that digit
template <bool FIRST>
__global__ __launch_bounds__(kRsThreads) void k_rs_pass(RadixWs w, Header* h, const int64_t* count_dev, int64_t cap,
                                                        int pass) {
    // the first pass always runs: it writes the compacted keys and the payload
    if (pass > 0 && (uint32_t)(kRsBits * pass) >= w.st->sort_bits) return;
    extern __shared__ __align__(16) unsigned char rs_smem[];
    rs_pass_tile<FIRST>(w, h, rs_count(count_dev, cap), (int64_t)gridDim.x, pass, rs_smem);
}

// Grid barrier (slot `slot` of the counters) of the first `parts` workgroups:
// each wave releases its writes before the arrival and acquires after it.  A
// wait past kRsSpinLimit polls records an error and goes on, so every
// workgroup ends.
__device__ inline void rs_grid_barrier(const RadixWs& w, Header* h, int slot, uint32_t parts) {
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t* bar = &w.ctr[kRsBarrierCtr + slot];
        atomicAdd(bar, 1u);
        uint32_t spins = 0;
        while (__hip_atomic_load(bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < parts) {
            if (++spins > kRsSpinLimit) {
                raise_flag(h, kFlagInternal);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    __syncthreads();
    __threadfence();
}

// The passes from `first` on by `parts` co-resident workgroups that loop over
// the tiles, a grid barrier between two passes (pass 0 always runs: it writes
// the compacted keys and the payload).  With first = 0 the workgroups first
// count the digits of every pass (the histogram kernel of the bucket sort
// counted only its fine bins).  smem: kRsPassLds bytes.  WINDOW: status words
// a look-back reads at a time (fewer where registers are scarcer).
template <int WINDOW = kRsWindow>
__device__ inline void rs_tail_run(const RadixWs& w, Header* h, int64_t count, int64_t ntiles, int first,
                                   uint32_t parts, unsigned char* smem) {
    const uint32_t bits = w.st->sort_bits;
    if (first == 0) {
        const SortStats st = *w.st;
        const int passes = rs_passes(st);
        uint32_t* hist = (uint32_t*)smem;  // [kRsPasses][kRsBins], 8 KB of the pass's LDS
        for (int e = threadIdx.x; e < kRsPasses * kRsBins; e += kRsThreads) hist[e] = 0u;
        __syncthreads();
        for (int64_t i = blockIdx.x * (int64_t)kRsThreads + threadIdx.x; i < count; i += (int64_t)parts * kRsThreads) {
            const uint64_t ck = rs_compact(w.ka[i], st);
            for (int p = 0; p < passes; ++p)
                atomicAdd(&hist[p * kRsBins + ((uint32_t)(ck >> (kRsBits * p)) & (kRsBins - 1))], 1u);  // LDS
        }
        __syncthreads();
        for (int e = threadIdx.x; e < passes * kRsBins; e += kRsThreads) {
            const uint32_t c = hist[e];
            if (c) atomicAdd(&w.ghist[e], c);
        }
        rs_grid_barrier(w, h, 0, parts);  // every count is in before pass 0 reads them
    }
    for (int pass = first; pass < kRsPasses && (pass == 0 || (uint32_t)(kRsBits * pass) < bits); ++pass) {
        if (pass > first) rs_grid_barrier(w, h, pass, parts);
        if (pass == 0) {
            while (rs_pass_tile<true, WINDOW>(w, h, count, ntiles, pass, smem)) __syncthreads();
        } else {
            while (rs_pass_tile<false, WINDOW>(w, h, count, ntiles, pass, smem)) __syncthreads();
        }
    }
}

// The passes from `first` on in one launch, one workgroup per tile, all
// resident.  A key of at most 8 * first significant bits (the usual case)
// makes it exit at once, so the passes that are not needed cost one launch,
// not one each.
__global__ __launch_bounds__(kRsThreads) void k_rs_tail(RadixWs w, Header* h, const int64_t* count_dev, int64_t cap,
                                                        int first, int64_t ntiles) {
    if ((uint32_t)(kRsBits * first) >= w.st->sort_bits) return;
    extern __shared__ __align__(16) unsigned char rs_smem[];
    rs_tail_run(w, h, rs_count(count_dev, cap), ntiles, first, gridDim.x, rs_smem);
}

// One workgroup per bucket: its items (in kb, grouped by fine bin, each
// block's share of a bin in index order) sorted by the key bits below the
// bucket's first fine bin and then by the item's block, 8 bits at a time, in
// LDS -- which leaves equal keys in index order.  Wave q holds the items
// [q * R * 64, (q + 1) * R * 64) of the current order, R = ceil(size / 512)
// rounds of 64; an item's new place is the count of items of smaller digit
// plus those of its digit in the waves before plus the wave's running count of
// that digit (in LDS, read by every lane and advanced by the digit's first
// lane, round by round).  The sorted bucket goes to ka / va at the same
// positions.  When the bucket sort cannot order the keys, the first ntiles
// workgroups run every pass instead (one tile each, all resident: two of these
// workgroups fit a CU) and the others exit.
__global__ __launch_bounds__(kMsThreads) void k_ms_bucket(RadixWs w, Header* h, const int64_t* count_dev, int64_t cap,
                                                          int64_t ntiles) {
    static_assert(kMsThreads == kRsThreads, "the fallback's pass tiles take the same workgroup");
    constexpr int NWV = kMsThreads / 64;
    static_assert(kRsBins * 2 == kMsThreads, "thread t scans digit t / 2 over waves 4 (t % 2) ..");
    static_assert(kMsMaxBlocks <= 256 && kRhTile == 1024, "an item's block is its index >> 10, 8 bits");
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    __shared__ uint64_t buf[kMsCap];
    const SortStats st = *w.st;
    if (!st.msd) {
        if (blockIdx.x < ntiles)
            rs_tail_run<8>(w, h, rs_count(count_dev, cap), ntiles, 0, (uint32_t)ntiles, (unsigned char*)buf);
        return;
    }
    const uint32_t b = blockIdx.x;
    if (b >= *ms_count(w)) return;
    const uint32_t start = ms_starts(w)[b];
    const uint32_t size = ms_starts(w)[b + 1] - start;
    if (size == 0) return;
    const MsGeom g = ms_geom(st);
    const uint32_t f0 = ms_firsts(w)[b];
    const uint32_t kbase = f0 << g.shF;  // the bucket's smallest possible key
    const uint32_t span = (ms_firsts(w)[b + 1] - f0) << g.shF;  // at most 2^24
    const int bits = (span > 1 ? 32 - __clz(span - 1) : 0) + 8;  // key below kbase, then the block
    const uint32_t R = (size + kMsThreads - 1) / kMsThreads;
    // this wave's rounds that hold items (rounds past the bucket are skipped)
    const uint32_t first = wave * R * 64;
    const uint32_t Rw = first >= size ? 0u : ((size - first + 63) / 64 < R ? (size - first + 63) / 64 : R);
    uint32_t key[kMsRounds], val[kMsRounds], rk[kMsRounds];
#pragma unroll
    for (int r = 0; r < kMsRounds; ++r) {
        const uint32_t e = (wave * R + r) * 64 + lane;
        const uint64_t x = ((uint32_t)r < R && e < size) ? w.kb[start + e] : 0ull;
        val[r] = (uint32_t)(x >> 32);
        key[r] = (((uint32_t)x - kbase) << 8) | (val[r] >> 10);
    }
    __shared__ uint32_t wc[NWV][kRsBins];
    __shared__ int lds[NWV + 1];
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int passes = (bits + kRsBits - 1) / kRsBits;
    for (int p = 0; p < passes; ++p) {
        // the wave's counts start at zero (the last pass's readers have passed
        // the barrier after the scatter)
        for (int e = lane; e < kRsBins; e += 64) wc[wave][e] = 0u;
        const int nb = bits - kRsBits * p < kRsBits ? bits - kRsBits * p : kRsBits;  // bits of this digit
#pragma unroll
        for (int r = 0; r < kMsRounds; ++r) {
            if ((uint32_t)r >= Rw) continue;
            const uint32_t e = (wave * R + r) * 64 + lane;
            const bool valid = e < size;
            const uint32_t d = (key[r] >> (kRsBits * p)) & (kRsBins - 1);
            const uint64_t peers = rs_peers(d, valid, nb);
            const uint32_t lr = (uint32_t)__popcll(peers & lt);
            // every lane reads the count before the digit's first lane adds this
            // round's (one wave's LDS accesses take effect in program order)
            const uint32_t prev = wc[wave][d];
            rk[r] = prev + lr;
            if (valid && lr == 0) wc[wave][d] = prev + (uint32_t)__popcll(peers);
        }
        __syncthreads();
        {
            // offsets in (digit, wave) order
            const int d = t >> 1, q0 = (t & 1) * 4;
            uint32_t c[4], sum = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                c[j] = wc[q0 + j][d];
                sum += c[j];
            }
            int tot;
            uint32_t run = (uint32_t)block_exclusive_scan((int)sum, lds, &tot);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                wc[q0 + j][d] = run;
                run += c[j];
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kMsRounds; ++r) {
            if ((uint32_t)r >= Rw) continue;
            const uint32_t e = (wave * R + r) * 64 + lane;
            if (e < size) {
                const uint32_t d = (key[r] >> (kRsBits * p)) & (kRsBins - 1);
                buf[wc[wave][d] + rk[r]] = ((uint64_t)val[r] << 32) | key[r];
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kMsRounds; ++r) {
            if ((uint32_t)r >= Rw) continue;
            const uint32_t e = (wave * R + r) * 64 + lane;
            if (e < size) {
                const uint64_t x = buf[e];
                key[r] = (uint32_t)x;
                val[r] = (uint32_t)(x >> 32);
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < kMsRounds; ++r) {
        if ((uint32_t)r >= Rw) continue;
        const uint32_t e = (wave * R + r) * 64 + lane;
        if (e < size) {
            w.ka[start + e] = (uint64_t)(kbase + (key[r] >> 8));
            w.va[start + e] = val[r];
        }
    }
}

void launch_radix_sort(hipStream_t s, const RadixWs& w, Header* h, const int64_t* count_dev, int64_t cap,
                       uint32_t nrec) {
    if (cap < 0) cap = 0;
    const unsigned nt = (unsigned)radix_tiles(cap);  // at least one tile: the first pass always writes its outputs
    static const bool lds_ok =
        hipFuncSetAttribute((const void*)k_rs_pass<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)kRsPassLds) == hipSuccess &&
        hipFuncSetAttribute((const void*)k_rs_pass<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)kRsPassLds) == hipSuccess &&
        hipFuncSetAttribute((const void*)k_rs_tail, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)kRsPassLds) == hipSuccess;
    (void)lds_ok;
    // at most kRhMaxBlocks blocks (each adds its counts with global atomics)
    unsigned nh = (unsigned)blocks_for(cap > 0 ? cap : 1, kRhTile);
    if (nh <= kMsMaxBlocks) {
        // the bucket sort; when it cannot order the keys, the bucket kernel's
        // first workgroups run the passes instead
        k_rs_hist<<<nh, kRhThreads, 0, s>>>(w, count_dev, cap, nrec, (int64_t)nt, 1);
        k_ms_scatter<<<nh, kRhThreads, 0, s>>>(w, count_dev, cap);
        k_ms_bucket<<<kMsMaxBuckets, kMsThreads, 0, s>>>(w, h, count_dev, cap, (int64_t)nt);
        return;
    }
    if (nh > kRhMaxBlocks) nh = kRhMaxBlocks;
    k_rs_hist<<<nh, kRhThreads, 0, s>>>(w, count_dev, cap, nrec, (int64_t)nt, 0);
    // the significant bits are known on the device only: the first kRsHeadPasses
    // passes are a launch each (a pass past the bits exits at once), and the
    // passes after them share one launch
    k_rs_pass<true><<<nt, kRsThreads, kRsPassLds, s>>>(w, h, count_dev, cap, 0);
    // up to kRsTailTiles tiles, the passes after the head share one launch
    // (one workgroup per tile, all resident for the grid barrier); a larger
    // sort launches them one by one, where a launch that exits at once is
    // cheap against the passes themselves
    const int head = nt <= kRsTailTiles ? kRsHeadPasses : kRsPasses;
    for (int p = 1; p < head; ++p) k_rs_pass<false><<<nt, kRsThreads, kRsPassLds, s>>>(w, h, count_dev, cap, p);
    if (head < kRsPasses) k_rs_tail<<<nt, kRsThreads, kRsPassLds, s>>>(w, h, count_dev, cap, head, (int64_t)nt);
}

}  // namespace spv
