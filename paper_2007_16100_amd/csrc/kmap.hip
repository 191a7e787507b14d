// kmap.hip -- kernel-map construction on the voxel hash (Sec. 3.2: the active
// synapses between input and output voxels; Sec. 3.3 "Feature Aggregation":
// built with the same GPU hash table as the voxelization).
//
// Outputs: CSR by offset k -- off[K^3+1] and pairs (in, out), each offset's
// pairs sorted by out.
//
// Submanifold 3x3x3 maps (outputs = inputs), blocks of 64 output voxels:
//   pass 1: the dense neighbour table nbr[j][k] = i + 1 (0 = no voxel), one
//           hash probe per (voxel, offset) with a wave's probes issued together,
//           and per-(offset, block) pair counts from wave ballots;
//   scan:   one exclusive scan over the offset-major (offset, block) counts
//           gives every block its write position inside every offset's segment;
//   pass 2: reads the table back and writes the pairs at their final, sorted
//           positions (rank inside the block from ballots) -> deterministic,
//           already-sorted output without atomics.
// The 3x3x3 convolution consumes the neighbour table directly, so a block that
// only needs the convolution stops after pass 1.
// Stride 2: the output voxels are the distinct floor(c/2), deduplicated in a
// second hash table and radix-sorted into canonical order.  K = 2: the pairs are
// a stable partition of the inputs by coordinate parity (a count pass, one scan,
// a write pass with one coarse-table lookup per input).  K = 3: the same three
// passes as the submanifold map, run over the output voxels, with output C
// probing the input table at 2C + delta (a probe outside the key range is
// absent: no input can sit there).
#include "spv_internal.hpp"

namespace spv {

constexpr int kMapThreads = 256;
constexpr int kNbrVox = 64;    // output voxels per block of the 3x3x3 passes (one per lane)
constexpr int kNbrWaves = 8;   // waves per block of the 3x3x3 passes
constexpr int kNbrProbes = 4;  // offsets per wave: wave w takes k = w, w + 8, ..., < 27

void plan_kmap_ws(Arena& a, KmapWs& w, int64_t m_cap, int K, int stride, bool own_fine_table, bool own_nbr) {
    int64_t mc = m_cap > 0 ? m_cap : 1;
    const int K3 = K * K * K;
    if (own_fine_table) {
        uint32_t S = table_capacity(mc);
        w.fine = take_table(a, S);
    }
    if (stride == 2) {
        uint32_t S = table_capacity(mc);
        w.coarse = take_table(a, S);
        plan_radix_ws(a, w.rs, mc);
    } else {
        w.coarse = Table{nullptr, 0};
    }
    size_t nblk = blocks_for(mc, K == 3 ? kNbrVox : kMapThreads);
    w.bcnt = a.take<uint32_t>(K3 * nblk);
    w.bbase = a.take<uint32_t>(K3 * nblk + 1);
    w.scan_tmp = a.take<int32_t>(scan_tmp_entries((int64_t)K3 * nblk));
    w.m_out = a.take<int64_t>(2);
    w.nbr = (K == 3 && own_nbr) ? a.take<int32_t>((size_t)mc * 27) : nullptr;
}

__device__ inline int64_t count_or_cap(const int64_t* d, int64_t cap) {
    if (!d) return cap;
    int64_t c = *d;
    return c < 0 ? 0 : (c > cap ? cap : c);
}

template <int K>
__device__ inline void offset_delta(int k, int& dx, int& dy, int& dz) {
    if constexpr (K == 3) {
        dx = k / 9 - 1;
        dy = (k / 3) % 3 - 1;
        dz = k % 3 - 1;
    } else {
        dx = (k >> 2) & 1;
        dy = (k >> 1) & 1;
        dz = k & 1;
    }
}

// outputs = inputs (stride 1)
__global__ void k_map_same_count(const int64_t* m_in_dev, int64_t cap, int64_t* m_out, int64_t* m_out_user) {
    int64_t m = count_or_cap(m_in_dev, cap);
    m_out[0] = m;
    if (m_out_user) *m_out_user = m;
}

// stride 2: coarse keys into the coarse table; each block appends the keys it
// created to the key list and records their per-field min / max for the sort
// Every input's coarse key floor(c / 2) into the coarse table; each key the
// table did not hold yet is appended to the sort's key list (rs.ka, counter
// cnt).  Grid-stride over the inputs, one sort record per block (per-field
// minima / maxima of the block's new keys, no invalid items); the same launch
// zeroes the sort's counters and histograms.
__global__ __launch_bounds__(kAppendThreads) void k_map_coarse_insert(Header* h, Table coarse, RadixWs rs,
                                                                      int64_t nzero, int64_t* cnt,
                                                                      const int32_t* in_coords,
                                                                      const int64_t* m_in_dev, int64_t cap) {
    const int64_t m = count_or_cap(m_in_dev, cap);
    const int64_t stride = (int64_t)gridDim.x * kAppendThreads;
    for (int64_t i = blockIdx.x * (int64_t)kAppendThreads + threadIdx.x; i < nzero; i += stride) rs.zero[i] = 0u;
    int mn[4] = {0x7fffffff, 0x7fffffff, 0x7fffffff, 0x7fffffff};
    int mx[4] = {(int)0x80000000, (int)0x80000000, (int)0x80000000, (int)0x80000000};
    for (int64_t b0 = blockIdx.x * (int64_t)kAppendThreads; b0 < m; b0 += stride) {  // the same trip count in the block
        const int64_t i = b0 + threadIdx.x;
        bool created = false;
        uint64_t key = kEmpty;
        int f[4] = {0, 0, 0, 0};
        if (i < m) {
            const int32_t* c = in_coords + 4 * i;
            // floor(c / 2) via arithmetic shift
            f[0] = c[0];
            f[1] = c[1] >> 1;
            f[2] = c[2] >> 1;
            f[3] = c[3] >> 1;
            key = pack_key(f[0], f[1], f[2], f[3]);
        }
        // sorted fine voxels: neighbours in z often share a coarse voxel, and a lane
        // whose key equals the previous lane's leaves the insert to its run's head
        const uint64_t prev_key = __shfl_up(key, 1, 64);
        if (key != kEmpty && ((threadIdx.x & 63) == 0 || prev_key != key)) {
            uint32_t slot;
            const int r = table_insert(coarse, key, &slot);
            created = r > 0;
            if (r < 0) raise_flag(h, kFlagTableFull);
        }
        if (created) {
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                mn[d] = min(mn[d], f[d]);
                mx[d] = max(mx[d], f[d]);
            }
        }
        block_append(created, key, rs.ka, cnt);
    }
    int32_t* rec = rs.rec + (size_t)kRsRecWords * blockIdx.x;
    block_minmax_record(mn, mx, rec);
    if (threadIdx.x == 0) rec[8] = rec[9] = 0;  // no invalid keys
}

// The sorted coarse keys in order: output r's coordinates, and r as its
// coarse-table value.
__global__ void k_map_coarse_rank(RadixWs rs, Table coarse, const int64_t* cnt, int64_t cap, int32_t* out_coords,
                                  int64_t* m_out, int64_t* m_out_user) {
    int64_t m = count_or_cap(cnt, cap);
    int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (r == 0) {
        m_out[0] = m;
        if (m_out_user) *m_out_user = m;
    }
    if (r >= m) return;
    const SortStats st = *rs.st;
    const uint64_t key = rs_expand(rs_keys(rs, st)[r], st);
    int64_t slot = table_slot(coarse, key);
    if (slot >= 0) *slot_val(coarse, (uint32_t)slot) = (int32_t)r;
    out_coords[4 * r + 0] = key_b(key);
    out_coords[4 * r + 1] = key_x(key);
    out_coords[4 * r + 2] = key_y(key);
    out_coords[4 * r + 3] = key_z(key);
}

// Stride 2 (K = 2): input voxel i is in exactly one pair, (i, j, k) with j the
// index of floor(c_i / 2) and k = 4 (x & 1) + 2 (y & 1) + (z & 1).  Inside one
// parity class, c -> floor(c / 2) is increasing, so offset k's pairs are the
// class-k inputs in input order, already sorted by output: the map is a stable
// partition of the inputs by parity (per-block class counts, one scan, then
// every input written at its place).  No table of the inputs is needed.
__device__ inline int parity_k(const int32_t* c) { return ((c[1] & 1) << 2) | ((c[2] & 1) << 1) | (c[3] & 1); }

__global__ __launch_bounds__(kMapThreads) void k_s2_count(const int32_t* in_coords, const int64_t* m_in_dev,
                                                          int64_t cap, uint32_t* bcnt) {
    __shared__ uint32_t cnt[8];
    if (threadIdx.x < 8) cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t m = count_or_cap(m_in_dev, cap);
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int k = i < m ? parity_k(in_coords + 4 * i) : -1;
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const uint64_t bal = __ballot(k == q);
        if (lane == 0 && bal) atomicAdd(&cnt[q], (uint32_t)__popcll(bal));
    }
    __syncthreads();
    if (threadIdx.x < 8) bcnt[threadIdx.x * gridDim.x + blockIdx.x] = cnt[threadIdx.x];  // offset-major
}

__global__ __launch_bounds__(kMapThreads) void k_s2_write(Header* h, Table coarse, const int32_t* in_coords,
                                                          const int64_t* m_in_dev, int64_t cap, const uint32_t* bbase,
                                                          int32_t* off, int32_t* pairs, int64_t pair_cap) {
    constexpr int NW = kMapThreads / 64;
    __shared__ uint32_t wtot[NW][8];
    const uint32_t nblk = gridDim.x;
    if (blockIdx.x == 0) {
        for (int k = threadIdx.x; k <= 8; k += blockDim.x) off[k] = (int32_t)bbase[k * nblk];
    }
    const int64_t m = count_or_cap(m_in_dev, cap);
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const bool valid = i < m;
    int c[4] = {0, 0, 0, 0};
    if (valid) {
#pragma unroll
        for (int d = 0; d < 4; ++d) c[d] = in_coords[4 * i + d];
    }
    const int k = valid ? parity_k(c) : -1;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint32_t rank = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const uint64_t bal = __ballot(k == q);
        if (k == q) rank = (uint32_t)__popcll(bal & lt);
        if (lane == 0) wtot[wave][q] = (uint32_t)__popcll(bal);
    }
    __syncthreads();
    if (!valid) return;
    uint32_t pos = bbase[k * nblk + blockIdx.x] + rank;
    for (int w = 0; w < wave; ++w) pos += wtot[w][k];
    // floor(c / 2) by arithmetic shift, as the coarse keys were made
    const int32_t j = table_find(coarse, pack_key(c[0], c[1] >> 1, c[2] >> 1, c[3] >> 1));
    if ((int64_t)pos < pair_cap) {
        pairs[2 * (int64_t)pos] = (int32_t)i;
        pairs[2 * (int64_t)pos + 1] = j;
    } else {
        raise_flag(h, kFlagCapacity);
    }
}

// pass 1 of a 3x3x3 map (see the file comment); bcnt may be null.  S2: coords
// are the stride-2 outputs and offset k of output C probes 2C + delta_k.
// The block's 64 rows of the table are assembled in LDS and written out as one
// contiguous run.
template <bool S2>
__global__ __launch_bounds__(64 * kNbrWaves) void k_map_nbr3(Table fine, const int32_t* coords, const int64_t* m_out,
                                                  int64_t cap, int32_t* nbr, uint32_t* bcnt) {
    __shared__ int32_t tile[kNbrVox * 27];  // row stride 27 words: conflict-free per-lane writes
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t m = count_or_cap(m_out, cap);
    const int64_t j = (int64_t)blockIdx.x * kNbrVox + lane;
    const bool valid = j < m;
    int c[4] = {0, 0, 0, 0};
    if (valid) {
#pragma unroll
        for (int d = 0; d < 4; ++d) c[d] = coords[4 * j + d];
    }
    uint64_t key[kNbrProbes];
    bool act[kNbrProbes];
    int32_t res[kNbrProbes];
#pragma unroll
    for (int q = 0; q < kNbrProbes; ++q) {
        const int k = wave + kNbrWaves * q;
        int dx, dy, dz;
        offset_delta<3>(k, dx, dy, dz);
        if constexpr (S2) {
            const int x = 2 * c[1] + dx, y = 2 * c[2] + dy, z = 2 * c[3] + dz;
            act[q] = valid && k < 27 && in_key_range(x) && in_key_range(y) && in_key_range(z);
            key[q] = pack_key(c[0], x, y, z);
        } else {
            // the centre offset of a submanifold map is the voxel itself
            act[q] = valid && k < 27 && k != 13;
            key[q] = pack_key(c[0], c[1] + dx, c[2] + dy, c[3] + dz);
        }
    }
    table_find_n<kNbrProbes>(fine, key, act, res);
    const uint32_t nblk = gridDim.x;
#pragma unroll
    for (int q = 0; q < kNbrProbes; ++q) {
        const int k = wave + kNbrWaves * q;
        if (k >= 27) break;
        const int32_t i = (!S2 && k == 13) ? (int32_t)j : res[q];
        const bool present = valid && i >= 0;
        tile[lane * 27 + k] = present ? i + 1 : 0;
        if (bcnt) {
            const uint64_t bal = __ballot(present);
            if (lane == 0) bcnt[k * nblk + blockIdx.x] = (uint32_t)__popcll(bal);
        }
    }
    __syncthreads();
    const int64_t j0 = (int64_t)blockIdx.x * kNbrVox;
    const int rows = m - j0 < kNbrVox ? (int)(m - j0) : kNbrVox;
    for (int e = threadIdx.x; e < rows * 27; e += blockDim.x) nbr[j0 * 27 + e] = tile[e];
}

// pass 2 of a submanifold 3x3x3 map: pairs from the neighbour table
__global__ __launch_bounds__(64 * kNbrWaves) void k_map_pairs3(Header* h, const int32_t* nbr, const int64_t* m_out, int64_t cap,
                                                    const uint32_t* bbase, int32_t* off, int32_t* pairs,
                                                    int64_t pair_cap) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t nblk = gridDim.x;
    if (blockIdx.x == 0) {
        for (int k = threadIdx.x; k <= 27; k += blockDim.x) off[k] = (int32_t)bbase[k * nblk];
    }
    const int64_t m = count_or_cap(m_out, cap);
    const int64_t j = (int64_t)blockIdx.x * kNbrVox + lane;
    const bool valid = j < m;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int q = 0; q < kNbrProbes; ++q) {
        const int k = wave + kNbrWaves * q;
        if (k >= 27) break;
        const int32_t e = valid ? nbr[j * 27 + k] : 0;
        const uint64_t bal = __ballot(e != 0);
        if (e != 0) {
            const int64_t pos = (int64_t)bbase[k * nblk + blockIdx.x] + __popcll(bal & lt);
            if (pos < pair_cap) {
                pairs[2 * pos] = e - 1;
                pairs[2 * pos + 1] = (int32_t)j;
            } else {
                raise_flag(h, kFlagCapacity);
            }
        }
    }
}

// The neighbour table alone, from half the probes: offset k of voxel j holds i
// exactly when offset 26 - k of voxel i holds j (the map of a set onto itself
// is symmetric), so only the 13 offsets below the centre are probed.  A block
// writes entries 0..13 of its 64 rows (the centre is the voxel itself) through
// an LDS tile, and every pair it finds also into entry 26 - k of the partner's
// row; entries 14..26 start at zero (the table build or the voxelization's
// inserts clear them), and the two kinds of write never touch the same entry.
constexpr int kSymWaves = 7;  // wave w probes k = w and w + 7 (< 13)
__global__ __launch_bounds__(64 * kSymWaves) void k_map_nbr3_sym(Table fine, const int32_t* coords,
                                                                 const int64_t* m_out, int64_t cap, int32_t* nbr) {
    constexpr int KL = 14;  // entries 0..13 of a row: the probed offsets and the centre
    __shared__ int32_t tile[kNbrVox * KL];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t m = count_or_cap(m_out, cap);
    const int64_t j = (int64_t)blockIdx.x * kNbrVox + lane;
    const bool valid = j < m;
    int c[4] = {0, 0, 0, 0};
    if (valid) {
#pragma unroll
        for (int d = 0; d < 4; ++d) c[d] = coords[4 * j + d];
    }
    uint64_t key[2];
    bool act[2];
    int32_t res[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int k = wave + kSymWaves * q;
        int dx, dy, dz;
        offset_delta<3>(k, dx, dy, dz);
        act[q] = valid && k < 13;
        key[q] = pack_key(c[0], c[1] + dx, c[2] + dy, c[3] + dz);
    }
    table_find_n<2>(fine, key, act, res);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int k = wave + kSymWaves * q;
        if (k >= 13) break;
        const int32_t i = res[q];
        const bool present = valid && i >= 0;
        tile[lane * KL + k] = present ? i + 1 : 0;
        if (present) nbr[(int64_t)i * 27 + (26 - k)] = (int32_t)j + 1;
    }
    if (wave == 0) tile[lane * KL + 13] = valid ? (int32_t)j + 1 : 0;
    __syncthreads();
    const int64_t j0 = (int64_t)blockIdx.x * kNbrVox;
    const int rows = m - j0 < kNbrVox ? (int)(m - j0) : kNbrVox;
    for (int e = threadIdx.x; e < rows * KL; e += blockDim.x) {
        const int r = e / KL, k = e - r * KL;
        nbr[(j0 + r) * 27 + k] = tile[e];
    }
}

// per-(offset, block) pair counts of a finished neighbour table (the pairs
// pass's layout: offset-major, one count per block of kNbrVox rows)
__global__ __launch_bounds__(64 * kNbrWaves) void k_map_count3(const int32_t* nbr, const int64_t* m_out, int64_t cap,
                                                               uint32_t* bcnt) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t m = count_or_cap(m_out, cap);
    const int64_t j = (int64_t)blockIdx.x * kNbrVox + lane;
    const bool valid = j < m;
#pragma unroll
    for (int q = 0; q < kNbrProbes; ++q) {
        const int k = wave + kNbrWaves * q;
        if (k >= 27) break;
        const bool present = valid && nbr[j * 27 + k] != 0;
        const uint64_t bal = __ballot(present);
        if (lane == 0) bcnt[k * gridDim.x + blockIdx.x] = (uint32_t)__popcll(bal);
    }
}

void launch_kernel_map_nbr(hipStream_t s, const KmapWs& w, const int32_t* coords, const int64_t* m_dev,
                           int64_t m_cap, int32_t* nbr) {
    const int64_t mc = m_cap > 0 ? m_cap : 1;
    k_map_nbr3_sym<<<blocks_for(mc, kNbrVox), 64 * kSymWaves, 0, s>>>(w.fine, coords, m_dev, mc, nbr);
}

void launch_kernel_map(hipStream_t s, const KmapWs& w, bool build_fine, const int32_t* in_coords,
                       const int64_t* m_in_dev, int64_t m_cap, int K, int stride, int32_t* out_coords,
                       int64_t* m_out_dev, int32_t* off, int32_t* pairs, int64_t pair_cap, bool clear_header) {
    const int64_t mc = m_cap > 0 ? m_cap : 1;
    const unsigned nblk = blocks_for(mc, kMapThreads);
    const int K3 = K * K * K;
    const bool fine = build_fine && K == 3;  // a K = 2 map needs no table of its inputs
    if (fine) {
        // a submanifold map's table build also hands the output count (= the
        // input count) on
        launch_clear(s, w.h, w.fine, clear_header);
        // a submanifold map clears entries 14..26 of its neighbour rows here
        // for the half-probe table
        launch_table_build(s, w.h, w.fine, in_coords, m_in_dev, m_cap, stride == 1 ? w.m_out : nullptr,
                           stride == 1 ? m_out_dev : nullptr, stride == 1 ? w.nbr : nullptr);
    } else if (clear_header && stride != 2) {
        launch_clear_header(s, w.h);
    }
    if (stride == 2) {
        // coarse table, status header (unless cleared above) and the coarse key
        // counter in one launch
        launch_clear(s, w.h, w.coarse, clear_header && !fine, w.m_out + 1);
        // at most kRsMaxRecords insert blocks: every histogram block reduces their records
        unsigned nins = blocks_for(mc, kAppendThreads);
        if (nins > kRsMaxRecords) nins = kRsMaxRecords;
        k_map_coarse_insert<<<nins, kAppendThreads, 0, s>>>(w.h, w.coarse, w.rs, (int64_t)radix_zero_words(mc),
                                                            w.m_out + 1, in_coords, m_in_dev, mc);
        launch_radix_sort(s, w.rs, w.h, w.m_out + 1, mc, nins);
        k_map_coarse_rank<<<nblk, kMapThreads, 0, s>>>(w.rs, w.coarse, w.m_out + 1, mc, out_coords, w.m_out,
                                                       m_out_dev);
    }
    if (K == 3) {
        const unsigned nb3 = blocks_for(mc, kNbrVox);
        if (stride == 2) {
            k_map_nbr3<true><<<nb3, 64 * kNbrWaves, 0, s>>>(w.fine, out_coords, w.m_out, mc, w.nbr, w.bcnt);
        } else {
            if (fine && w.nbr) {
                // the table from half the probes, then the per-block counts from it
                k_map_nbr3_sym<<<nb3, 64 * kSymWaves, 0, s>>>(w.fine, in_coords, w.m_out, mc, w.nbr);
                k_map_count3<<<nb3, 64 * kNbrWaves, 0, s>>>(w.nbr, w.m_out, mc, w.bcnt);
            } else {
                k_map_same_count<<<1, 1, 0, s>>>(m_in_dev, m_cap, w.m_out, m_out_dev);
                k_map_nbr3<false><<<nb3, 64 * kNbrWaves, 0, s>>>(w.fine, in_coords, w.m_out, mc, w.nbr, w.bcnt);
            }
        }
        launch_exclusive_scan(s, (const int32_t*)w.bcnt, (int32_t*)w.bbase, nullptr, (int64_t)27 * nb3, w.scan_tmp);
        k_map_pairs3<<<nb3, 64 * kNbrWaves, 0, s>>>(w.h, w.nbr, w.m_out, mc, w.bbase, off, pairs, pair_cap);
    } else {
        k_s2_count<<<nblk, kMapThreads, 0, s>>>(in_coords, m_in_dev, mc, w.bcnt);
        launch_exclusive_scan(s, (const int32_t*)w.bcnt, (int32_t*)w.bbase, nullptr, (int64_t)K3 * nblk, w.scan_tmp);
        k_s2_write<<<nblk, kMapThreads, 0, s>>>(w.h, w.coarse, in_coords, m_in_dev, mc, w.bbase, off, pairs, pair_cap);
    }
}

}  // namespace spv
