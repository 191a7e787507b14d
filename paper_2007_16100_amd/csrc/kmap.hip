// kmap.hip -- kernel-map construction on the voxel hash (Sec. 3.2: the active
// synapses between input and output voxels; Sec. 3.3 "Feature Aggregation":
// built with the same GPU hash table as the voxelization).
//
// Outputs: CSR by offset k -- off[K^3+1] and pairs (in, out), each offset's
// pairs sorted by out.  Two passes over the outputs, 256 per block:
//   pass 1: probe the K^3 neighbour coordinates of each output, keep a bit mask
//           of the present offsets, count per (offset, block) with wave ballots;
//   scan:   one exclusive scan over the offset-major (offset, block) counts gives
//           every block its write position inside every offset's segment;
//   pass 2: re-probe only the present offsets and write the pairs, the rank
//           inside the block coming from the same ballots -> deterministic,
//           already-sorted output without atomics.
// Stride 2: the output voxels are the distinct floor(c/2), deduplicated in a
// second hash table and radix-sorted into canonical order first.
#include "spv_internal.hpp"

namespace spv {

constexpr int kMapThreads = 256;

void plan_kmap_ws(Arena& a, KmapWs& w, int64_t m_cap, int K, int stride, bool own_fine_table) {
    int64_t mc = m_cap > 0 ? m_cap : 1;
    const int K3 = K * K * K;
    if (own_fine_table) {
        uint32_t S = table_capacity(mc);
        w.fine.keys = a.take<uint64_t>(S);
        w.fine.vals = a.take<int32_t>(S);
        w.fine.mask = S - 1;
    }
    if (stride == 2) {
        uint32_t S = table_capacity(mc);
        w.coarse.keys = a.take<uint64_t>(S);
        w.coarse.vals = a.take<int32_t>(S);
        w.coarse.mask = S - 1;
        plan_sort_ws(a, w.sort, mc);
    } else {
        w.coarse = Table{nullptr, nullptr, 0};
    }
    size_t nblk = blocks_for(mc, kMapThreads);
    w.mask = a.take<uint32_t>(mc);
    w.bcnt = a.take<uint32_t>(K3 * nblk);
    w.bbase = a.take<uint32_t>(K3 * nblk + 1);
    w.m_out = a.take<int64_t>(2);
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

__global__ void k_map_zero_i64(int64_t* p) { *p = 0; }

// stride 2: coarse keys into the coarse table; creators append to the key list
__global__ void k_map_coarse_insert(Header* h, Table coarse, uint64_t* ukeys, int64_t* cnt, const int32_t* in_coords,
                                    const int64_t* m_in_dev, int64_t cap) {
    int64_t m = count_or_cap(m_in_dev, cap);
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i >= m) return;
    const int32_t* c = in_coords + 4 * i;
    // floor(c / 2) via arithmetic shift
    uint64_t key = pack_key(c[0], c[1] >> 1, c[2] >> 1, c[3] >> 1);
    uint32_t slot;
    int r = table_insert(coarse, key, &slot);
    if (r > 0) {
        unsigned long long idx = atomicAdd((unsigned long long*)cnt, 1ull);
        ukeys[idx] = key;
    } else if (r < 0) {
        raise_flag(h, kFlagTableFull);
    }
}

__global__ void k_map_coarse_rank(SortBufs sb, Table coarse, const int64_t* cnt, int64_t cap, int32_t* out_coords,
                                  int64_t* m_out, int64_t* m_out_user) {
    int64_t m = count_or_cap(cnt, cap);
    int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (r == 0) {
        m_out[0] = m;
        if (m_out_user) *m_out_user = m;
    }
    if (r >= m) return;
    uint64_t key = sorted_key(sb, r);
    int64_t slot = table_slot(coarse, key);
    if (slot >= 0) coarse.vals[slot] = (int32_t)r;
    out_coords[4 * r + 0] = key_b(key);
    out_coords[4 * r + 1] = key_x(key);
    out_coords[4 * r + 2] = key_y(key);
    out_coords[4 * r + 3] = key_z(key);
}

// pass 1: offset masks + per-(offset, block) counts
template <int K, int S>
__global__ __launch_bounds__(kMapThreads) void k_map_mask(Table fine, const int32_t* out_coords, const int64_t* m_out,
                                                          int64_t cap, uint32_t* mask, uint32_t* bcnt) {
    constexpr int K3 = K * K * K;
    __shared__ uint32_t cnt[K3];
    for (int k = threadIdx.x; k < K3; k += blockDim.x) cnt[k] = 0;
    __syncthreads();
    int64_t m = count_or_cap(m_out, cap);
    int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    bool valid = j < m;
    uint32_t bits = 0;
    if (valid) {
        const int32_t* c = out_coords + 4 * j;
#pragma unroll
        for (int k = 0; k < K3; ++k) {
            int dx, dy, dz;
            offset_delta<K>(k, dx, dy, dz);
            if (K == 3 && k == 13) {
                bits |= 1u << k;  // an output of a submanifold map is its own centre neighbour
                continue;
            }
            int32_t i = table_find(fine, pack_key(c[0], S * c[1] + dx, S * c[2] + dy, S * c[3] + dz));
            if (i >= 0) bits |= 1u << k;
        }
        mask[j] = bits;
    }
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int k = 0; k < K3; ++k) {
        uint64_t bal = __ballot((bits >> k) & 1);
        if (lane == 0 && bal) atomicAdd(&cnt[k], (uint32_t)__popcll(bal));
    }
    __syncthreads();
    for (int k = threadIdx.x; k < K3; k += blockDim.x) bcnt[k * gridDim.x + blockIdx.x] = cnt[k];
}

// pass 2: pairs at their final, sorted positions
template <int K, int S>
__global__ __launch_bounds__(kMapThreads) void k_map_write(Header* h, Table fine, const int32_t* out_coords,
                                                           const int64_t* m_out, int64_t cap, const uint32_t* mask,
                                                           const uint32_t* bbase, int32_t* off, int32_t* pairs,
                                                           int64_t pair_cap) {
    constexpr int K3 = K * K * K;
    constexpr int NW = kMapThreads / 64;
    __shared__ uint32_t wtot[NW][K3];
    const uint32_t nblk = gridDim.x;
    if (blockIdx.x == 0) {
        for (int k = threadIdx.x; k <= K3; k += blockDim.x) off[k] = (int32_t)bbase[k * nblk];
    }
    int64_t m = count_or_cap(m_out, cap);
    int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    bool valid = j < m;
    uint32_t bits = valid ? mask[j] : 0u;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint32_t rank[K3];
#pragma unroll
    for (int k = 0; k < K3; ++k) {
        uint64_t bal = __ballot((bits >> k) & 1);
        rank[k] = (uint32_t)__popcll(bal & lt);
        if (lane == 0) wtot[wave][k] = (uint32_t)__popcll(bal);
    }
    __syncthreads();
    if (!valid) return;
    const int32_t* c = out_coords + 4 * j;
#pragma unroll
    for (int k = 0; k < K3; ++k) {
        if (!((bits >> k) & 1)) continue;
        uint32_t pos = bbase[k * nblk + blockIdx.x] + rank[k];
        for (int w = 0; w < wave; ++w) pos += wtot[w][k];
        int32_t i;
        if (K == 3 && k == 13) {
            i = (int32_t)j;
        } else {
            int dx, dy, dz;
            offset_delta<K>(k, dx, dy, dz);
            i = table_find(fine, pack_key(c[0], S * c[1] + dx, S * c[2] + dy, S * c[3] + dz));
        }
        if ((int64_t)pos < pair_cap) {
            pairs[2 * (int64_t)pos] = i;
            pairs[2 * (int64_t)pos + 1] = (int32_t)j;
        } else {
            raise_flag(h, kFlagCapacity);
        }
    }
}

void launch_kernel_map(hipStream_t s, const KmapWs& w, bool build_fine, const int32_t* in_coords,
                       const int64_t* m_in_dev, int64_t m_cap, int K, int stride, int32_t* out_coords,
                       int64_t* m_out_dev, int32_t* off, int32_t* pairs, int64_t pair_cap) {
    const int64_t mc = m_cap > 0 ? m_cap : 1;
    const unsigned nblk = blocks_for(mc, kMapThreads);
    const int K3 = K * K * K;
    if (build_fine) {
        launch_clear(s, w.h, w.fine, false);
        launch_table_build(s, w.h, w.fine, in_coords, m_in_dev, m_cap);
    }
    const int32_t* oc = in_coords;
    if (stride == 1) {
        k_map_same_count<<<1, 1, 0, s>>>(m_in_dev, m_cap, w.m_out, m_out_dev);
    } else {
        launch_clear(s, w.h, w.coarse, false);
        k_map_zero_i64<<<1, 1, 0, s>>>(w.m_out + 1);
        k_map_coarse_insert<<<nblk, kMapThreads, 0, s>>>(w.h, w.coarse, w.sort.a, w.m_out + 1, in_coords, m_in_dev,
                                                         m_cap);
        launch_sort_keys(s, w.sort, w.m_out + 1, mc);
        k_map_coarse_rank<<<nblk, kMapThreads, 0, s>>>(w.sort, w.coarse, w.m_out + 1, mc, out_coords, w.m_out,
                                                       m_out_dev);
        oc = out_coords;
    }
    if (K == 3) {
        k_map_mask<3, 1><<<nblk, kMapThreads, 0, s>>>(w.fine, oc, w.m_out, mc, w.mask, w.bcnt);
        launch_exclusive_scan_small(s, w.bcnt, w.bbase, (int64_t)K3 * nblk);
        k_map_write<3, 1><<<nblk, kMapThreads, 0, s>>>(w.h, w.fine, oc, w.m_out, mc, w.mask, w.bbase, off, pairs,
                                                       pair_cap);
    } else {
        k_map_mask<2, 2><<<nblk, kMapThreads, 0, s>>>(w.fine, oc, w.m_out, mc, w.mask, w.bcnt);
        launch_exclusive_scan_small(s, w.bcnt, w.bbase, (int64_t)K3 * nblk);
        k_map_write<2, 2><<<nblk, kMapThreads, 0, s>>>(w.h, w.fine, oc, w.m_out, mc, w.mask, w.bbase, off, pairs,
                                                       pair_cap);
    }
}

}  // namespace spv
