// spv_internal.hpp -- host-side launchers shared between the translation units of
// libspv.so.  Every launcher only enqueues kernels on `s`; none synchronizes.
#pragma once

#include "spv_common.hpp"

namespace spv {

// --- block-level helpers (device) -------------------------------------------
// exclusive prefix sum of v over the block (blockDim.x threads, multiple of 64);
// lds must hold blockDim.x/64 + 1 ints.  *total receives the block sum.
__device__ inline int block_exclusive_scan(int v, int* lds, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    if (lane == 63) lds[wave] = x;
    __syncthreads();
    if (wave == 0) {
        // the wave totals scanned by wave 0
        const int t = lane < nw ? lds[lane] : 0;
        int y = t;
        for (int d = 1; d < nw; d <<= 1) {
            const int u = __shfl_up(y, d, 64);
            if (lane >= d) y += u;
        }
        if (lane < nw) lds[lane] = y - t;
        if (lane == nw - 1) lds[nw] = y;
    }
    __syncthreads();
    int r = lds[wave] + x - v;
    *total = lds[nw];
    __syncthreads();
    return r;
}

// Threads per block of the kernels that append new keys to a list.
constexpr int kAppendThreads = 1024;

// Appends `key` for every thread with `take` set to list[*counter ...] with one
// counter atomic per block (order inside the list is unspecified).  Every thread
// of the block must call it.
__device__ inline void block_append(bool take, uint64_t key, uint64_t* list, int64_t* counter) {
    __shared__ int lds[kAppendThreads / 64 + 1];
    __shared__ unsigned long long base;
    int tot;
    const int r = block_exclusive_scan(take ? 1 : 0, lds, &tot);
    if (threadIdx.x == 0) base = tot ? atomicAdd((unsigned long long*)counter, (unsigned long long)tot) : 0ull;
    __syncthreads();
    if (take) list[base + (unsigned long long)r] = key;
}

// The block's per-field minimum / maximum (4 + 4 ints) into rec[0..8).  Every
// thread of the block must call it; neutral values come from threads without keys.
__device__ inline void block_minmax_record(int (&mn)[4], int (&mx)[4], int32_t* rec) {
    __shared__ int32_t red[8];
    if (threadIdx.x < 8) red[threadIdx.x] = threadIdx.x < 4 ? 0x7fffffff : (int32_t)0x80000000;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            mn[d] = min(mn[d], __shfl_xor(mn[d], o, 64));
            mx[d] = max(mx[d], __shfl_xor(mx[d], o, 64));
        }
    }
    __syncthreads();
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            atomicMin(&red[d], mn[d]);  // LDS
            atomicMax(&red[4 + d], mx[d]);
        }
    }
    __syncthreads();
    if (threadIdx.x < 8) rec[threadIdx.x] = red[threadIdx.x];
}

// --- hash tables (hash_sort_scan.hip) ----------------------------------------
// Clear the header (status, counters, key statistics) and a table's key slots.
// empties the table; clear_header also clears the status header; zero64 (when
// given) is set to 0 in the same launch
void launch_clear(hipStream_t s, Header* h, Table t, bool clear_header, int64_t* zero64 = nullptr);
void launch_clear_header(hipStream_t s, Header* h);
// Insert coords[0..count) (count = *count_dev or cap) with value = row index;
// raises kFlagDuplicate on a repeated coordinate, kFlagRange on a coordinate
// outside the key range.
// count_out / count_out2 (when given) receive the clamped count in the same launch
// nbr_upper (optional): entries 14..26 of each inserted row's neighbour-table row -> 0
void launch_table_build(hipStream_t s, Header* h, Table t, const int32_t* coords, const int64_t* count_dev,
                        int64_t cap, int64_t* count_out = nullptr, int64_t* count_out2 = nullptr,
                        int32_t* nbr_upper = nullptr);
void launch_table_lookup(hipStream_t s, Table t, const int32_t* q, int64_t nq, int32_t* idx);

// --- statistics of the keys being sorted (radix.hip) -------------------------
// The per-field minima and maxima of the keys; a key is sorted in compacted form
// (minimum subtracted, fields packed into the fewest bits).
struct SortStats {
    int32_t fmin[4];    // per-field minimum of the keys being sorted (b, x, y, z)
    int32_t fmax[4];
    uint32_t fbits[4];  // bit width of each compacted field
    uint32_t sort_bits; // significant bits of the compacted key (64 when any item is invalid)
    uint32_t n_invalid; // items with an invalid key
    uint32_t invalid_kinds;  // bit 0: a non-finite item, bit 1: an item out of the key range
    uint32_t msd;       // 1 when the bucket sort ordered the keys (result in ka / va)
};
// --- radix sort of (key, payload) pairs (radix.hip) ---------------------------
// The producer writes raw packed keys (kEmpty: invalid item) to ka[0..count) and,
// per block of kRsProducerBlock items, a record of kRsRecWords ints: per-field
// minima (4) and maxima (4) of its valid keys, then its non-finite and
// out-of-range item counts.  It also zeroes zero[0..radix_zero_words).  After
// launch_radix_sort the compacted keys, ascending, and the items' original
// indices sit in rs_keys / rs_vals (which of the two buffers depends on the
// path taken and the number of passes, both known on the device only).
constexpr int kRsThreads = 512;
constexpr int kRsItems = 4;
constexpr int kRsTile = kRsThreads * kRsItems;  // keys per tile
constexpr int kRsBits = 8;                      // digit width
constexpr int kRsBins = 1 << kRsBits;
constexpr int kRsPasses = (64 + kRsBits - 1) / kRsBits;  // digits of a 64-bit key
constexpr int kRsRecWords = 12;
constexpr int kRsProducerBlock = 256;
constexpr unsigned kRsMaxRecords = 1024;  // producer records (blocks) at most
struct RadixWs {
    uint64_t* ka;
    uint64_t* kb;
    uint32_t* va;
    uint32_t* vb;
    int32_t* rec;       // producer records
    SortStats* st;
    int64_t ntiles;     // tiles of the capacity (a pass grid)
    uint32_t* zero;     // the region the producer zeroes (radix_zero_words):
    uint32_t* ghist;    //   [kRsPasses][kRsBins] digit counts over all keys
    uint32_t* ctr;      //   [64] tile counters (0 .. kRsPasses-1 the passes, 8.. for the consumers)
    uint32_t* fhist;    //   [4096] the bucket sort's item counts per fine bin (top 12 key bits)
    uint32_t* fcur;     //   [4096] ... and the items of each fine bin claimed so far
    uint32_t* sb;       // the bucket sort's bucket table: starts, first fine bins, count
    uint64_t* status;   // [kRsPasses][ntiles][kRsBins] look-back words, then [ntiles] for a consumer's scan:
                        // the histogram kernel clears pass 0's and the consumer's, pass p clears pass p+1's
};
size_t radix_tiles(int64_t cap);
size_t radix_zero_words(int64_t cap);
void plan_radix_ws(Arena& a, RadixWs& w, int64_t cap);
// count_dev: device item count (nullptr: cap); nrec: producer records
void launch_radix_sort(hipStream_t s, const RadixWs& w, Header* h, const int64_t* count_dev, int64_t cap,
                       uint32_t nrec);
__host__ __device__ inline int rs_passes(const SortStats& st) {
    const int p = (int)((st.sort_bits + kRsBits - 1) / kRsBits);
    return p > 0 ? p : 1;
}
// the look-back words a consumer of the sort may use for a scan of its own over the tiles
__host__ __device__ inline uint64_t* rs_consumer_status(const RadixWs& w) { return w.status + (size_t)kRsPasses * kRsBins * w.ntiles; }
__device__ inline const uint64_t* rs_keys(const RadixWs& w, const SortStats& st) {
    return (!st.msd && (rs_passes(st) & 1)) ? w.kb : w.ka;
}
__device__ inline const uint32_t* rs_vals(const RadixWs& w, const SortStats& st) {
    return (!st.msd && (rs_passes(st) & 1)) ? w.vb : w.va;
}
// the packed key of a compacted key
__device__ inline uint64_t rs_expand(uint64_t ck, const SortStats& st) {
    const uint32_t bz = st.fbits[3], by = st.fbits[2], bx = st.fbits[1];
    const int z = (int)(ck & ((1ull << bz) - 1)) + st.fmin[3];
    ck >>= bz;
    const int y = (int)(ck & ((1ull << by) - 1)) + st.fmin[2];
    ck >>= by;
    const int x = (int)(ck & ((1ull << bx) - 1)) + st.fmin[1];
    ck >>= bx;
    return pack_key((int)ck + st.fmin[0], x, y, z);
}

// --- prefix sums with a device-side count (hash_sort_scan.hip) ----------------
// out[i] = sum_{j<i} in[j] for i in [0, count]; out must hold cap + 1 ints;
// tmp must hold scan_tmp_entries(cap) ints.
size_t scan_tmp_entries(int64_t cap);
void launch_exclusive_scan(hipStream_t s, const int32_t* in, int32_t* out, const int64_t* count_dev, int64_t cap,
                           int32_t* tmp);
// single-block exclusive scan of a host-sized array (n small), out[n] = total
void launch_exclusive_scan_small(hipStream_t s, const uint32_t* in, uint32_t* out, int64_t n);

// --- voxelize (voxelize.hip) ---------------------------------------------------
struct PackJob;
struct VoxelizeWs {
    Header* h;          // assigned by the caller (workspace offset 0)
    Table table;
    RadixWs rs;         // the points sorted by key
    int32_t* seg;       // [n + 1] CSR offsets of the points of each voxel
    int32_t* fill;      // [n]
    int32_t* plist;     // [n] point ids grouped by voxel
    int32_t* longv;     // [n] voxels whose mean takes a whole workgroup (count in h->aux[0])
    int32_t* scan_tmp;  // [scan_tmp_entries(n)]
    int32_t* nbr_upper = nullptr;  // optional [m][27] neighbour table: entries 14..26 of each voxel's row
                                   // are zeroed where the voxel is entered into the table
};
void plan_voxelize_ws(Arena& a, VoxelizeWs& w, int64_t n);
// coords/counts/pt2vox and (if feat) vfeat; m into h->m and *m_dev.  The first
// launch clears the status header and the table and also runs the weight
// packings `jobs` (a block call packs its layers' weights there).
void launch_voxelize(hipStream_t s, const VoxelizeWs& w, const float* xyz, const int32_t* batch, int64_t n,
                     float voxel_size, const void* feat, int32_t C, int dt, int32_t* coords, void* vfeat,
                     int32_t* counts, int32_t* pt2vox, int64_t* m_dev, const PackJob* jobs = nullptr,
                     int njobs = 0);
// scatter-mean onto the given voxel set coords[min(*m_dev, m_cap)] (value = row);
// points whose voxel is not in the set get pt2vox -1; ws planned for max(n, m_cap)
void launch_voxelize_onto(hipStream_t s, const VoxelizeWs& w, const int32_t* coords, const int64_t* m_dev,
                          int64_t m_cap, const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                          const void* feat, int32_t C, int dt, void* vfeat, int32_t* counts, int32_t* pt2vox);

// --- kernel map (kmap.hip) -----------------------------------------------------
struct KmapWs {
    Header* h;          // assigned by the caller
    Table fine;         // table of the input coords (assigned by the caller when shared)
    Table coarse;       // stride 2: table of the output coords
    RadixWs rs;         // stride 2: coarse key sort
    uint32_t* bcnt;     // [K3 * nblk] per-block per-offset counts (k-major)
    uint32_t* bbase;    // [K3 * nblk + 1]
    int32_t* scan_tmp;  // [scan_tmp_entries(K3 * nblk)]
    int64_t* m_out;     // device count of outputs
    int32_t* nbr;       // K = 3: [m_cap][27] neighbour table i + 1 (0 = none)
};
// own_nbr: reserve the 3x3x3 neighbour table here (otherwise the caller assigns w.nbr)
void plan_kmap_ws(Arena& a, KmapWs& w, int64_t m_cap, int K, int stride, bool own_fine_table, bool own_nbr);
// build_fine: clear + insert the input coords into w.fine first (otherwise the
// table must already map every input coordinate to its row)
// clear_header: the map's first launch also clears the status header
void launch_kernel_map(hipStream_t s, const KmapWs& w, bool build_fine, const int32_t* in_coords,
                       const int64_t* m_in_dev, int64_t m_cap, int K, int stride, int32_t* out_coords,
                       int64_t* m_out_dev, int32_t* off, int32_t* pairs, int64_t pair_cap, bool clear_header = false);
// submanifold 3x3x3 neighbour table only (pass 1, no pairs): nbr[j][k] = i + 1,
// 0 where offset k of voxel j holds no voxel; w.fine must map every coordinate,
// and entries 14..26 of rows 0 .. m-1 must be zero already (the table build or
// the voxelization's inserts clear them): offsets below the centre are probed,
// and each pair found fills both rows (offset k of j, offset 26 - k of i)
void launch_kernel_map_nbr(hipStream_t s, const KmapWs& w, const int32_t* coords, const int64_t* m_dev,
                           int64_t m_cap, int32_t* nbr);
// entries 14..26 of neighbour-table row v -> 0
__device__ inline void clear_nbr_upper(int32_t* nbr, int64_t v) {
#pragma unroll
    for (int k = 14; k < 27; ++k) nbr[v * 27 + k] = 0;
}

// --- sparse conv (conv.hip) ----------------------------------------------------
// Two MFMA kernels share one plan.
//  * 3x3x3 maps (K3 = 27): output-stationary blocks of 16 rows with register
//    accumulators; the plan builds a dense neighbour table nbr[j][k] = i + 1
//    (0 = no pair) from the kernel map.
//  * other maps (K3 = 8) and wide shapes: output rows in tiles of `tile_rows`
//    with an LDS accumulator; the plan records, per offset k and tile t, the
//    first pair of offset k whose output row lies in tile t or later (the
//    pairs of one offset are sorted by output row, so those of (tile, offset)
//    form the range [bnd[k][t], bnd[k][t+1])).
struct ConvPlan {
    int64_t m_cap;      // output row capacity
    int K3;
    int use_union;      // 1: neighbour-table kernel, 0: tile kernel (or vector ALU)
    int tile_rows;      // output rows per tile (power of two)
    int64_t ntile_cap;  // ceil(m_cap / tile_rows)
    int32_t* bnd;       // [K3][ntile_cap + 1]
    int32_t* nbr;       // [m_cap][K3] when use_union
    const int64_t* m_out_dev;
    Header* h;          // status word (unsorted or out-of-range pairs)
    // residual input [m][Cout] of the storage type (nullptr = none), added after
    // scale and shift and before the activation; it must not alias the output
    const void* res = nullptr;
    // W strides in elements for the vector-ALU kernel, which reads W itself
    // (0: a dense [K3][Cin][Cout] tensor)
    int w_ldc = 0;
    int64_t w_ldk = 0;
    int w_ldcol = 0;
};
// The kernel a conv runs on, decided on the host from the shape and the sizes
// (kConvUnion needs every neighbour-table and input offset within 32 bits; a
// transposed map with fewer inputs than outputs -- sparse_transposed -- goes to
// the tile kernel, which visits pairs only).
enum ConvKernel { kConvUnion = 0, kConvTile = 1, kConvValu = 2 };
int conv_kernel_choice(int K3, int Cin, int Cout, int dt, int64_t m_out_cap, int64_t in_rows, int64_t pair_bound,
                       bool sparse_transposed);
// in_rows: rows of the conv's input (the plan's kernel choice depends on it)
void plan_conv_ws(Arena& a, ConvPlan& p, int64_t m_out_cap, int K3, int Cin, int Cout, int dt, int64_t in_rows,
                  bool sparse_transposed = false);
struct PackJob;
// plans the conv on a kernel map (neighbour table or tile bounds), runs the
// weight packing pk (total = 0: none) in one of its launches and, with
// clear_header, first clears the status header the plan may raise flags in
void launch_conv_plan(hipStream_t s, const ConvPlan& p, const int32_t* off, const int32_t* pairs, int K3,
                      int transposed, int64_t pair_bound, int64_t in_rows, const PackJob& pk,
                      bool clear_header = false);
bool conv_mfma_supported(int Cin, int Cout, int dt);
void* plan_wpack_ws(Arena& a, int K3, int Cin, int Cout);
// One weight packing into MFMA operand fragments, as a job for the block prologue
// (total = 0: nothing to pack, the layer runs on a kernel that reads W itself).
struct PackJob {
    const uint16_t* W;  // W[k][c][col] at W[k * ldk + c * ldc + col]
    uint4* wpack;
    int K3, Cin, Cout, KCH, NB;
    int64_t total;      // fragments * 64 lanes
    int ldc;            // elements between input channels (Cout when dense)
    int64_t ldk;        // elements between offsets (Cin * Cout when dense)
    int ldcol = 1;      // elements between output channels (1 when dense)
};
// fragment t of the packing (t = ((k * KCH + kc) * NB + nb) * 64 + lane)
// W[k][c][col] sits at W[k * ldk + c * ldc + col * ldcol] (ldc = Cout, ldcol = 1,
// ldk = Cin * Cout for a dense [K3][Cin][Cout] tensor; larger ldc / ldk for a
// channel slice of a wider one; ldc = 1, ldcol = the stored row length to read
// every W[k] transposed)
__device__ inline uint4 pack_fragment(const uint16_t* W, int Cin, int Cout, int ldc, int ldcol, int64_t ldk, int KCH,
                                     int NB, int64_t t) {
    const int lane = (int)(t & 63);
    int64_t f = t >> 6;
    const int nb = (int)(f % NB);
    f /= NB;
    const int kc = (int)(f % KCH);
    const int k = (int)(f / KCH);
    const int col = nb * 16 + (lane & 15);
    const int ci0 = kc * 32 + 8 * (lane >> 4);
    uint32_t w[4];
    for (int e = 0; e < 4; ++e) {
        uint32_t lo = 0, hi = 0;
        const int c0 = ci0 + 2 * e, c1 = ci0 + 2 * e + 1;
        // zeros past the last input channel and past the last output column
        if (c0 < Cin && col < Cout) lo = W[(int64_t)k * ldk + (int64_t)c0 * ldc + (int64_t)col * ldcol];
        if (c1 < Cin && col < Cout) hi = W[(int64_t)k * ldk + (int64_t)c1 * ldc + (int64_t)col * ldcol];
        w[e] = lo | (hi << 16);
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// a weight packing run alongside another kernel's work (grid-stride)
__device__ inline void pack_job_run(const PackJob& q) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < q.total; t += (int64_t)gridDim.x * blockDim.x)
        q.wpack[t] = pack_fragment(q.W, q.Cin, q.Cout, q.ldc, q.ldcol, q.ldk, q.KCH, q.NB, t);
}

// ldc / ldk <= 0: W is a dense [K3][Cin][Cout] tensor; otherwise the leading
// Cin x Cout block of each offset of a wider tensor (a channel slice)
// W[26 - k]^T for every offset k of a 3x3x3 W [27][Cin][Cout] (a [27][Cout][Cin] packing)
PackJob conv_pack_job_mirrored(const void* W, void* wpack, int Cin, int Cout, int dt);
PackJob conv_pack_job(int K3, const void* W, void* wpack, int Cin, int Cout, int dt, int ldc = 0, int64_t ldk = 0,
                      int ldcol = 0);
// the weight packing q as a launch of its own
void launch_pack_job(hipStream_t s, const PackJob& q);

// --- pointwise linear layer (linear.hip) -----------------------------------------
struct LinearArgs {
    const void* in;          // [m][Cin]
    const int64_t* m_dev;    // device row count (nullptr = m_cap)
    int64_t m_cap;
    int Cin, Cout, dt;
    const void* W;           // W[ci][co] at W[ci * ldw + co]
    int ldw;
    const float* scale;      // [Cout] or nullptr
    const float* shift;      // [Cout] or nullptr
    int relu;
    const void* res;         // [m][Cout] or nullptr
    int res_after;           // 1: res added after the activation
    void* out;               // [m][Cout]
    int wt = 0;              // 1: W read transposed, W[ci][co] at W[co * ldw + ci]
};
bool linear_mfma_supported(int Cin, int Cout, int dt);
void* plan_linear_ws(Arena& a, int Cin, int Cout);
// packs W into wpack (MFMA path) and runs the layer
// prepacked: wpack already holds W's fragments (spv_pack_weights), no packing launch
void launch_linear(hipStream_t s, const LinearArgs& a, void* wpack, bool prepacked = false);

// --- transposed k=2 s=2 conv on a child table (conv_up.hip) -----------------------
struct UpArgs {
    const int32_t* children;  // [m_cap][8]: fine row + 1 of the child at offset k, 0 = none
    const int64_t* m_dev;     // coarse row count (nullptr = m_cap)
    int64_t m_cap;
    const void* in;           // [m_cap][Cin] coarse rows
    int Cin, Cout, dt;
    const float* scale;
    const float* shift;
    int relu;
    const void* res;          // [out_rows][Cout] or nullptr
    void* out;                // [out_rows][Cout] fine rows
    int64_t out_rows;
};
bool up_supported(int Cin, int Cout, int dt);
void launch_conv_up(hipStream_t s, const UpArgs& a, const void* wpack);
// the neighbour table nbr[j][k] = i + 1 of a map's pairs (i, j) (rows by output),
// cleared first; unsorted or repeated pairs raise the header's flags
void launch_nbr_table(hipStream_t s, const int32_t* off, const int32_t* pairs, int K3, int64_t pair_bound,
                      const int64_t* m_out_dev, int64_t m_cap, int64_t in_rows, int32_t* nbr, Header* h);

// --- backward passes (backward.hip) --------------------------------------------
struct WgradArgs {
    const void* x;           // [x_rows][Cin] conv input
    int64_t x_rows;
    int Cin;
    const void* dy;          // [dy_rows][Cout] gradient of the conv output
    int64_t dy_rows;
    int Cout;
    const int32_t* off;      // [K3 + 1]
    const int32_t* pairs;    // [pair_bound][2]
    int64_t pair_bound;
    int K3, transposed, dt;
    int slot_k3 = 0;         // K3 the partial buffer was sized for (0: K3)
};
bool wgrad_supported(int Cin, int Cout);
void* plan_wgrad_ws(Arena& a, int K3, int Cin, int Cout);
// dW [K3][Cin][Cout] fp32 via per-slice partials in `partial`
void launch_wgrad(hipStream_t s, const WgradArgs& a, float* partial, float* dW);
void launch_voxelize_backward(hipStream_t s, const void* dv, int C, const int32_t* counts, const int32_t* pt2vox,
                              int64_t n, int64_t m, void* dfeat, int dt);
// backward of the conv / linear epilogue (scale, shift, ReLU, residual)
struct EpiBwdArgs {
    const void* dy;          // [m][C] gradient of the epilogue's output
    const void* a;           // [m][C] the raw product the epilogue was applied to
    const float* scale;      // [C] or nullptr (1)
    const float* shift;      // [C] or nullptr (0)
    int relu;
    const void* res;         // [m][C] or nullptr
    int res_after;
    int64_t m;
    int C, dt;
    void* da;                // [m][C] or nullptr
    void* dres;              // [m][C] or nullptr
    float* dscale;           // [C] or nullptr
    float* dshift;           // [C] or nullptr
};
// fp64 entries of the per-workgroup sums
size_t epilogue_backward_part_entries(int64_t m, int C);
void launch_epilogue_backward(hipStream_t s, const EpiBwdArgs& a, double* part);

// devoxelization backward: the counting sort of the (point, corner) entries by
// voxel; entries hold 8 * point + corner, rec the (entry, coefficient) pairs of
// every voxel in ascending entry order
struct DvbWs {
    Header* h;
    int32_t* cnt;   // [m + 1] entries per voxel
    int32_t* off;   // [m + 1] exclusive scan of cnt
    int32_t* tmp;   // [scan_tmp_entries(m)]
    int32_t* slot;  // [8n] each entry's slot in its voxel's range (-1: corner absent)
    int32_t* ent;   // [8n] entry numbers in fill order
    float* coef;    // [8n] their coefficients
    int32_t* vox;   // [8n] their voxels
    int2* rec;      // [8n] (entry, coefficient bits), sorted within each voxel
    int2* chk;      // [8n] the same, sorted within chunks of a long voxel's range
    int32_t* longv; // [m + 1] the voxels gathered by a workgroup each (count in h->aux[0])
};
DvbWs plan_devox_backward_ws(Arena& a, int64_t n, int64_t m);
void launch_devoxelize_backward(hipStream_t s, const DvbWs& w, const int32_t* cidx, const float* cw, const void* dout,
                                int64_t n, int C, float* dv, int64_t m, int dt);

// weight packings a block call runs inside its voxelization's first launch
constexpr int kMaxPackJobs = 3;
// the convolution itself (one kernel); wpack must have been packed from W
void launch_conv_run(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, const int32_t* pairs,
                     int64_t pair_bound, int transposed, const void* W, const void* wpack, const float* scale,
                     const float* shift, int relu, void* out, int Cout, int dt);

// --- devoxelize (devox.hip) ----------------------------------------------------
struct DevoxArgs {
    Table table;
    int stride_log2;
    const float* xyz;
    const int32_t* batch;
    int64_t n;
    float voxel_size;
    int mode;
    const void* vfeat;
    int C;
    const void* pfeat;
    int Cp;
    const void* Wp;
    const float* scale_p;
    const float* shift_p;
    int relu_p;
    void* out;
    int dt;
    int32_t* corner_idx;
    float* corner_w;
    Header* h;
    // optional, when the grid is the points' own voxelization at stride 1:
    // each point's voxel (pt2vox), the grid's coordinates and its 3x3x3
    // neighbour table (nbr[j][k] = i + 1); corners are then read from the
    // table instead of probed
    const int32_t* pt2vox = nullptr;
    const int32_t* grid_coords = nullptr;
    const int32_t* nbr = nullptr;
    int64_t nbr_rows = 0;  // rows of nbr / grid_coords: a pt2vox entry outside [0, nbr_rows) has no corners
    const int64_t* nbr_m_dev = nullptr;  // live row count of the grid (bounds pt2vox entries further when given)
};
bool devox_mfma_supported(int C, int Cp, int dt);
void* plan_devox_ws(Arena& a, int C, int Cp);
// wp_packed: the point-MLP weight is already in wpack (a block prologue packed it)
void launch_devox(hipStream_t s, const DevoxArgs& a, void* wpack, int32_t* cidx_tmp, float* cw_tmp,
                  bool wp_packed = false);
PackJob devox_pack_job(const DevoxArgs& a, void* wpack);

}  // namespace spv
