// conv.hip -- sparse convolution on a kernel map (Sec. 3.2 / 3.3):
//   out[j] = act(scale * sum_{(i, j, k)} in[i] @ W[k] + shift)
//
// Two matrix-core kernels, both deterministic (no atomics; every output element
// is summed in ascending offset order) and both writing every output row once:
//
// * k_conv_union (3x3x3 maps): a wave owns blocks of 16 output rows with all
//   output channels, accumulated in registers.  For each of the 27 offsets it
//   gathers the 16 rows' neighbours (zeros where a neighbour is absent) and
//   multiplies them by W[k] on v_mfma_f32_16x16x32_{bf16,f16}; blocks whose
//   rows have no neighbour at that offset skip it.  The weights of a phase of
//   offsets are staged per workgroup in LDS (global->LDS copies), and each
//   wave's gathers for the next offset are in flight while the current one is
//   multiplied.  The cost is MFMA work on absent neighbours: on a LiDAR sweep
//   the 16-row unions of present offsets are ~3x the pairs.  Widths C_in,
//   C_out in {32, 64, 96, 128, 256}; submanifold and strided 3x3x3 maps.
//
// * k_conv_tile (K = 2 maps, transposed maps -- where a 16-row union would be
//   mostly empty -- and the other widths): output rows in tiles of T with an
//   LDS fp32 accumulator; the pairs of each (tile, offset) are a contiguous
//   slice of the kernel map, multiplied 16 at a time and added into their
//   output rows.
//
// A vector-ALU tile kernel covers fp32 and shapes the MFMA kernels do not take.
#include "conv_common.hpp"

namespace spv {


// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------
static int conv_tile_rows(int Cin, int Cout, int dt);

// The boundary array is sized for the smallest tile (16 rows) and the neighbour
// table is reserved for every 3x3x3 plan, so the workspace size does not depend
// on the channel counts or the dtype.
void plan_conv_ws(Arena& a, ConvPlan& p, int64_t m_out_cap, int K3, int Cin, int Cout, int dt, int64_t in_rows,
                  bool sparse_transposed) {
    p.m_cap = m_out_cap > 0 ? m_out_cap : 1;
    p.K3 = K3;
    // decided once here: launch_conv_plan builds what this kernel reads
    // (neighbour table or tile bounds) and launch_conv_run runs it
    p.use_union = conv_kernel_choice(K3, Cin, Cout, dt, p.m_cap, in_rows, 0, sparse_transposed) == kConvUnion ? 1 : 0;
    p.tile_rows = conv_tile_rows(Cin, Cout, dt);
    p.ntile_cap = (p.m_cap + p.tile_rows - 1) / p.tile_rows;
    p.bnd = a.take<int32_t>((size_t)K3 * ((p.m_cap + kChunk - 1) / kChunk + 1));
    // reserved for every 3x3x3 plan, so that a workspace sized for one dtype / width serves all
    p.nbr = K3 == 27 ? a.take<int32_t>((size_t)p.m_cap * K3) : nullptr;
    p.h = nullptr;
    p.m_out_dev = nullptr;
}

// the offset k of pair p (off is non-decreasing)
__device__ inline int pair_offset(const int32_t* soff, int K3, int64_t p) {
    int k = 0;
    while (k + 1 < K3 && p >= soff[k + 1]) ++k;
    return k;
}

// tile of output row j; rows outside [0, m) are placed where they sort
// (negative rows before tile 0's rows, rows >= m after the last tile)
__device__ inline int64_t tile_of(int64_t j, int64_t m, int64_t nt, int T) {
    if (j < 0) return 0;
    if (j >= m) return nt;
    return j / T;
}

// For every offset k and tile t in [0, nt]: bnd[k][t] = first pair of offset k
// with tile_of(out) >= t.  Each pair writes the entries of the tiles that begin
// at it; one extra item per offset writes the entries past its last pair.
__global__ void k_conv_bounds(const int32_t* off, const int32_t* pairs, int K3, int transposed, int64_t pair_bound,
                              const int64_t* m_out_dev, int64_t cap, int T, int64_t ntc, int32_t* bnd, Header* h,
                              PackJob pk) {
    pack_job_run(pk);
    __shared__ int32_t soff[kMaxK3 + 1];
    if (threadIdx.x <= K3) soff[threadIdx.x] = off[threadIdx.x];
    __syncthreads();
    int64_t total = soff[K3];
    if (total > pair_bound) total = pair_bound;
    if (total < 0) total = 0;
    const int64_t m = clamp_rows(m_out_dev, cap);
    const int64_t nt = (m + T - 1) / T;
    const int osel = transposed ? 0 : 1;  // column of the output row in a pair
    const int64_t stride = ntc + 1;
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < total + K3;
         p += (int64_t)gridDim.x * blockDim.x) {
        if (p < total) {
            const int k = pair_offset(soff, K3, p);
            const int64_t j = pairs[2 * p + osel];
            const int64_t cur = tile_of(j, m, nt, T);
            int64_t prev = -1;
            if (p > 0 && p != soff[k]) {
                const int64_t jp = pairs[2 * (p - 1) + osel];
                prev = tile_of(jp, m, nt, T);
                if (j <= jp) raise_flag(h, j < jp ? kFlagUnsorted : kFlagDuplicate);
            }
            if (cur < prev) continue;
            for (int64_t t = prev + 1; t <= cur; ++t) bnd[k * stride + t] = (int32_t)p;
        } else {
            const int k = (int)(p - total);
            int64_t lo = soff[k], hi = soff[k + 1];
            if (lo > total) lo = total;
            if (hi > total) hi = total;
            if (lo < 0) lo = 0;
            if (hi < 0) hi = 0;
            const int64_t prev = (hi > lo) ? tile_of(pairs[2 * (hi - 1) + osel], m, nt, T) : -1;
            for (int64_t t = prev + 1; t <= nt; ++t) bnd[k * stride + t] = (int32_t)hi;
        }
    }
}

// neighbour table: nbr[j][k] = i + 1 for every pair (i, j) of offset k, 0 elsewhere.
// The clearing launch also clears the status header (h, when given) and runs
// the layer's weight packing; the scatter that follows may then raise flags.
__global__ void k_nbr_clear(int32_t* nbr, const int64_t* m_out_dev, int64_t cap, int K3, Header* h, PackJob pk) {
    if (h && blockIdx.x == 0 && threadIdx.x == 0) {
        h->status = 0;
        h->m = 0;
        for (int i = 0; i < 4; ++i) h->aux[i] = 0;
    }
    pack_job_run(pk);
    const int64_t n = clamp_rows(m_out_dev, cap) * K3;
    for (int64_t e = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4; e < n;
         e += (int64_t)gridDim.x * blockDim.x * 4) {
        if (e + 4 <= n && ((e & 3) == 0)) {
            *(int4*)(nbr + e) = make_int4(0, 0, 0, 0);
        } else {
            for (int64_t q = e; q < n && q < e + 4; ++q) nbr[q] = 0;
        }
    }
}

// A kernel map holds at most one pair per (output, offset), and each offset's
// pairs come in increasing output order; a map that breaks either raises a flag
// (a repeated pair would otherwise overwrite instead of adding).
__global__ void k_nbr_scatter(const int32_t* off, const int32_t* pairs, int K3, int transposed, int64_t pair_bound,
                              const int64_t* m_out_dev, int64_t cap, int64_t in_rows, int32_t* nbr, Header* h) {
    __shared__ int32_t soff[kMaxK3 + 1];
    if (threadIdx.x <= K3) soff[threadIdx.x] = off[threadIdx.x];
    __syncthreads();
    int64_t total = soff[K3];
    if (total > pair_bound) total = pair_bound;
    const int64_t m = clamp_rows(m_out_dev, cap);
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < total; p += (int64_t)gridDim.x * blockDim.x) {
        const int k = pair_offset(soff, K3, p);
        const int64_t i = transposed ? pairs[2 * p + 1] : pairs[2 * p];
        const int64_t j = transposed ? pairs[2 * p] : pairs[2 * p + 1];
        if (p > 0 && p != soff[k]) {
            const int64_t jp = transposed ? pairs[2 * (p - 1)] : pairs[2 * (p - 1) + 1];
            if (j <= jp) raise_flag(h, j < jp ? kFlagUnsorted : kFlagDuplicate);
        }
        if (i >= 0 && i < in_rows && j >= 0 && j < m) nbr[j * K3 + k] = (int32_t)(i + 1);
    }
}

void launch_nbr_table(hipStream_t s, const int32_t* off, const int32_t* pairs, int K3, int64_t pair_bound,
                      const int64_t* m_out_dev, int64_t m_cap, int64_t in_rows, int32_t* nbr, Header* h) {
    unsigned gc = blocks_for(m_cap * K3, 1024);
    if (gc > 2048) gc = 2048;
    k_nbr_clear<<<gc, 256, 0, s>>>(nbr, m_out_dev, m_cap, K3, h, PackJob{});
    unsigned g = blocks_for(pair_bound + K3, 256);
    if (g > 2048) g = 2048;
    k_nbr_scatter<<<g, 256, 0, s>>>(off, pairs, K3, 0, pair_bound, m_out_dev, m_cap, in_rows, nbr, h);
}

void launch_conv_plan(hipStream_t s, const ConvPlan& p, const int32_t* off, const int32_t* pairs, int K3,
                      int transposed, int64_t pair_bound, int64_t in_rows, const PackJob& pk, bool clear_header) {
    unsigned g = blocks_for(pair_bound + K3, 256);
    if (g > 2048) g = 2048;
    if (p.use_union) {
        unsigned gc = blocks_for(p.m_cap * K3, 1024);
        if (gc > 2048) gc = 2048;
        k_nbr_clear<<<gc, 256, 0, s>>>(p.nbr, p.m_out_dev, p.m_cap, K3, clear_header ? p.h : nullptr, pk);
        k_nbr_scatter<<<g, 256, 0, s>>>(off, pairs, K3, transposed, pair_bound, p.m_out_dev, p.m_cap, in_rows, p.nbr,
                                        p.h);
    } else {
        if (clear_header) launch_clear_header(s, p.h);
        k_conv_bounds<<<g, 256, 0, s>>>(off, pairs, K3, transposed, pair_bound, p.m_out_dev, p.m_cap, p.tile_rows,
                                        p.ntile_cap, p.bnd, p.h, pk);
    }
}

// ---------------------------------------------------------------------------
// weight packing into MFMA operand fragments:
// wpack[((k * KCH + kc) * NB + nb) * 64 + lane] holds, for e = 0..7,
//   W[k][kc*32 + 8*(lane/16) + e][nb*16 + lane%16]
// i.e. lane l carries output channel nb*16 + l%16 and 8 consecutive input
// channels: the A operand of D = W^T G^T (or the B operand of D = G W).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_pack_job(PackJob q) { pack_job_run(q); }

void launch_pack_job(hipStream_t s, const PackJob& q) {
    if (q.total <= 0) return;
    int64_t g = (q.total + 255) / 256;
    if (g > 1024) g = 1024;
    k_pack_job<<<(unsigned)g, 256, 0, s>>>(q);
}

static int conv_kch(int Cin);

void* plan_wpack_ws(Arena& a, int K3, int Cin, int Cout) {
    int KCH = conv_kch(Cin), NB = (Cout + 15) / 16;
    return a.take<uint4>((size_t)K3 * KCH * NB * 64);
}

// ---------------------------------------------------------------------------
// MFMA tile kernel
// ---------------------------------------------------------------------------
// LDS layout (dynamic, in this order):
//   float acc[T + 1][Cout + 4]        fp32 accumulator of the tile (+ a spill row)
//   uint4 wslot[NW][KCH*NBW*64]       each wave's weight fragments of the next offset
//   int2  tab[T/16*K3 + K3]           chunk -> (first pair, offset | pairs << 8)
//   int   nextk[K3], nchunk
struct ConvTileSmem {
    static __host__ __device__ int acc_stride(int Cout) { return Cout + 4; }
    static __host__ __device__ int tab_entries(int T, int K3) { return T / kChunk * K3 + K3; }
    static __host__ __device__ size_t acc_bytes(int T, int Cout) { return (size_t)(T + 1) * acc_stride(Cout) * 4; }
    static __host__ __device__ size_t wslot_bytes(int KCH, int NBW) { return (size_t)KCH * NBW * 64 * 16; }
    static __host__ __device__ size_t bytes(int T, int Cout, int K3, int KCH, int NBW, int NW) {
        return acc_bytes(T, Cout) + (size_t)NW * wslot_bytes(KCH, NBW) + (size_t)tab_entries(T, K3) * 8 +
               (size_t)(K3 + 1) * 4;
    }
};

// Every wave runs a software pipeline over the chunks of its tile: the pair
// (input row, output row) of chunk c + kPairAhead and the gathered input rows
// of chunk c + kRowAhead are loaded while chunk c is multiplied.  The chunk
// loop is unrolled by kPairAhead so that each pipeline slot is a fixed
// register, and every load writes straight into the slot just consumed (a
// register copy of a value still in flight would wait for it).  Gathers and
// pair loads are raw buffer loads: 32-bit offsets from a scalar base, and the
// hardware range check returns zeros for an absent row.
//
// Weights take a separate path.  Vector-memory loads complete in issue order
// and are waited for by count, so a register load of the next offset's weights
// would, when waited for, also wait for every gather issued before it.  Instead
// each wave copies the weight fragments of the next offset straight into its
// own LDS slot (global_load_lds_dwordx4, one 1 KB fragment block per
// instruction) when it enters an offset, and at the next offset change waits
// only until those copies are older than the loads issued since; it then reads
// the fragments from LDS.  Every pipeline step issues exactly KCH + 1
// vector-memory loads, which makes that count exact.
constexpr int kRowAhead = 4;
constexpr int kPairAhead = 8;
template <int DT, int KCH, int NBW, int TR>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_conv_tile(ConvPlan p, const uint16_t* __restrict__ in, int Cin,
                                                    int64_t in_rows, const int32_t* __restrict__ pairs,
                                                    int64_t pair_bound,
                                                    const uint4* __restrict__ wpack, int NB,
                                                    const float* __restrict__ scale, const float* __restrict__ shift,
                                                    int relu, uint16_t* __restrict__ out, int Cout) {
    constexpr int kStepLoads = KCH + 1;  // vector-memory loads per pipeline step
    constexpr int kFrag = KCH * NBW;     // weight fragments per wave and offset
    extern __shared__ __align__(16) unsigned char smem[];
    const int T = p.tile_rows, K3 = p.K3;
    const int nthr = blockDim.x, NW = nthr >> 6;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r16 = lane & 15, g = lane >> 4;

    // tiles of one XCD are contiguous (blocks are dispatched round-robin over the 8 XCDs)
    const int64_t G = gridDim.x;
    const int64_t bid = blockIdx.x;
    const int64_t xq = G / 8, xr = G % 8, x = bid % 8;
    const int64_t t = x * xq + (x < xr ? x : xr) + bid / 8;

    const int64_t m = clamp_rows(p.m_out_dev, p.m_cap);
    const int64_t nt = (m + T - 1) / T;
    if (t >= nt) return;
    const int64_t row0 = t * T;
    const int rows = (int)((m - row0) < T ? (m - row0) : T);

    const int ACS = ConvTileSmem::acc_stride(Cout);
    float* acc = (float*)smem;  // T + 1 rows: row T absorbs the lanes without a pair
    uint4* wslots = (uint4*)(smem + ConvTileSmem::acc_bytes(T, Cout));
    uint4* wslot = wslots + (size_t)wave * kFrag * 64;
    int2* tab = (int2*)(wslots + (size_t)NW * kFrag * 64);
    int* nextk = (int*)(tab + ConvTileSmem::tab_entries(T, K3));
    int* s_nchunk = nextk + K3;

    // chunk table of this tile: offsets in ascending order, 16 pairs per chunk
    if (wave == 0) {
        const int64_t bs = p.ntile_cap + 1;
        int lo = 0, n = 0;
        if (lane < K3) {
            // clamped into [0, pair_bound): a map that is not a valid kernel map
            // (unsorted groups, repeated output rows) gives wrong sums, never a
            // read outside the pair list or the chunk table
            int64_t l = p.bnd[lane * bs + t], hh = p.bnd[lane * bs + t + 1];
            l = l < 0 ? 0 : (l > pair_bound ? pair_bound : l);
            hh = hh < l ? l : (hh > pair_bound ? pair_bound : hh);
            if (hh - l > T) {
                raise_flag(p.h, kFlagUnsorted);
                hh = l + T;
            }
            lo = (int)l;
            n = (int)(hh - l);
        }
        const int nch = (n + kChunk - 1) / kChunk;
        int incl = nch;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            int y = __shfl_up(incl, d, 64);
            if (lane >= d) incl += y;
        }
        const int start = incl - nch;
        for (int c = 0; c < nch; ++c) {
            const int np = (n - c * kChunk) < kChunk ? (n - c * kChunk) : kChunk;
            tab[start + c] = make_int2(lo + c * kChunk, lane | (np << 8));
        }
        const uint64_t has = __ballot(nch > 0);
        if (lane < K3) {
            const uint64_t later = has & ~((2ull << lane) - 1ull);
            nextk[lane] = later ? __builtin_ctzll(later) : -1;
        }
        if (lane == 63) *s_nchunk = incl;
    }
    // zero the accumulator (and the spill row)
    for (int e = tid; e < (T + 1) * ACS / 4; e += nthr) ((float4*)acc)[e] = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();
    const int NC = *s_nchunk;

    const uint32_t row_bytes = (uint32_t)Cin * 2u;
    const __amdgpu_buffer_rsrc_t in_rs = make_rsrc(in, (uint32_t)(in_rows * (int64_t)row_bytes));
    const __amdgpu_buffer_rsrc_t pr_rs = make_rsrc(pairs, (uint32_t)(pair_bound * 8));
    const int qin = Cin / 8;                      // 16-byte pieces of an input row
    const bool ragged = Cin != KCH * 32;          // some pieces of the last K block are padding
    const int nb0 = wave * NBW;                   // the wave's output channel blocks

    // weight fragments of offset k -> this wave's LDS slot (asynchronous)
    const uint64_t wbase = (uint64_t)(uintptr_t)wpack + (uint64_t)nb0 * 1024u;
    const uint32_t wslot_lds = __builtin_amdgcn_readfirstlane(lds_addr(wslot));
    const uint32_t wlane = (uint32_t)lane * 16u;
    auto dma_w = [&](int k) {
        lds_wait();  // the slot's previous contents have been read
        const uint64_t kb = wbase + (uint64_t)(k * KCH) * (uint64_t)NB * 1024u;
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                lds_dma_x4(kb + (uint64_t)(kc * NB + nb) * 1024u, wlane,
                           wslot_lds + (uint32_t)((kc * NBW + nb) * 1024));
    };
    uint4 wc[KCH][NBW];
    auto read_w = [&]() {
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) wc[kc][nb] = wslot[(kc * NBW + nb) * 64 + lane];
    };

    // --- pipeline registers ------------------------------------------------
    // ps[c % kPairAhead]: raw (in, out) pair of chunk c for lane row r16, valid
    // iff bit c % kPairAhead of pv; rs[c % kRowAhead]: its gathered row pieces
    // (zeros for an absent or out-of-range row)
    i32x2 ps[kPairAhead];
    uint32_t pv = 0;
    i32x4 rs[kRowAhead][KCH];

    // chunks past NC (the loop runs whole groups of kPairAhead) are empty:
    // their loads read past every record and return zeros
    auto load_pair = [&](int cc, i32x2& dst) -> bool {
        const int2 te = tab[cc < NC ? cc : NC - 1];
        const bool valid = cc < NC && r16 < (te.y >> 8);
        dst = __builtin_amdgcn_raw_buffer_load_b64(pr_rs, valid ? (uint32_t)(te.x + r16) * 8u : kOutOfRange, 0, 0);
        return valid;
    };
    const uint32_t in_rows32 = (uint32_t)in_rows;  // in_rows * row_bytes < 2^32 (checked by the host)
    auto load_rows = [&](const i32x2& pr, bool valid, i32x4 (&dst)[KCH]) {
        const uint32_t i = (uint32_t)(TR ? pr.y : pr.x);
        const uint32_t base = (valid && i < in_rows32) ? i * row_bytes + (uint32_t)g * 16u : kOutOfRange;
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc) {
            uint32_t off = base + kc * 64;
            if (ragged && kc * 4 + g >= qin) off = kOutOfRange;
            dst[kc] = __builtin_amdgcn_raw_buffer_load_b128(in_rs, off, 0, 0);
        }
    };

    int kcur = -1;
    int since = kRowAhead;  // pipeline steps since the last weight copy was issued
    if (NC > 0) {
        kcur = tab[0].y & 0xFF;
        dma_w(kcur);
        vm_wait<0>();
        read_w();
        const int kn = nextk[kcur];
        if (kn >= 0) dma_w(kn);
#pragma unroll
        for (int j = 0; j < kPairAhead; ++j)
            if (load_pair(j, ps[j])) pv |= 1u << j;
#pragma unroll
        for (int j = 0; j < kRowAhead; ++j) load_rows(ps[j], (pv >> j) & 1u, rs[j]);
    }

    for (int c0 = 0; c0 < NC; c0 += kPairAhead) {
#pragma unroll
        for (int u = 0; u < kPairAhead; ++u) {
            const int c = c0 + u;
            const int sr = u % kRowAhead;
            // (a) entering a new offset: its weights were copied one offset ago
            const int k = c < NC ? __builtin_amdgcn_readfirstlane(tab[c].y & 0xFF) : kcur;
            if (k != kcur) {
                // loads issued after that copy: `since` steps of kStepLoads each;
                // after kRowAhead steps the row waits below have covered it
                if (since >= kRowAhead) vm_wait<kRowAhead * kStepLoads>();
                else if (since == 3) vm_wait<3 * kStepLoads>();
                else if (since == 2) vm_wait<2 * kStepLoads>();
                else vm_wait<1 * kStepLoads>();
                read_w();
                kcur = k;
                const int kn = nextk[k];
                if (kn >= 0) {
                    dma_w(kn);
                    since = 0;
                }
            }
            // (c) this chunk: read the output-row slices, multiply, add, write back
            const int o = (TR ? ps[u].x : ps[u].y) - (int)row0;
            const bool live = ((pv >> u) & 1u) && (uint32_t)o < (uint32_t)rows;
            float4* arow = (float4*)(acc + (live ? o : T) * ACS) + nb0 * 4 + g;
            float4 av[NBW];
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) av[nb] = arow[nb * 4];
            f32x4 d[NBW];
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) d[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    d[nb] = mfma16x16x32<DT>(wc[kc][nb], __builtin_bit_cast(uint4, rs[sr][kc]), d[nb]);
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                arow[nb * 4] = make_float4(av[nb].x + d[nb][0], av[nb].y + d[nb][1], av[nb].z + d[nb][2],
                                           av[nb].w + d[nb][3]);
            // (b) refill the consumed slots: rows of chunk c + kRowAhead, pair of chunk c + kPairAhead
            const int ur = (u + kRowAhead) % kPairAhead;
            load_rows(ps[ur], (pv >> ur) & 1u, rs[sr]);
            const bool pnv = load_pair(c + kPairAhead, ps[u]);
            pv = (pv & ~(1u << u)) | (pnv ? (1u << u) : 0u);
            ++since;
        }
    }
    vm_wait<0>();  // no weight copy may still target LDS past this point
    __syncthreads();

    // epilogue: 8 channels per item, one 16-byte store each
    const int c8n = Cout / 8;
    for (int e = tid; e < rows * c8n; e += nthr) {
        const int r = e / c8n, c8 = e - r * c8n;
        const float4 a0 = *(const float4*)(acc + (size_t)r * ACS + 8 * c8);
        const float4 a1 = *(const float4*)(acc + (size_t)r * ACS + 8 * c8 + 4);
        float v[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        float rv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        if (p.res) {
            const uint4 u = *(const uint4*)((const uint16_t*)p.res + (row0 + r) * Cout + 8 * c8);
            const uint32_t uu[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                rv[2 * j] = from16<DT>(uu[j] & 0xFFFF);
                rv[2 * j + 1] = from16<DT>(uu[j] >> 16);
            }
        }
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int col = 8 * c8 + j;
            float y = v[j] * (scale ? scale[col] : 1.f) + (shift ? shift[col] : 0.f) + rv[j];
            if (relu) y = fmaxf(y, 0.f);
            v[j] = y;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = (uint32_t)to16<DT>(v[2 * j]) | ((uint32_t)to16<DT>(v[2 * j + 1]) << 16);
        *(uint4*)(out + (row0 + r) * Cout + 8 * c8) = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

// ---------------------------------------------------------------------------
// vector-ALU tile kernel (f32, or shapes the MFMA kernel does not take):
// 64 output channels per workgroup (grid.y), 4 pair lanes; LDS accumulator
// [T][64]; a barrier between offsets keeps the updates of one row ordered.
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(256) void k_conv_tile_valu(ConvPlan p, const void* in, int Cin, int64_t in_rows,
                                                        const int32_t* pairs, int64_t pair_bound, int transposed,
                                                        const void* W,
                                                        const float* scale, const float* shift, int relu, void* out,
                                                        int Cout) {
    extern __shared__ __align__(16) unsigned char smem[];
    float* acc = (float*)smem;
    const int T = p.tile_rows, K3 = p.K3;
    const int64_t t = blockIdx.x;
    const int64_t m = clamp_rows(p.m_out_dev, p.m_cap);
    const int64_t nt = (m + T - 1) / T;
    if (t >= nt) return;
    const int64_t row0 = t * T;
    const int rows = (int)((m - row0) < T ? (m - row0) : T);
    const int cl = threadIdx.x & 63, rl = threadIdx.x >> 6;
    const int col = blockIdx.y * 64 + cl;
    const bool cok = col < Cout;
    for (int e = threadIdx.x; e < T * 64; e += blockDim.x) acc[e] = 0.f;
    __syncthreads();
    const int isel = transposed ? 1 : 0;
    const int64_t bs = p.ntile_cap + 1;
    const int64_t ldc = p.w_ldc > 0 ? p.w_ldc : Cout, ldk = p.w_ldk > 0 ? p.w_ldk : (int64_t)Cin * Cout;
    const int64_t ldcol = p.w_ldcol > 0 ? p.w_ldcol : 1;
    for (int k = 0; k < K3; ++k) {
        int64_t lo = p.bnd[k * bs + t], hi = p.bnd[k * bs + t + 1];
        lo = lo < 0 ? 0 : (lo > pair_bound ? pair_bound : lo);
        hi = hi < lo ? lo : (hi > pair_bound ? pair_bound : hi);
        for (int64_t pi = lo + rl; pi < hi; pi += 4) {
            const int32_t i = pairs[2 * pi + isel];
            const int64_t o = (int64_t)pairs[2 * pi + 1 - isel] - row0;
            if (!cok || o < 0 || o >= rows || i < 0 || i >= in_rows) continue;
            float s = 0.f;
            for (int ci = 0; ci < Cin; ++ci)
                s += ld_feat<DT>(in, (int64_t)i * Cin + ci) * ld_feat<DT>(W, k * ldk + ci * ldc + col * ldcol);
            acc[o * 64 + cl] += s;
        }
        __syncthreads();
    }
    if (!cok) return;
    const float sc = scale ? scale[col] : 1.f, sh = shift ? shift[col] : 0.f;
    for (int r = rl; r < rows; r += 4) {
        float y = acc[r * 64 + cl] * sc + sh;
        if (p.res) y += ld_feat<DT>(p.res, (row0 + r) * Cout + col);
        if (relu) y = fmaxf(y, 0.f);
        st_feat<DT>(out, (row0 + r) * Cout + col, y);
    }
}

// ---------------------------------------------------------------------------
// host dispatch
// ---------------------------------------------------------------------------
static int conv_kch(int Cin) {
    const int k = (Cin + 31) / 32;
    return k <= 4 ? k : (k <= 6 ? 6 : 8);
}

// channel blocks per wave of the tile kernel: the largest of 4, 3, 2, 1 that
// divides Cout / 16 while the wave's weight fragments stay within 12 registers
// of 16 bytes
static int conv_nbw(int KCH, int NB) {
    for (int w = 4; w > 1; --w)
        if (NB % w == 0 && KCH * w <= 12 && KCH < 6 && NB / w <= 8) return w;
    // wide inputs and outputs (e.g. 256 -> 256): two blocks per wave where one
    // each would take more than 8 waves
    if (KCH >= 6 && NB > 8 && NB % 2 == 0 && NB / 2 <= 8) return 2;
    return 1;
}

bool conv_mfma_supported(int Cin, int Cout, int dt) {
    if (dt == SPV_F32 || Cin % 8 != 0 || Cout % 16 != 0 || Cin > 256 || Cout > 256) return false;
    const int NB = Cout / 16;
    return NB / conv_nbw(conv_kch(Cin), NB) <= 8;  // at most 8 waves per workgroup
}

static int conv_tile_rows(int Cin, int Cout, int dt) {
    if (!conv_mfma_supported(Cin, Cout, dt)) return 128;
    const int KCH = conv_kch(Cin), NB = Cout / 16, NBW = conv_nbw(KCH, NB), NW = NB / NBW;
    // the largest tile with which two workgroups share a compute unit's 160 KB of LDS
    for (int T = 128; T > 16; T >>= 1)
        if (ConvTileSmem::bytes(T, Cout, kMaxK3, KCH, NBW, NW) <= 80 * 1024) return T;
    return 16;
}

template <int DT, int KCH, int NBW>
static void launch_tile3(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows,
                         const int32_t* pairs, int64_t pair_bound, int transposed, const void* wpack,
                         const float* scale, const float* shift, int relu, void* out, int Cout) {
    const int NB = Cout / 16, NW = NB / NBW;
    const size_t lds = ConvTileSmem::bytes(p.tile_rows, Cout, p.K3, KCH, NBW, NW);
    const unsigned grid = (unsigned)(p.ntile_cap > 0 ? p.ntile_cap : 1);
    // opt in to more than 64 KB of dynamic LDS (once per instantiation)
    static const bool lds_ok = hipFuncSetAttribute((const void*)k_conv_tile<DT, KCH, NBW, 0>,
                                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                                   160 * 1024) == hipSuccess &&
                               hipFuncSetAttribute((const void*)k_conv_tile<DT, KCH, NBW, 1>,
                                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                                   160 * 1024) == hipSuccess;
    (void)lds_ok;
    if (transposed)
        k_conv_tile<DT, KCH, NBW, 1><<<grid, 64 * NW, lds, s>>>(p, (const uint16_t*)in, Cin, in_rows, pairs,
                                                                pair_bound, (const uint4*)wpack, NB, scale, shift,
                                                                relu, (uint16_t*)out, Cout);
    else
        k_conv_tile<DT, KCH, NBW, 0><<<grid, 64 * NW, lds, s>>>(p, (const uint16_t*)in, Cin, in_rows, pairs,
                                                                pair_bound, (const uint4*)wpack, NB, scale, shift,
                                                                relu, (uint16_t*)out, Cout);
}

template <int DT, int KCH>
static void launch_tile_kch(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows,
                            const int32_t* pairs, int64_t pair_bound, int transposed, const void* wpack,
                            const float* scale, const float* shift, int relu, void* out, int Cout) {
    switch (conv_nbw(KCH, Cout / 16)) {
#define SPV_NBW_CASE(W)                                                                                        \
    case W:                                                                                                    \
        if constexpr ((KCH * W <= 12 && (KCH < 6 || W == 1)) || (KCH >= 6 && W == 2))                         \
            launch_tile3<DT, KCH, W>(s, p, in, Cin, in_rows, pairs, pair_bound, transposed, wpack, scale, shift, \
                                     relu, out, Cout);                                                         \
        break;
        SPV_NBW_CASE(1)
        SPV_NBW_CASE(2)
        SPV_NBW_CASE(3)
        SPV_NBW_CASE(4)
#undef SPV_NBW_CASE
    }
}

template <int DT>
static void launch_tile(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows,
                        const int32_t* pairs, int64_t pair_bound, int transposed, const void* wpack,
                        const float* scale, const float* shift, int relu, void* out, int Cout) {
    switch (conv_kch(Cin)) {
#define SPV_KCH_CASE(K)                                                                                       \
    case K:                                                                                                   \
        launch_tile_kch<DT, K>(s, p, in, Cin, in_rows, pairs, pair_bound, transposed, wpack, scale, shift, relu, \
                               out, Cout);                                                                    \
        break;
        SPV_KCH_CASE(1)
        SPV_KCH_CASE(2)
        SPV_KCH_CASE(3)
        SPV_KCH_CASE(4)
        SPV_KCH_CASE(6)
        SPV_KCH_CASE(8)
#undef SPV_KCH_CASE
    }
}

PackJob conv_pack_job(int K3, const void* W, void* wpack, int Cin, int Cout, int dt, int ldc, int64_t ldk,
                      int ldcol) {
    PackJob q{(const uint16_t*)W, (uint4*)wpack, K3, Cin, Cout, 0, 0, 0, ldc > 0 ? ldc : Cout,
              ldk > 0 ? ldk : (int64_t)Cin * Cout, ldcol > 0 ? ldcol : 1};
    if (!conv_mfma_supported(Cin, Cout, dt)) return q;
    q.KCH = conv_kch(Cin);
    q.NB = Cout / 16;
    q.total = (int64_t)K3 * q.KCH * q.NB * 64;
    return q;
}

// The packing of W'[k] = W[26 - k]^T ([27][Cout][Cin] from W [27][Cin][Cout]):
// the input gradient of a submanifold conv as a conv on the same neighbour
// table.  W'[k][c][col] = W[26 - k][col][c] sits at (W + 26 Cin Cout) +
// k (-Cin Cout) + c + col Cout.
PackJob conv_pack_job_mirrored(const void* W, void* wpack, int Cin, int Cout, int dt) {
    const int64_t per = (int64_t)Cin * Cout;
    PackJob q{(const uint16_t*)W + 26 * per, (uint4*)wpack, 27, Cout, Cin, 0, 0, 0, 1, -per, Cout};
    if (!conv_mfma_supported(Cout, Cin, dt)) return q;
    q.KCH = conv_kch(Cout);
    q.NB = Cin / 16;
    q.total = (int64_t)27 * q.KCH * q.NB * 64;
    return q;
}

// the MFMA kernels address the input rows, the neighbour table and the pair
// list with 32-bit buffer offsets
static bool conv_fits_buffers(int64_t in_rows, int Cin, int64_t pair_bound) {
    return in_rows * (int64_t)Cin * 2 <= (int64_t)0xFFFFE000 && pair_bound * 8 <= (int64_t)0xFFFFE000;
}

int conv_kernel_choice(int K3, int Cin, int Cout, int dt, int64_t m_out_cap, int64_t in_rows, int64_t pair_bound,
                       bool sparse_transposed) {
    if (!sparse_transposed && union_supported(K3, Cin, Cout, dt) && m_out_cap * K3 * 4 <= (int64_t)0xFFFFE000 &&
        conv_fits_buffers(in_rows, Cin, 0))
        return kConvUnion;
    if (conv_mfma_supported(Cin, Cout, dt) && conv_fits_buffers(in_rows, Cin, pair_bound)) return kConvTile;
    return kConvValu;
}

void launch_conv_run(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, const int32_t* pairs,
                     int64_t pair_bound, int transposed, const void* W, const void* wpack, const float* scale,
                     const float* shift, int relu, void* out, int Cout, int dt) {
    if (p.use_union) {  // the plan checked every bound this kernel needs
        launch_conv_union(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out, dt);
        return;
    }
    if (conv_mfma_supported(Cin, Cout, dt) && conv_fits_buffers(in_rows, Cin, pair_bound)) {
        if (dt == SPV_BF16)
            launch_tile<SPV_BF16>(s, p, in, Cin, in_rows, pairs, pair_bound, transposed, wpack, scale, shift, relu,
                                  out, Cout);
        else
            launch_tile<SPV_F16>(s, p, in, Cin, in_rows, pairs, pair_bound, transposed, wpack, scale, shift, relu,
                                 out, Cout);
        return;
    }
    dim3 grid((unsigned)(p.ntile_cap > 0 ? p.ntile_cap : 1), (unsigned)((Cout + 63) / 64));
    const size_t lds = (size_t)p.tile_rows * 64 * 4;
    if (dt == SPV_F32)
        k_conv_tile_valu<SPV_F32><<<grid, 256, lds, s>>>(p, in, Cin, in_rows, pairs, pair_bound, transposed, W, scale,
                                                         shift, relu, out, Cout);
    else if (dt == SPV_BF16)
        k_conv_tile_valu<SPV_BF16><<<grid, 256, lds, s>>>(p, in, Cin, in_rows, pairs, pair_bound, transposed, W,
                                                          scale, shift, relu, out, Cout);
    else
        k_conv_tile_valu<SPV_F16><<<grid, 256, lds, s>>>(p, in, Cin, in_rows, pairs, pair_bound, transposed, W,
                                                         scale, shift, relu, out, Cout);
}

}  // namespace spv
