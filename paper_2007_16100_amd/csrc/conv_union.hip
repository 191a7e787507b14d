// conv_union.hip -- sparse convolution on a 3x3x3 kernel map (Sec. 3.2 / 3.3)
// with register accumulators: the neighbour-table kernel described in conv.hip.
#include <type_traits>

#include "conv_common.hpp"

namespace spv {

// f(integral_constant<int, i>) for i = B .. E-1, each i a compile-time constant
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// ---------------------------------------------------------------------------
// neighbour-table kernel (3x3x3 maps)
// ---------------------------------------------------------------------------
// One workgroup of NW waves per CU; wave w owns RB blocks of 16 output rows and
// all output channels (NB blocks of 16).  The accumulators of a block are
// D = W^T G^T fragments: lane (r16, g) holds output channels nb*16 + 4g .. 4g+3
// of row r16, which is also the order in which they are stored.
//
// The 27 offsets run in phases of PH: at the start of a phase the workgroup
// copies W of the phase's offsets into LDS with global->LDS loads (one barrier
// before, one wait for every load of the wave and one barrier after);
// inside a phase the waves never synchronize and load no weights, each one
// streaming its own rows:
//   step k: loads the neighbour indices of offset k+3 and gathers the rows of
//           offset k+1 (a block with no neighbour at that offset, or a lane
//           whose row has none, reads zeros from outside the buffer), then
//           multiplies the rows gathered for offset k by W[k] one 32-channel
//           slab at a time, skipping blocks without a neighbour at k.
// All other loads are ordinary vector-memory loads the compiler sees, the same
// number every step, so its waits (which count outstanding loads in issue
// order) stay exact and a step waits for its own rows only: the weight copies
// it does not see are all complete (vmcnt 0) before the phase starts.
constexpr int kUK3 = 27;
constexpr int kNAhead = 3;  // neighbour indices: steps ahead
constexpr int kRAhead = 1;  // gathered rows: steps ahead

template <int DT, int KCH, int NB, int RB, int NW, int PH>
__global__ __launch_bounds__(64 * NW) void k_conv_union(
    const int32_t* __restrict__ nbr, const int64_t* __restrict__ m_out_dev, int64_t m_cap,
    const uint16_t* __restrict__ in, int Cin, int64_t in_rows, const uint4* __restrict__ wpack,
    const float* __restrict__ scale, const float* __restrict__ shift, int relu, const uint16_t* __restrict__ res,
    uint16_t* __restrict__ out) {
    constexpr int K3 = kUK3;
    constexpr int FR = KCH * NB;  // 1 KB weight fragments per offset
    constexpr int Cout = NB * 16;
    __shared__ __align__(16) uint4 wl[PH * FR * 64];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r16 = lane & 15, g = lane >> 4;

    // Workgroups are dispatched round-robin over the 8 XCDs (workgroup b to XCD
    // b % 8).  The row tiles that exist (from the live row count, not the
    // capacity the grid was sized for) are split into 8 consecutive ranges, one
    // per XCD, so neighbouring tiles share an L2 and every XCD gets work.
    const int64_t m = clamp_rows(m_out_dev, m_cap);
    constexpr int64_t rows_wg = (int64_t)NW * RB * 16;
    const int64_t bid = blockIdx.x, x = bid % 8, seq = bid / 8;
    const int64_t ga = (m + rows_wg - 1) / rows_wg, xq = ga / 8, xr = ga % 8;
    if (seq >= xq + (x < xr ? 1 : 0)) return;  // the whole workgroup
    const int64_t wg = x * xq + (x < xr ? x : xr) + seq;
    const int64_t blk0 = (wg * NW + wave) * RB;

    const __amdgpu_buffer_rsrc_t nb_rs = make_rsrc(nbr, (uint32_t)(m * K3 * 4));
    const uint32_t row_bytes = (uint32_t)Cin * 2u;
    const __amdgpu_buffer_rsrc_t in_rs = make_rsrc(in, (uint32_t)(in_rows * (int64_t)row_bytes));
    const uint32_t in_rows32 = (uint32_t)in_rows;

    // nbr byte offset of (row of block b, offset 0) for this lane; rows past m read zeros
    uint32_t nboff[RB];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
        const int64_t row = (blk0 + b) * 16 + r16;
        nboff[b] = row < m ? (uint32_t)(row * K3 * 4) : kOutOfRange;
    }
    // offsets present in each block (union over its 16 rows), wave-uniform
    uint32_t umask[RB];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
        uint32_t bits = 0;
#pragma unroll
        for (int k = 0; k < K3; k += 4) {
            if (k + g < K3) {
                const int v = __builtin_amdgcn_raw_buffer_load_b32(nb_rs, nboff[b] + (uint32_t)(k + g) * 4u, 0, 0);
                bits |= (v > 0 ? 1u : 0u) << (k + g);
            }
        }
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) bits |= __shfl_xor(bits, d, 64);
        umask[b] = __builtin_amdgcn_readfirstlane(bits);
    }

    auto load_nbr = [&](int k, int (&dst)[RB]) __attribute__((always_inline)) {
#pragma unroll
        for (int b = 0; b < RB; ++b)
            dst[b] = __builtin_amdgcn_raw_buffer_load_b32(nb_rs, nboff[b] + (uint32_t)k * 4u, 0, 0);
    };
    // gathered rows of offset kr (16-byte chunks g + 4 kc of row i)
    // Every step issues the same RB * KCH loads, so the compiler's vmcnt waits
    // are exact and a step waits for its own rows only, never for the rows it
    // prefetches: a block without a neighbour at kr, or a lane whose row has
    // none, loads from an out-of-range offset, which returns zeros and touches
    // no memory.
    auto load_rows = [&](int kr, const int (&nb1)[RB], i32x4 (&dst)[RB][KCH]) __attribute__((always_inline)) {
#pragma unroll
        for (int b = 0; b < RB; ++b) {
            const uint32_t i = (uint32_t)(nb1[b] - 1);  // stored as row + 1; 0 = absent
            const bool have = ((umask[b] >> kr) & 1u) && i < in_rows32;
            const uint32_t base = have ? i * row_bytes + (uint32_t)g * 16u : kOutOfRange;
#pragma unroll
            for (int kc = 0; kc < KCH; ++kc)
                dst[b][kc] = __builtin_amdgcn_raw_buffer_load_b128(in_rs, base + (uint32_t)kc * 64u, 0, 0);
        }
    };

    int ns[kNAhead + 1][RB];         // neighbour indices of offset j in slot j % (kNAhead + 1)
    i32x4 rs[kRAhead + 1][RB][KCH];  // gathered rows of offset j in slot j % (kRAhead + 1)
#pragma unroll
    for (int j = 0; j < kNAhead; ++j) load_nbr(j, ns[j]);
#pragma unroll
    for (int j = 0; j < kRAhead; ++j) load_rows(j, ns[j], rs[j]);

    f32x4 acc[RB][NB];
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[b][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const i32x4* wsrc = (const i32x4*)wpack;
    static_for<0, K3>([&](auto kk) __attribute__((always_inline)) {
        constexpr int k = decltype(kk)::value;
        if constexpr (k % PH == 0) {
            // a new phase: once every wave is done with the previous weights,
            // copy W[k .. k+PH) into LDS
            // (global->LDS copies, all issued before one wait: a copy through
            // registers would wait for each fragment -- and every gather in
            // flight -- in turn)
            constexpr int nf = (K3 - k < PH ? K3 - k : PH) * FR;
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            const uint64_t gw = (uint64_t)(wsrc + (int64_t)k * FR * 64);
            for (int f = wave; f < nf; f += NW)
                lds_dma_x4(gw + (uint64_t)f * 1024u, (uint32_t)lane * 16u, lds_addr(wl + f * 64));
            vm_wait<0>();
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
        }
        if constexpr (k + kNAhead < K3) load_nbr(k + kNAhead, ns[(k + kNAhead) % (kNAhead + 1)]);
        if constexpr (k + kRAhead < K3)
            load_rows(k + kRAhead, ns[(k + kRAhead) % (kNAhead + 1)], rs[(k + kRAhead) % (kRAhead + 1)]);
        const i32x4* wk = (const i32x4*)wl + (k % PH) * FR * 64;
        uint32_t present = 0;
#pragma unroll
        for (int b = 0; b < RB; ++b) present |= ((umask[b] >> k) & 1u) << b;
        if (present) {
#pragma unroll
            for (int kc = 0; kc < KCH; ++kc) {
                i32x4 wf[NB];
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) wf[nb] = wk[(kc * NB + nb) * 64 + lane];
#pragma unroll
                for (int b = 0; b < RB; ++b) {
                    if ((present >> b) & 1u) {
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb)
                            acc[b][nb] = mfma16x16x32<DT>(__builtin_bit_cast(uint4, wf[nb]),
                                                          __builtin_bit_cast(uint4, rs[k % (kRAhead + 1)][b][kc]),
                                                          acc[b][nb]);
                    }
                }
            }
        }
    });

    // epilogue: act(scale * acc + shift), 4 channels (8 bytes) per store
    float sc[NB][4], sh[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sc[nb][e] = scale ? scale[nb * 16 + 4 * g + e] : 1.f;
            sh[nb][e] = shift ? shift[nb * 16 + 4 * g + e] : 0.f;
        }
#pragma unroll
    for (int b = 0; b < RB; ++b) {
        const int64_t row = (blk0 + b) * 16 + r16;
        if (row >= m) continue;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            float y[4], rv[4] = {0.f, 0.f, 0.f, 0.f};
            if (res) {  // the residual input, same layout as the output
                const uint2 u = *(const uint2*)(res + row * Cout + nb * 16 + 4 * g);
                rv[0] = from16<DT>(u.x & 0xFFFF);
                rv[1] = from16<DT>(u.x >> 16);
                rv[2] = from16<DT>(u.y & 0xFFFF);
                rv[3] = from16<DT>(u.y >> 16);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                y[e] = acc[b][nb][e] * sc[nb][e] + sh[nb][e] + rv[e];
                if (relu) y[e] = fmaxf(y[e], 0.f);
            }
            const uint32_t lo = (uint32_t)to16<DT>(y[0]) | ((uint32_t)to16<DT>(y[1]) << 16);
            const uint32_t hi = (uint32_t)to16<DT>(y[2]) | ((uint32_t)to16<DT>(y[3]) << 16);
            *(uint2*)(out + row * Cout + nb * 16 + 4 * g) = make_uint2(lo, hi);
        }
    }
}

// instantiated for C_in, C_out in {32, 64, 96, 128, 256} (the widths of the
// blocks and networks built here, square layers and the channel changes
// between stages); other shapes use the tile kernel
bool union_supported(int K3, int Cin, int Cout, int dt) {
    if (K3 != 27 || dt == SPV_F32) return false;
    const auto width_ok = [](int c) { return c == 32 || c == 64 || c == 96 || c == 128 || c == 256; };
    return width_ok(Cin) && width_ok(Cout);
}

// Launch shape per width: 11 waves of 2 blocks (352 rows per workgroup: a
// ~9*10^4-voxel scan gives ~250 workgroups, one round over the 256 CUs with
// nearly every CU busy), phases of as many offsets as fit in 128 KB of LDS.
// 128 -> 128 takes one block per wave: two would not fit the 168 registers a
// wave has at 11 waves per workgroup.
template <int DT, int KCH, int NB>
static void launch_union_c(hipStream_t s, const ConvPlan& p, const void* in, int64_t in_rows, const void* wpack,
                           const float* scale, const float* shift, int relu, void* out) {
    constexpr int FR = KCH * NB;
    // 256 channels in or out: 8 waves (256 registers each); 256 -> 256 holds one
    // offset's 128 KB of weights per phase
    constexpr int RB = FR >= 32 ? 1 : 2, NW = (NB >= 16 || KCH >= 8) ? 8 : 11;
    constexpr int PH = (128 / FR) < kUK3 ? (128 / FR) : kUK3;  // 27, 14, 7, 4 for C -> C = 32, 64, 96, 128
    constexpr int64_t rows_wg = (int64_t)NW * RB * 16;
    // a multiple of 8 workgroups: the kernel spreads the live tiles over the 8 XCDs
    const unsigned grid = (unsigned)(((p.m_cap + rows_wg - 1) / rows_wg + 7) / 8 * 8);
    k_conv_union<DT, KCH, NB, RB, NW, PH><<<grid, 64 * NW, 0, s>>>(
        p.nbr, p.m_out_dev, p.m_cap, (const uint16_t*)in, 32 * KCH, in_rows, (const uint4*)wpack, scale, shift, relu,
        (const uint16_t*)p.res, (uint16_t*)out);
}

template <int DT, int KCH>
static void launch_union_cin(hipStream_t s, const ConvPlan& p, const void* in, int Cout, int64_t in_rows,
                             const void* wpack, const float* scale, const float* shift, int relu, void* out) {
    switch (Cout) {
        case 32: launch_union_c<DT, KCH, 2>(s, p, in, in_rows, wpack, scale, shift, relu, out); break;
        case 64: launch_union_c<DT, KCH, 4>(s, p, in, in_rows, wpack, scale, shift, relu, out); break;
        case 96: launch_union_c<DT, KCH, 6>(s, p, in, in_rows, wpack, scale, shift, relu, out); break;
        case 128: launch_union_c<DT, KCH, 8>(s, p, in, in_rows, wpack, scale, shift, relu, out); break;
        case 256: launch_union_c<DT, KCH, 16>(s, p, in, in_rows, wpack, scale, shift, relu, out); break;
    }
}

template <int DT>
static void launch_union(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int Cout, int64_t in_rows,
                         const void* wpack, const float* scale, const float* shift, int relu, void* out) {
    switch (Cin) {
        case 32: launch_union_cin<DT, 1>(s, p, in, Cout, in_rows, wpack, scale, shift, relu, out); break;
        case 64: launch_union_cin<DT, 2>(s, p, in, Cout, in_rows, wpack, scale, shift, relu, out); break;
        case 96: launch_union_cin<DT, 3>(s, p, in, Cout, in_rows, wpack, scale, shift, relu, out); break;
        case 128: launch_union_cin<DT, 4>(s, p, in, Cout, in_rows, wpack, scale, shift, relu, out); break;
        case 256: launch_union_cin<DT, 8>(s, p, in, Cout, in_rows, wpack, scale, shift, relu, out); break;
    }
}

void launch_conv_union(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, int Cout,
                       const void* wpack, const float* scale, const float* shift, int relu, void* out, int dt) {
    if (dt == SPV_BF16) launch_union<SPV_BF16>(s, p, in, Cin, Cout, in_rows, wpack, scale, shift, relu, out);
    else launch_union<SPV_F16>(s, p, in, Cin, Cout, in_rows, wpack, scale, shift, relu, out);
}

}  // namespace spv
