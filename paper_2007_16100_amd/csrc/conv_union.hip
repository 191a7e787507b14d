// conv_union.hip -- sparse convolution on a 3x3x3 kernel map (Sec. 3.2 / 3.3)
// with register accumulators: the neighbour-table kernel described in conv.hip.
#include "conv_common.hpp"

namespace spv {

// ---------------------------------------------------------------------------
// neighbour-table kernel (3x3x3 maps)
// ---------------------------------------------------------------------------
// Workgroup = 4 waves; wave w owns RB blocks of 16 output rows and all output
// channels (NB blocks of 16).  The accumulators of a block are D = W^T G^T
// fragments: lane (r16, g) holds output channels nb*16 + 4g .. 4g+3 of row r16,
// which is also the order in which they are stored.
//
// Step k of the (fully unrolled) offset loop:
//   wait for the wave's own copies of W[k] and for the barrier (every wave has
//   copied its share), read the W[k] fragments from LDS buffer k % 3, then
//   issue the copies of W[k+2] into buffer (k+2) % 3, the neighbour indices of
//   offset k+2 and the gathered rows of offset k+1, and finally multiply the
//   rows of offset k.  Every load thus has one or two steps of matrix work to
//   arrive in, and the compiler's own waits stay exact because every load it
//   waits for is one it issued (the LDS copies use the compiler's builtin).
constexpr int kUnionWaves = 4;

template <int DT, int KCH, int NB, int RB, int FULL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_conv_union(
    const int32_t* __restrict__ nbr, const int64_t* __restrict__ m_out_dev, int64_t m_cap,
    const uint16_t* __restrict__ in, int Cin, int64_t in_rows, const uint4* __restrict__ wpack,
    const float* __restrict__ scale, const float* __restrict__ shift, int relu, uint16_t* __restrict__ out) {
    constexpr int K3 = 27;
    constexpr int FR = KCH * NB;  // 1 KB weight fragments per offset
    constexpr int Cout = NB * 16;
    __shared__ __align__(16) uint4 wbuf[3][FR * 64];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r16 = lane & 15, g = lane >> 4;

    // workgroups of one XCD take consecutive row ranges (round-robin dispatch over 8 XCDs)
    const int64_t G = gridDim.x, bid = blockIdx.x;
    const int64_t xq = G / 8, xr = G % 8, x = bid % 8;
    const int64_t wg = x * xq + (x < xr ? x : xr) + bid / 8;

    const int64_t m = clamp_rows(m_out_dev, m_cap);
    if (wg * (kUnionWaves * RB * 16) >= m) return;  // the whole workgroup
    const int64_t blk0 = (wg * kUnionWaves + wave) * RB;

    const __amdgpu_buffer_rsrc_t nb_rs = make_rsrc(nbr, (uint32_t)(m * K3 * 4));
    const uint32_t row_bytes = (uint32_t)Cin * 2u;
    const __amdgpu_buffer_rsrc_t in_rs = make_rsrc(in, (uint32_t)(in_rows * (int64_t)row_bytes));
    const uint32_t in_rows32 = (uint32_t)in_rows;
    const int qin = Cin / 8;

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

    // this wave's share of the weight copies: fragments wave, wave + 4, ...
    auto copy_w = [&](int k, int buf) {
#pragma unroll
        for (int f = 0; f < FR; f += kUnionWaves) {
            if (f + wave < FR)
                __builtin_amdgcn_global_load_lds(
                    (const void*)(wpack + ((int64_t)k * FR + f + wave) * 64 + lane),
                    (__attribute__((address_space(3))) void*)&wbuf[buf][(f + wave) * 64], 16, 0, 0);
        }
    };
    auto load_nbr = [&](int k, int (&dst)[RB]) {
#pragma unroll
        for (int b = 0; b < RB; ++b)
            dst[b] = __builtin_amdgcn_raw_buffer_load_b32(nb_rs, nboff[b] + (uint32_t)k * 4u, 0, 0);
    };
    auto load_rows = [&](const int (&nb1)[RB], i32x4 (&dst)[RB][KCH]) {
#pragma unroll
        for (int b = 0; b < RB; ++b) {
            const uint32_t i = (uint32_t)(nb1[b] - 1);  // stored as row + 1; 0 = absent
            const uint32_t base = i < in_rows32 ? i * row_bytes + (uint32_t)g * 16u : kOutOfRange;
#pragma unroll
            for (int kc = 0; kc < KCH; ++kc) {
                uint32_t o = base + kc * 64;
                if (!FULL && kc * 4 + g >= qin) o = kOutOfRange;
                dst[b][kc] = __builtin_amdgcn_raw_buffer_load_b128(in_rs, o, 0, 0);
            }
        }
    };

    f32x4 acc[RB][NB];
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[b][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    int ns[3][RB];        // neighbour indices of offsets k, k+1, k+2 (slot k % 3)
    i32x4 rs[2][RB][KCH]; // gathered rows of offsets k, k+1 (slot k % 2)
    copy_w(0, 0);
    copy_w(1, 1);
    load_nbr(0, ns[0]);
    load_nbr(1, ns[1]);
    load_rows(ns[0], rs[0]);

#pragma unroll
    for (int k = 0; k < K3; ++k) {
        // every wave's copies of W[k] have landed: at most the loads of the last
        // step's neighbour indices and rows may still be outstanding
        vm_wait<RB + KCH * RB>();
        __syncthreads();
        uint4 wf[KCH][NB];
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) wf[kc][nb] = wbuf[k % 3][(kc * NB + nb) * 64 + lane];
        asm volatile("" ::: "memory");  // the copies below stay after these reads
        if (k + 2 < K3) {
            copy_w(k + 2, (k + 2) % 3);
            load_nbr(k + 2, ns[(k + 2) % 3]);
        }
        if (k + 1 < K3) load_rows(ns[(k + 1) % 3], rs[(k + 1) % 2]);
#pragma unroll
        for (int b = 0; b < RB; ++b) {
            if ((umask[b] >> k) & 1u) {
#pragma unroll
                for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
                        acc[b][nb] = mfma16x16x32<DT>(wf[kc][nb], __builtin_bit_cast(uint4, rs[k % 2][b][kc]),
                                                      acc[b][nb]);
            }
        }
    }

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
            float y[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                y[e] = acc[b][nb][e] * sc[nb][e] + sh[nb][e];
                if (relu) y[e] = fmaxf(y[e], 0.f);
            }
            const uint32_t lo = (uint32_t)to16<DT>(y[0]) | ((uint32_t)to16<DT>(y[1]) << 16);
            const uint32_t hi = (uint32_t)to16<DT>(y[2]) | ((uint32_t)to16<DT>(y[3]) << 16);
            *(uint2*)(out + row * Cout + nb * 16 + 4 * g) = make_uint2(lo, hi);
        }
    }
}

// blocks of 16 rows per wave of the neighbour-table kernel: accumulators
// (RB*NB), weight fragments (KCH*NB) and two stages of gathered rows
// (2*RB*KCH), in 16-byte registers, within ~56 of them (two waves per SIMD)
constexpr int union_rb(int KCH, int NB) {
    for (int rb = 4; rb > 1; --rb)
        if (rb * NB + KCH * NB + 2 * rb * KCH <= 56) return rb;
    return 1;
}

bool union_supported(int K3, int Cin, int Cout, int dt) {
    if (K3 != 27 || dt == SPV_F32 || Cin % 8 != 0 || Cout % 16 != 0 || Cin > 128) return false;
    const int NB = Cout / 16, KCH = (Cin + 31) / 32;
    if (!(NB == 1 || NB == 2 || NB == 4 || NB == 6 || NB == 8)) return false;
    return KCH * NB <= 24 && KCH * NB + NB + 2 * KCH <= 56;
}

template <int DT, int KCH, int NB, int FULL>
static void launch_union3(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows,
                          const void* wpack, const float* scale, const float* shift, int relu, void* out) {
    constexpr int RB = union_rb(KCH, NB);
    constexpr int64_t rows_wg = (int64_t)kUnionWaves * RB * 16;
    const unsigned grid = (unsigned)((p.m_cap + rows_wg - 1) / rows_wg);
    k_conv_union<DT, KCH, NB, RB, FULL><<<grid, 64 * kUnionWaves, 0, s>>>(
        p.nbr, p.m_out_dev, p.m_cap, (const uint16_t*)in, Cin, in_rows, (const uint4*)wpack, scale, shift, relu,
        (uint16_t*)out);
}

template <int DT, int KCH, int NB>
static void launch_union_nb(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows,
                            const void* wpack, const float* scale, const float* shift, int relu, void* out) {
    if (Cin == KCH * 32) launch_union3<DT, KCH, NB, 1>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out);
    else launch_union3<DT, KCH, NB, 0>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out);
}

template <int DT, int KCH>
static void launch_union_kch(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, int Cout,
                             const void* wpack, const float* scale, const float* shift, int relu, void* out) {
    switch (Cout / 16) {
#define SPV_NB_CASE(N)                                                                             \
    case N:                                                                                        \
        if constexpr (KCH * N <= 24 && KCH * N + N + 2 * KCH <= 56)                                \
            launch_union_nb<DT, KCH, N>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out);  \
        break;
        SPV_NB_CASE(1)
        SPV_NB_CASE(2)
        SPV_NB_CASE(4)
        SPV_NB_CASE(6)
        SPV_NB_CASE(8)
#undef SPV_NB_CASE
    }
}

template <int DT>
static void launch_union(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, int Cout,
                         const void* wpack, const float* scale, const float* shift, int relu, void* out) {
    switch ((Cin + 31) / 32) {
        case 1: launch_union_kch<DT, 1>(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out); break;
        case 2: launch_union_kch<DT, 2>(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out); break;
        case 3: launch_union_kch<DT, 3>(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out); break;
        case 4: launch_union_kch<DT, 4>(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out); break;
    }
}

void launch_conv_union(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, int Cout,
                       const void* wpack, const float* scale, const float* shift, int relu, void* out, int dt) {
    if (dt == SPV_BF16) launch_union<SPV_BF16>(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out);
    else launch_union<SPV_F16>(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out);
}

}  // namespace spv
