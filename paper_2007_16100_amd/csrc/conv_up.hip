// conv_up.hip -- the transposed k=2 s=2 sparse convolution (the decoder's
// upsampling, Sec. 3.2) as an output-scattered GEMM.
//
// On a stride-2 map every fine voxel has exactly one parent: fine voxel i with
// parent j at offset k receives in[j] @ W[k] and nothing else.  So instead of
// gathering, per output, the inputs of its pairs, the kernel walks the coarse
// rows: a wave loads the rows of 16 coarse voxels once (the B operand of
// v_mfma_f32_16x16x32), and for each of the 8 offsets at which any of the 16
// has a child it multiplies them by W[k] (A operand, staged in LDS for a phase
// of offsets per workgroup) and writes each product row, finished by
// act(scale * . + shift + res), straight to its child's row.  Every output row
// is written once, by one lane group; nothing accumulates across pairs.
// children[j][k] = i + 1 (0 = none) is the stride-2 map's neighbour table.
#include "conv_common.hpp"

namespace spv {

constexpr int kUpK = 8;
constexpr int kUpWaves = 8;

template <int DT, int KCH, int NB, int PH>
__global__ __launch_bounds__(64 * kUpWaves) void k_conv_up(
    const int32_t* __restrict__ children, const int64_t* __restrict__ m_dev, int64_t m_cap,
    const uint16_t* __restrict__ in, int Cin, const uint4* __restrict__ wpack, const float* __restrict__ scale,
    const float* __restrict__ shift, int relu, const uint16_t* __restrict__ res, uint16_t* __restrict__ out,
    int64_t out_rows) {
    constexpr int FR = KCH * NB;  // 1 KB weight fragments per offset
    constexpr int Cout = NB * 16;
    __shared__ __align__(16) uint4 wl[PH * FR * 64];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r16 = lane & 15, g = lane >> 4;
    const int64_t m = clamp_rows(m_dev, m_cap);
    const int64_t row0 = (int64_t)blockIdx.x * kUpWaves * 16;
    if (row0 >= m) return;  // the whole workgroup
    const int64_t row = row0 + wave * 16 + r16;
    const bool live = row < m;

    // B operand: lane (r16, g) holds channels kc*32 + 8g .. +7 of coarse row r16
    i32x4 xv[KCH];
#pragma unroll
    for (int kc = 0; kc < KCH; ++kc) {
        const int c0 = kc * 32 + 8 * g;
        xv[kc] = (live && c0 < Cin) ? *(const i32x4*)(in + row * Cin + c0) : i32x4{0, 0, 0, 0};
    }
    int32_t ch[kUpK];
    uint32_t present = 0;  // offsets at which some row of the wave's block has a child (wave-uniform)
#pragma unroll
    for (int k = 0; k < kUpK; ++k) {
        const int32_t c = live ? children[row * kUpK + k] : 0;
        ch[k] = (c > 0 && (int64_t)c <= out_rows) ? c : 0;
        present |= (__ballot(ch[k] > 0) ? 1u : 0u) << k;
    }
    const i32x4* wsrc = (const i32x4*)wpack;
#pragma unroll
    for (int k0 = 0; k0 < kUpK; k0 += PH) {
        // the phase's weights into LDS (global->LDS copies, one wait, barriers around)
        const int nk = (kUpK - k0) < PH ? (kUpK - k0) : PH;
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        const uint64_t gw = (uint64_t)(wsrc + (int64_t)k0 * FR * 64);
        for (int f = wave; f < nk * FR; f += kUpWaves)
            lds_dma_x4(gw + (uint64_t)f * 1024u, (uint32_t)lane * 16u, lds_addr(wl + f * 64));
        vm_wait<0>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
#pragma unroll
        for (int kk = 0; kk < PH; ++kk) {
            const int k = k0 + kk;
            if (k >= kUpK || !((present >> k) & 1u)) continue;  // wave-uniform
            f32x4 acc[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
            const i32x4* wk = (const i32x4*)wl + kk * FR * 64;
#pragma unroll
            for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    acc[nb] = mfma16x16x32<DT>(__builtin_bit_cast(uint4, wk[(kc * NB + nb) * 64 + lane]),
                                               __builtin_bit_cast(uint4, xv[kc]), acc[nb]);
            if (ch[k] == 0) continue;
            // lane (r16, g) holds output channels nb*16 + 4g .. 4g+3 of coarse row r16's child
            const int64_t orow = (int64_t)ch[k] - 1;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const int c = nb * 16 + 4 * g;
                float rv[4] = {0.f, 0.f, 0.f, 0.f};
                if (res) {
                    const uint2 u = *(const uint2*)(res + orow * Cout + c);
                    rv[0] = from16<DT>(u.x & 0xFFFF);
                    rv[1] = from16<DT>(u.x >> 16);
                    rv[2] = from16<DT>(u.y & 0xFFFF);
                    rv[3] = from16<DT>(u.y >> 16);
                }
                float y[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    y[e] = acc[nb][e] * (scale ? scale[c + e] : 1.f) + (shift ? shift[c + e] : 0.f) + rv[e];
                    if (relu) y[e] = fmaxf(y[e], 0.f);
                }
                const uint32_t lo = (uint32_t)to16<DT>(y[0]) | ((uint32_t)to16<DT>(y[1]) << 16);
                const uint32_t hi = (uint32_t)to16<DT>(y[2]) | ((uint32_t)to16<DT>(y[3]) << 16);
                *(uint2*)(out + orow * Cout + c) = make_uint2(lo, hi);
            }
        }
    }
}

bool up_supported(int Cin, int Cout, int dt) {
    if (dt == SPV_F32) return false;
    const auto width_ok = [](int c) { return c == 32 || c == 64 || c == 96 || c == 128 || c == 256; };
    return width_ok(Cin) && width_ok(Cout);
}

template <int DT, int KCH, int NB>
static void launch_up_c(hipStream_t s, const UpArgs& a, const void* wpack) {
    constexpr int FR = KCH * NB;
    constexpr int PH = (128 / FR) < kUpK ? (128 / FR) : kUpK;  // offsets per 128 KB LDS phase
    const int64_t rows_wg = (int64_t)kUpWaves * 16;
    const unsigned grid = (unsigned)((a.m_cap + rows_wg - 1) / rows_wg);
    k_conv_up<DT, KCH, NB, PH><<<grid > 0 ? grid : 1, 64 * kUpWaves, 0, s>>>(
        a.children, a.m_dev, a.m_cap, (const uint16_t*)a.in, a.Cin, (const uint4*)wpack, a.scale, a.shift, a.relu,
        (const uint16_t*)a.res, (uint16_t*)a.out, a.out_rows);
}

template <int DT, int KCH>
static void launch_up_cin(hipStream_t s, const UpArgs& a, const void* wpack) {
    switch (a.Cout) {
        case 32: launch_up_c<DT, KCH, 2>(s, a, wpack); break;
        case 64: launch_up_c<DT, KCH, 4>(s, a, wpack); break;
        case 96: launch_up_c<DT, KCH, 6>(s, a, wpack); break;
        case 128: launch_up_c<DT, KCH, 8>(s, a, wpack); break;
        case 256: launch_up_c<DT, KCH, 16>(s, a, wpack); break;
    }
}

template <int DT>
static void launch_up_dt(hipStream_t s, const UpArgs& a, const void* wpack) {
    switch (a.Cin) {
        case 32: launch_up_cin<DT, 1>(s, a, wpack); break;
        case 64: launch_up_cin<DT, 2>(s, a, wpack); break;
        case 96: launch_up_cin<DT, 3>(s, a, wpack); break;
        case 128: launch_up_cin<DT, 4>(s, a, wpack); break;
        case 256: launch_up_cin<DT, 8>(s, a, wpack); break;
    }
}

void launch_conv_up(hipStream_t s, const UpArgs& a, const void* wpack) {
    if (a.m_cap <= 0) return;
    if (a.dt == SPV_BF16) launch_up_dt<SPV_BF16>(s, a, wpack);
    else launch_up_dt<SPV_F16>(s, a, wpack);
}

}  // namespace spv
