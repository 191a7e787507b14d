// linear.hip -- pointwise linear layer on feature rows:
//   out[i] = act(scale * (in[i] @ W) + shift + res[i])      (res before act)
//   out[i] = act(scale * (in[i] @ W) + shift) + res[i]      (res after act)
// The point branch's MLP followed by the fusion by addition (Sec. 3.3 "Point
// Transformation and Feature Fusion") is the second form with res = the
// devoxelized voxel features; the 1x1 shortcut of a residual block is the first;
// a classifier is shift = bias, no activation.
//
// MFMA path (bf16/f16, C_in % 8 == 0, ceil(C_out / 16) in {1, 2, 4, 6, 8, 16};
// a C_out that is not a multiple of 16 -- a classifier's -- computes zero
// columns up to the next multiple and stores only the real ones):
// the packed W (the conv's operand fragments, one offset) and scale / shift are
// staged in LDS once per workgroup; each wave then takes blocks of 16 rows in
// turn (grid-stride), multiplies them on v_mfma_f32_16x16x32 with W^T as the A
// operand and the rows as B, and writes each row's channels once from the
// accumulators.  Other shapes and fp32 run on a vector-ALU kernel.
#include "conv_common.hpp"

namespace spv {

constexpr int kLinWaves = 4;

template <int DT, int KCH, int NB, bool RAGGED>
__global__ __launch_bounds__(64 * kLinWaves) void k_linear_mfma(
    const uint16_t* __restrict__ in, int Cin, const int64_t* __restrict__ m_dev, int64_t m_cap,
    const uint4* __restrict__ wpack, const float* __restrict__ scale, const float* __restrict__ shift, int relu,
    const uint16_t* __restrict__ res, int res_after, uint16_t* __restrict__ out, int Cout) {
    constexpr int C = NB * 16;
    constexpr int FR = KCH * NB;
    __shared__ __align__(16) uint4 wl[FR * 64];
    __shared__ float ssc[C], ssh[C];
    for (int f = threadIdx.x; f < FR * 64; f += blockDim.x) wl[f] = wpack[f];
    for (int c = threadIdx.x; c < C; c += blockDim.x) {
        ssc[c] = (scale && c < Cout) ? scale[c] : 1.f;
        ssh[c] = (shift && c < Cout) ? shift[c] : 0.f;
    }
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r16 = lane & 15, g = lane >> 4;
    const int64_t m = clamp_rows(m_dev, m_cap);
    const int64_t nblk = (m + 15) / 16;
    // the loop bound and the block index are wave-uniform: every MFMA runs with
    // the whole wave
    for (int64_t blk = (int64_t)blockIdx.x * kLinWaves + wave; blk < nblk; blk += (int64_t)gridDim.x * kLinWaves) {
        const int64_t row = blk * 16 + r16;
        const bool live = row < m;
        // B operand: lane (r16, g) holds channels kc*32 + 8g .. +7 of row r16
        i32x4 xv[KCH];
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc) {
            const int c0 = kc * 32 + 8 * g;
            xv[kc] = (live && c0 < Cin) ? *(const i32x4*)(in + row * Cin + c0) : i32x4{0, 0, 0, 0};
        }
        f32x4 acc[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[nb] = mfma16x16x32<DT>(wl[(kc * NB + nb) * 64 + lane], __builtin_bit_cast(uint4, xv[kc]), acc[nb]);
        if (!live) continue;
        // lane (r16, g) holds output channels nb*16 + 4g .. 4g+3 of row r16
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int c = nb * 16 + 4 * g;
            float rv[4] = {0.f, 0.f, 0.f, 0.f};
            if (res) {
                if constexpr (RAGGED) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (c + e < Cout) rv[e] = from16<DT>(res[row * Cout + c + e]);
                } else {
                    const uint2 u = *(const uint2*)(res + row * C + c);
                    rv[0] = from16<DT>(u.x & 0xFFFF);
                    rv[1] = from16<DT>(u.x >> 16);
                    rv[2] = from16<DT>(u.y & 0xFFFF);
                    rv[3] = from16<DT>(u.y >> 16);
                }
            }
            float y[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                y[e] = acc[nb][e] * ssc[c + e] + ssh[c + e];
                if (!res_after) y[e] += rv[e];
                if (relu) y[e] = fmaxf(y[e], 0.f);
                if (res_after) y[e] += rv[e];
            }
            if constexpr (RAGGED) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (c + e < Cout) out[row * Cout + c + e] = to16<DT>(y[e]);
            } else {
                const uint32_t lo = (uint32_t)to16<DT>(y[0]) | ((uint32_t)to16<DT>(y[1]) << 16);
                const uint32_t hi = (uint32_t)to16<DT>(y[2]) | ((uint32_t)to16<DT>(y[3]) << 16);
                *(uint2*)(out + row * C + c) = make_uint2(lo, hi);
            }
        }
    }
}

// one thread per output element, grid-stride; W[ci][co] at W[ci * ldw + co]
template <int DT>
__global__ __launch_bounds__(256) void k_linear_valu(const void* __restrict__ in, int Cin,
                                                     const int64_t* __restrict__ m_dev, int64_t m_cap,
                                                     const void* __restrict__ W, int ldc, int ldcol,
                                                     const float* __restrict__ scale, const float* __restrict__ shift,
                                                     int relu, const void* __restrict__ res, int res_after,
                                                     void* __restrict__ out, int Cout) {
    const int64_t m = clamp_rows(m_dev, m_cap);
    const int64_t total = m * Cout;
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = t / Cout;
        const int co = (int)(t - i * Cout);
        float s = 0.f;
        for (int ci = 0; ci < Cin; ++ci)
            s += ld_feat<DT>(in, i * Cin + ci) * ld_feat<DT>(W, (int64_t)ci * ldc + (int64_t)co * ldcol);
        float y = s * (scale ? scale[co] : 1.f) + (shift ? shift[co] : 0.f);
        const float r = res ? ld_feat<DT>(res, t) : 0.f;
        if (!res_after) y += r;
        if (relu) y = fmaxf(y, 0.f);
        if (res_after) y += r;
        st_feat<DT>(out, t, y);
    }
}

static int linear_kch(int Cin) { return (Cin + 31) / 32; }

bool linear_mfma_supported(int Cin, int Cout, int dt) {
    if (dt == SPV_F32 || Cin % 8 != 0) return false;
    const int KCH = linear_kch(Cin), NB = (Cout + 15) / 16;
    const bool kch_ok = KCH == 1 || KCH == 2 || KCH == 3 || KCH == 4 || KCH == 8;
    const bool nb_ok = NB == 1 || NB == 2 || NB == 4 || NB == 6 || NB == 8 || NB == 16;
    // ragged widths (not a multiple of 16) are built for classifier sizes only
    return kch_ok && nb_ok && (Cout % 16 == 0 || NB <= 2);
}

void* plan_linear_ws(Arena& a, int Cin, int Cout) {
    const int KCH = linear_kch(Cin) < 1 ? 1 : linear_kch(Cin), NB = (Cout + 15) / 16 < 1 ? 1 : (Cout + 15) / 16;
    return a.take<uint4>((size_t)KCH * NB * 64);
}

template <int DT, int KCH, int NB>
static void launch_lin(hipStream_t s, const LinearArgs& a, const void* wpack) {
    const int64_t blocks16 = (a.m_cap + 15) / 16;
    int64_t grid = (blocks16 + kLinWaves - 1) / kLinWaves;
    if (grid > 1024) grid = 1024;
    if (grid < 1) grid = 1;
    if (a.Cout == NB * 16)
        k_linear_mfma<DT, KCH, NB, false><<<(unsigned)grid, 64 * kLinWaves, 0, s>>>(
            (const uint16_t*)a.in, a.Cin, a.m_dev, a.m_cap, (const uint4*)wpack, a.scale, a.shift, a.relu,
            (const uint16_t*)a.res, a.res_after, (uint16_t*)a.out, a.Cout);
    else if constexpr (NB <= 2)
        k_linear_mfma<DT, KCH, NB, true><<<(unsigned)grid, 64 * kLinWaves, 0, s>>>(
            (const uint16_t*)a.in, a.Cin, a.m_dev, a.m_cap, (const uint4*)wpack, a.scale, a.shift, a.relu,
            (const uint16_t*)a.res, a.res_after, (uint16_t*)a.out, a.Cout);
}

template <int DT, int KCH>
static void launch_lin_nb(hipStream_t s, const LinearArgs& a, const void* wpack) {
    switch ((a.Cout + 15) / 16) {
        case 1: launch_lin<DT, KCH, 1>(s, a, wpack); break;
        case 2: launch_lin<DT, KCH, 2>(s, a, wpack); break;
        case 4: launch_lin<DT, KCH, 4>(s, a, wpack); break;
        case 6: launch_lin<DT, KCH, 6>(s, a, wpack); break;
        case 8: launch_lin<DT, KCH, 8>(s, a, wpack); break;
        case 16: launch_lin<DT, KCH, 16>(s, a, wpack); break;
    }
}

template <int DT>
static void launch_lin_dt(hipStream_t s, const LinearArgs& a, const void* wpack) {
    switch (linear_kch(a.Cin)) {
        case 1: launch_lin_nb<DT, 1>(s, a, wpack); break;
        case 2: launch_lin_nb<DT, 2>(s, a, wpack); break;
        case 3: launch_lin_nb<DT, 3>(s, a, wpack); break;
        case 4: launch_lin_nb<DT, 4>(s, a, wpack); break;
        case 8: launch_lin_nb<DT, 8>(s, a, wpack); break;
    }
}

void launch_linear(hipStream_t s, const LinearArgs& a, void* wpack, bool prepacked) {
    if (a.m_cap <= 0) return;
    if (linear_mfma_supported(a.Cin, a.Cout, a.dt)) {
        const int KCH = linear_kch(a.Cin), NB = (a.Cout + 15) / 16;
        PackJob q{(const uint16_t*)a.W, (uint4*)wpack, 1, a.Cin, a.Cout, KCH, NB, (int64_t)KCH * NB * 64,
                  a.wt ? 1 : a.ldw, (int64_t)a.Cin * a.ldw, a.wt ? a.ldw : 1};
        if (!prepacked) launch_pack_job(s, q);
        if (a.dt == SPV_BF16) launch_lin_dt<SPV_BF16>(s, a, wpack);
        else launch_lin_dt<SPV_F16>(s, a, wpack);
        return;
    }
    const int ldc = a.wt ? 1 : a.ldw, ldcol = a.wt ? a.ldw : 1;
    int64_t grid = (a.m_cap * a.Cout + 255) / 256;
    if (grid > 4096) grid = 4096;
    if (grid < 1) grid = 1;
    if (a.dt == SPV_F32)
        k_linear_valu<SPV_F32><<<(unsigned)grid, 256, 0, s>>>(a.in, a.Cin, a.m_dev, a.m_cap, a.W, ldc, ldcol, a.scale,
                                                              a.shift, a.relu, a.res, a.res_after, a.out, a.Cout);
    else if (a.dt == SPV_BF16)
        k_linear_valu<SPV_BF16><<<(unsigned)grid, 256, 0, s>>>(a.in, a.Cin, a.m_dev, a.m_cap, a.W, ldc, ldcol, a.scale,
                                                               a.shift, a.relu, a.res, a.res_after, a.out, a.Cout);
    else
        k_linear_valu<SPV_F16><<<(unsigned)grid, 256, 0, s>>>(a.in, a.Cin, a.m_dev, a.m_cap, a.W, ldc, ldcol, a.scale,
                                                              a.shift, a.relu, a.res, a.res_after, a.out, a.Cout);
}

}  // namespace spv
