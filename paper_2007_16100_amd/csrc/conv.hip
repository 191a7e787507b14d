// conv.hip -- sparse convolution on a kernel map (Sec. 3.2 / 3.3):
//   out[j] = act(scale * sum_{(i, j, k)} in[i] @ W[k] + shift)
//
// Output-stationary gather-GEMM on matrix cores.  Output rows are taken in
// blocks of 16 (one MFMA M-tile); a plan built from the kernel map records, per
// block, the union of the offsets its rows use and, per (block, offset, row),
// the input row.  A wave owns R blocks x all output channels in registers
// (fp32 accumulators) and walks the offsets of its blocks: for each offset the
// packed weight slice W[k] is loaded once into registers and reused by every
// block that has the offset, the A operand is gathered straight from the
// input feature rows (16 bytes per lane, absent rows masked to zero), and
// v_mfma_f32_16x16x32_{bf16,f16} accumulates.  The epilogue applies the
// per-channel scale/shift and ReLU and writes each output row exactly once:
// no atomics, deterministic results.
#include "spv_internal.hpp"

namespace spv {

constexpr int kRowsPerTile = 16;

void plan_conv_ws(Arena& a, ConvPlan& p, int64_t m_out_cap, int K3) {
    p.m_cap = m_out_cap > 0 ? m_out_cap : 1;
    p.K3 = K3;
    int64_t nb = (p.m_cap + kRowsPerTile - 1) / kRowsPerTile;
    p.mask = a.take<uint32_t>(p.m_cap);
    p.umask = a.take<uint32_t>(nb);
    p.ucnt = a.take<uint32_t>(nb + 1);
    p.table = a.take<int32_t>((size_t)K3 * nb * kRowsPerTile);
}

__device__ inline int64_t clamp_rows(const int64_t* d, int64_t cap) {
    if (!d) return cap;
    int64_t c = *d;
    return c < 0 ? 0 : (c > cap ? cap : c);
}

__global__ void k_plan_zero(uint32_t* mask, int64_t cap) {
    int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (j < cap) mask[j] = 0;
}

// the offset k of pair p (off is non-decreasing)
__device__ inline int pair_offset(const int32_t* soff, int K3, int64_t p) {
    int k = 0;
    while (k + 1 < K3 && p >= soff[k + 1]) ++k;
    return k;
}

__global__ void k_plan_mask(const int32_t* off, const int32_t* pairs, int K3, int transposed, int64_t pair_bound,
                            const int64_t* m_out_dev, int64_t cap, uint32_t* mask) {
    __shared__ int32_t soff[28];
    if (threadIdx.x <= K3) soff[threadIdx.x] = off[threadIdx.x];
    __syncthreads();
    int64_t total = soff[K3];
    if (total > pair_bound) total = pair_bound;
    int64_t m = clamp_rows(m_out_dev, cap);
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < total; p += (int64_t)gridDim.x * blockDim.x) {
        int k = pair_offset(soff, K3, p);
        int64_t j = transposed ? pairs[2 * p] : pairs[2 * p + 1];
        if (j >= 0 && j < m) atomicOr(&mask[j], 1u << k);
    }
}

__global__ void k_plan_union(const uint32_t* mask, const int64_t* m_out_dev, int64_t cap, int64_t nblk,
                             uint32_t* umask, uint32_t* ucnt) {
    int64_t b = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (b >= nblk) return;
    int64_t m = clamp_rows(m_out_dev, cap);
    uint32_t u = 0;
    for (int r = 0; r < kRowsPerTile; ++r) {
        int64_t j = b * kRowsPerTile + r;
        if (j < m) u |= mask[j];
    }
    umask[b] = u;
    ucnt[b] = (uint32_t)__popc(u);
}

__global__ void k_plan_scatter(const int32_t* off, const int32_t* pairs, int K3, int transposed, int64_t pair_bound,
                               const int64_t* m_out_dev, int64_t cap, const uint32_t* umask, const uint32_t* ucnt,
                               int32_t* table) {
    __shared__ int32_t soff[28];
    if (threadIdx.x <= K3) soff[threadIdx.x] = off[threadIdx.x];
    __syncthreads();
    int64_t total = soff[K3];
    if (total > pair_bound) total = pair_bound;
    int64_t m = clamp_rows(m_out_dev, cap);
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < total; p += (int64_t)gridDim.x * blockDim.x) {
        int k = pair_offset(soff, K3, p);
        int64_t i = transposed ? pairs[2 * p + 1] : pairs[2 * p];
        int64_t j = transposed ? pairs[2 * p] : pairs[2 * p + 1];
        if (j < 0 || j >= m) continue;
        int64_t b = j / kRowsPerTile;
        uint32_t u = umask[b];
        uint32_t slot = (uint32_t)__popc(u & ((1u << k) - 1u));
        table[((int64_t)ucnt[b] + slot) * kRowsPerTile + (j % kRowsPerTile)] = (int32_t)i;
    }
}

void launch_conv_plan(hipStream_t s, const ConvPlan& p, const int32_t* off, const int32_t* pairs, int K3,
                      int transposed, int64_t pair_bound) {
    int64_t nblk = (p.m_cap + kRowsPerTile - 1) / kRowsPerTile;
    unsigned gp = blocks_for(pair_bound, 256);
    if (gp > 4096) gp = 4096;
    k_plan_zero<<<blocks_for(p.m_cap, 256), 256, 0, s>>>(p.mask, p.m_cap);
    k_plan_mask<<<gp, 256, 0, s>>>(off, pairs, K3, transposed, pair_bound, p.m_out_dev, p.m_cap, p.mask);
    k_plan_union<<<blocks_for(nblk, 256), 256, 0, s>>>(p.mask, p.m_out_dev, p.m_cap, nblk, p.umask, p.ucnt);
    launch_exclusive_scan_small(s, p.ucnt, p.ucnt, nblk);
    k_plan_scatter<<<gp, 256, 0, s>>>(off, pairs, K3, transposed, pair_bound, p.m_out_dev, p.m_cap, p.umask, p.ucnt,
                                      p.table);
}

// ---------------------------------------------------------------------------
// weight packing into MFMA B-operand fragments:
// wpack[((k * KCH + kc) * NB + nb) * 64 + lane] = W[k][kc*32 + 8*(lane/16) + e][nb*16 + lane%16], e = 0..7
// ---------------------------------------------------------------------------
__global__ void k_pack_w(const uint16_t* W, int K3, int Cin, int Cout, int KCH, int NB, uint4* wpack) {
    int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t total = (int64_t)K3 * KCH * NB * 64;
    if (t >= total) return;
    int lane = (int)(t & 63);
    int64_t f = t >> 6;
    int nb = (int)(f % NB);
    f /= NB;
    int kc = (int)(f % KCH);
    int k = (int)(f / KCH);
    int col = nb * 16 + (lane & 15);
    int ci0 = kc * 32 + 8 * (lane >> 4);
    uint32_t w[4];
    for (int e = 0; e < 4; ++e) {
        uint32_t lo = 0, hi = 0;
        int c0 = ci0 + 2 * e, c1 = ci0 + 2 * e + 1;
        if (c0 < Cin) lo = W[((int64_t)k * Cin + c0) * Cout + col];
        if (c1 < Cin) hi = W[((int64_t)k * Cin + c1) * Cout + col];
        w[e] = lo | (hi << 16);
    }
    wpack[t] = make_uint4(w[0], w[1], w[2], w[3]);
}

void* plan_wpack_ws(Arena& a, int K3, int Cin, int Cout) {
    int KCH = (Cin + 31) / 32, NB = Cout / 16;
    return a.take<uint4>((size_t)K3 * KCH * NB * 64);
}

// ---------------------------------------------------------------------------
// MFMA conv
// ---------------------------------------------------------------------------
template <int DT, int KCH, int NB, int R>
__global__ __launch_bounds__(256) void k_conv_mfma(ConvPlan p, const uint16_t* __restrict__ in, int Cin, int64_t in_rows,
                                                   const uint4* __restrict__ wpack, const float* __restrict__ scale,
                                                   const float* __restrict__ shift, int relu,
                                                   uint16_t* __restrict__ out, int Cout) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, g = lane >> 4;
    const int64_t m = clamp_rows(p.m_out_dev, p.m_cap);
    const int64_t nblk = (m + kRowsPerTile - 1) / kRowsPerTile;
    const int64_t b0 = ((int64_t)blockIdx.x * 4 + wave) * R;
    if (b0 >= nblk) return;

    uint32_t U[R], base[R], mrow[R];
    uint32_t Uall = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        int64_t b = b0 + r;
        bool vb = b < nblk;
        U[r] = vb ? p.umask[b] : 0u;
        base[r] = vb ? p.ucnt[b] : 0u;
        int64_t row = b * kRowsPerTile + r16;
        mrow[r] = (vb && row < m) ? p.mask[row] : 0u;
        Uall |= U[r];
    }
    f32x4 acc[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[r][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    while (Uall) {
        const int k = __builtin_ctz(Uall);
        Uall &= Uall - 1;
        const uint16_t* src[R];
        bool has[R], ok[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            has[r] = (U[r] >> k) & 1u;
            int32_t i = -1;
            if (has[r] && ((mrow[r] >> k) & 1u)) {
                const uint32_t slot = (uint32_t)__popc(U[r] & ((1u << k) - 1u));
                i = p.table[((int64_t)base[r] + slot) * kRowsPerTile + r16];
            }
            ok[r] = i >= 0 && i < in_rows;
            src[r] = in + (int64_t)(ok[r] ? i : 0) * Cin + 8 * g;
        }
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc) {
            uint4 bf[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bf[nb] = wpack[((int64_t)(k * KCH + kc) * NB + nb) * 64 + lane];
            const bool chok = kc * 32 + 8 * g < Cin;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (!has[r]) continue;
                uint4 a = make_uint4(0, 0, 0, 0);
                if (ok[r] && chok) a = *(const uint4*)(src[r] + kc * 32);
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) acc[r][nb] = mfma16x16x32<DT>(a, bf[nb], acc[r][nb]);
            }
        }
    }
    // epilogue: lane holds rows 4g..4g+3 of each 16-row block, column nb*16 + r16
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int col = nb * 16 + r16;
        const float sc = scale ? scale[col] : 1.f;
        const float sh = shift ? shift[col] : 0.f;
#pragma unroll
        for (int r = 0; r < R; ++r) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t row = (b0 + r) * kRowsPerTile + 4 * g + e;
                if (row >= m) continue;
                float v = acc[r][nb][e] * sc + sh;
                if (relu) v = fmaxf(v, 0.f);
                out[row * Cout + col] = to16<DT>(v);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// vector-ALU conv (f32, or shapes the MFMA kernel does not take)
// ---------------------------------------------------------------------------
template <int DT>
__global__ void k_conv_generic(ConvPlan p, const void* in, int Cin, int64_t in_rows, const void* W, const float* scale,
                               const float* shift, int relu, void* out, int Cout) {
    const int64_t m = clamp_rows(p.m_out_dev, p.m_cap);
    int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t j = t / Cout;
    int co = (int)(t - j * Cout);
    if (j >= m) return;
    const int64_t b = j / kRowsPerTile;
    const uint32_t U = p.umask[b], base = p.ucnt[b];
    uint32_t bits = p.mask[j];
    float acc = 0.f;
    while (bits) {
        const int k = __builtin_ctz(bits);
        bits &= bits - 1;
        const uint32_t slot = (uint32_t)__popc(U & ((1u << k) - 1u));
        const int32_t i = p.table[((int64_t)base + slot) * kRowsPerTile + (j % kRowsPerTile)];
        if (i < 0 || i >= in_rows) continue;
        for (int ci = 0; ci < Cin; ++ci)
            acc += ld_feat<DT>(in, (int64_t)i * Cin + ci) * ld_feat<DT>(W, ((int64_t)k * Cin + ci) * Cout + co);
    }
    float v = acc * (scale ? scale[co] : 1.f) + (shift ? shift[co] : 0.f);
    if (relu) v = fmaxf(v, 0.f);
    st_feat<DT>(out, j * Cout + co, v);
}

bool conv_mfma_supported(int Cin, int Cout, int dt) {
    if (dt == SPV_F32 || Cin % 8 != 0 || Cout % 16 != 0) return false;
    int KCH = (Cin + 31) / 32, NB = Cout / 16;
    return KCH <= 8 && (NB == 1 || NB == 2 || NB == 4 || NB == 6 || NB == 8 || NB == 16);
}

template <int DT, int KCH, int NB>
static void launch_mfma_nb(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows,
                           const void* wpack, const float* scale, const float* shift, int relu, void* out, int Cout) {
    constexpr int R = (NB <= 2) ? 8 : (NB <= 6 ? 4 : (NB <= 8 ? 3 : 2));
    int64_t nblk = (p.m_cap + kRowsPerTile - 1) / kRowsPerTile;
    int64_t waves = (nblk + R - 1) / R;
    k_conv_mfma<DT, KCH, NB, R><<<blocks_for(waves, 4), 256, 0, s>>>(p, (const uint16_t*)in, Cin, in_rows,
                                                                   (const uint4*)wpack, scale, shift, relu,
                                                                   (uint16_t*)out, Cout);
}

template <int DT, int KCH>
static void launch_mfma_kch(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows,
                            const void* wpack, const float* scale, const float* shift, int relu, void* out, int Cout) {
    switch (Cout / 16) {
        case 1: launch_mfma_nb<DT, KCH, 1>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 2: launch_mfma_nb<DT, KCH, 2>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 4: launch_mfma_nb<DT, KCH, 4>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 6: launch_mfma_nb<DT, KCH, 6>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 8: launch_mfma_nb<DT, KCH, 8>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 16: launch_mfma_nb<DT, KCH, 16>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
    }
}

template <int DT>
static void launch_mfma(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, const void* wpack,
                        const float* scale, const float* shift, int relu, void* out, int Cout) {
    switch ((Cin + 31) / 32) {
        case 1: launch_mfma_kch<DT, 1>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 2: launch_mfma_kch<DT, 2>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 3: launch_mfma_kch<DT, 3>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 4: launch_mfma_kch<DT, 4>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 5: launch_mfma_kch<DT, 5>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 6: launch_mfma_kch<DT, 6>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 7: launch_mfma_kch<DT, 7>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
        case 8: launch_mfma_kch<DT, 8>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout); break;
    }
}

void launch_conv_pack(hipStream_t s, int K3, const void* W, void* wpack, int Cin, int Cout, int dt) {
    if (!conv_mfma_supported(Cin, Cout, dt)) return;
    int KCH = (Cin + 31) / 32, NB = Cout / 16;
    int64_t tot = (int64_t)K3 * KCH * NB * 64;
    k_pack_w<<<blocks_for(tot, 256), 256, 0, s>>>((const uint16_t*)W, K3, Cin, Cout, KCH, NB, (uint4*)wpack);
}

void launch_conv_run(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, const void* W,
                     const void* wpack, const float* scale, const float* shift, int relu, void* out, int Cout,
                     int dt) {
    if (conv_mfma_supported(Cin, Cout, dt)) {
        if (dt == SPV_BF16) launch_mfma<SPV_BF16>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout);
        else launch_mfma<SPV_F16>(s, p, in, Cin, in_rows, wpack, scale, shift, relu, out, Cout);
        return;
    }
    int64_t threads = p.m_cap * Cout;
    unsigned g = blocks_for(threads, 256);
    if (dt == SPV_F32) k_conv_generic<SPV_F32><<<g, 256, 0, s>>>(p, in, Cin, in_rows, W, scale, shift, relu, out, Cout);
    else if (dt == SPV_BF16)
        k_conv_generic<SPV_BF16><<<g, 256, 0, s>>>(p, in, Cin, in_rows, W, scale, shift, relu, out, Cout);
    else k_conv_generic<SPV_F16><<<g, 256, 0, s>>>(p, in, Cin, in_rows, W, scale, shift, relu, out, Cout);
}

}  // namespace spv
