// backward.hip -- gradients of the SPVConv path's operations:
//
// * weight gradient of a sparse convolution (Sec. 3.2):
//     dW[k] = sum over the pairs (i, j) of offset k of x[i]^T dy[j]
//   a GEMM per offset with the pairs as its K dimension.  Workgroup (s, k)
//   takes chunks s, s + S, ... of 64 pairs of offset k: the chunk's input and
//   gradient rows are gathered into LDS transposed (channel-major, the pairs
//   contiguous), so that each lane reads the 8 pairs of its operand as one
//   16-byte word; v_mfma_f32_16x16x32 then accumulates 16 x 16 tiles of
//   dW[k] (x^T as the A operand, dy as B), the tiles spread over the waves.
//   Each workgroup writes its fp32 partial sums; a second kernel adds the S
//   partials of every offset in slice order, so the result does not depend on
//   scheduling.  The input gradient needs no kernel of its own: it is the conv
//   over the same map with the pairs' roles swapped and W read transposed.
// * backward of the scatter-mean (Eq. 2): dfeat[k] = dv[v(k)] / N_v(k);
// * backward of the trilinear devoxelization w.r.t. the voxel features (Sec.
//   3.3): each point scatters its gradient to its present corners with the
//   weights the forward used (fp32 atomics: the order of the additions, and so
//   the last bits, vary from run to run).
#include "conv_common.hpp"

namespace spv {

constexpr int kWgWaves = 8;
constexpr int kWgChunk = 64;  // pairs per LDS fill: two MFMA K-steps of 32
constexpr int kWgLd = kWgChunk + 8;  // LDS row length in 16-bit elements (padded)
constexpr int kWgMaxRowPair = 512;    // Cin + Cout the MFMA kernel takes (8 pieces per thread)

// slices per offset: as many as a 64 MB partial-sum buffer holds (the centre
// offset of a submanifold map has ~15% of the pairs: more slices spread it
// over more compute units), a power of two in [8, 64]
static int wgrad_slices(int Cin, int Cout) {
    const int64_t per = (int64_t)27 * Cin * Cout * 4;
    int S = 64;
    while (S > 8 && per * S > ((int64_t)64 << 20)) S >>= 1;
    return S;
}

bool wgrad_supported(int Cin, int Cout) { return (int64_t)Cin * Cout <= 256 * 256; }

void* plan_wgrad_ws(Arena& a, int K3, int Cin, int Cout) {
    return a.take<float>((size_t)K3 * wgrad_slices(Cin, Cout) * Cin * Cout);
}

__device__ inline void pair_range(const int32_t* off, int k, int64_t pair_bound, int64_t& lo, int64_t& hi) {
    lo = off[k];
    hi = off[k + 1];
    lo = lo < 0 ? 0 : (lo > pair_bound ? pair_bound : lo);
    hi = hi < lo ? lo : (hi > pair_bound ? pair_bound : hi);
}

// PPT: 16-byte pieces each thread gathers per chunk (>= chunk pieces / threads)
template <int DT, int TPW, int PPT>
__global__ __launch_bounds__(64 * kWgWaves) void k_conv_wgrad_mfma(
    const uint16_t* __restrict__ x, int64_t x_rows, int Cin, const uint16_t* __restrict__ dy, int64_t dy_rows,
    int Cout, const int32_t* __restrict__ off, const int32_t* __restrict__ pairs, int64_t pair_bound, int transposed,
    float* __restrict__ partial) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* xt = (uint16_t*)smem;             // [Cin][kWgLd]
    uint16_t* gt = xt + (size_t)Cin * kWgLd;    // [Cout][kWgLd]
    const int k = blockIdx.y, S = gridDim.x, sl = blockIdx.x;
    int64_t lo, hi;
    pair_range(off, k, pair_bound, lo, hi);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r16 = lane & 15, g = lane >> 4;
    const int NTc = Cout / 16, NT = (Cin / 16) * NTc;
    const int qx = Cin / 8, qq = (Cin + Cout) / 8;  // 16-byte pieces of a pair's two rows
    const int isel = transposed ? 1 : 0;
    f32x4 acc[TPW];
#pragma unroll
    for (int u = 0; u < TPW; ++u) acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};

    // the thread's pieces of chunk c0 into registers: item e = threadIdx.x + r * threads
    // is piece e / 64 of pair e % 64 -- a wave's lanes take the same piece of 64
    // pairs, so their transposed LDS writes below fill consecutive columns of one
    // row (pieces of one pair in consecutive lanes would all hit one bank);
    // zeros past the chunk's pairs and the rows
    static_assert(kWgChunk == 64, "one pair per lane");
    uint4 pv[PPT];
    auto gather = [&](int64_t c0) {
        const int np = (hi - c0) < kWgChunk ? (int)(hi - c0) : kWgChunk;
#pragma unroll
        for (int r = 0; r < PPT; ++r) {
            const int e = threadIdx.x + r * 64 * kWgWaves;
            const int p = e & (kWgChunk - 1), q = e / kWgChunk;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (q < qq && p < np && c0 < hi) {
                const int64_t pp = c0 + p;
                if (q < qx) {
                    const int64_t i = pairs[2 * pp + isel];
                    if (i >= 0 && i < x_rows) v = *(const uint4*)(x + i * Cin + q * 8);
                } else {
                    const int64_t j = pairs[2 * pp + 1 - isel];
                    if (j >= 0 && j < dy_rows) v = *(const uint4*)(dy + j * Cout + (q - qx) * 8);
                }
            }
            pv[r] = v;
        }
    };
    const int64_t step = (int64_t)S * kWgChunk;
    int64_t c0 = lo + (int64_t)sl * kWgChunk;
    if (c0 < hi) gather(c0);
    for (; c0 < hi; c0 += step) {
        // the pieces in registers -> LDS, channel-major
#pragma unroll
        for (int r = 0; r < PPT; ++r) {
            const int e = threadIdx.x + r * 64 * kWgWaves;
            const int p = e & (kWgChunk - 1), q = e / kWgChunk;
            if (q < qq) {
                uint16_t* dst = (q < qx ? xt + (size_t)(q * 8) * kWgLd : gt + (size_t)((q - qx) * 8) * kWgLd) + p;
                const uint32_t w[4] = {pv[r].x, pv[r].y, pv[r].z, pv[r].w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    dst[(2 * h) * kWgLd] = (uint16_t)(w[h] & 0xFFFF);
                    dst[(2 * h + 1) * kWgLd] = (uint16_t)(w[h] >> 16);
                }
            }
        }
        __syncthreads();
        // the next chunk's gathers are in flight while this one is multiplied
        gather(c0 + step);
#pragma unroll
        for (int ks = 0; ks < kWgChunk / 32; ++ks) {
#pragma unroll
            for (int u = 0; u < TPW; ++u) {
                const int t = wave + u * kWgWaves;  // wave-uniform
                if (t < NT) {
                    const int ci0 = (t / NTc) * 16, co0 = (t - (t / NTc) * NTc) * 16;
                    const uint4 a = *(const uint4*)(xt + (size_t)(ci0 + r16) * kWgLd + ks * 32 + 8 * g);
                    const uint4 b = *(const uint4*)(gt + (size_t)(co0 + r16) * kWgLd + ks * 32 + 8 * g);
                    acc[u] = mfma16x16x32<DT>(a, b, acc[u]);
                }
            }
        }
        __syncthreads();
    }
    // lane (r16, g) of tile (ci0, co0) holds dW[ci0 + 4g + e][co0 + r16]
    float* pk = partial + ((int64_t)k * S + sl) * Cin * Cout;
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
        const int t = wave + u * kWgWaves;
        if (t < NT) {
            const int ci0 = (t / NTc) * 16, co0 = (t - (t / NTc) * NTc) * 16;
#pragma unroll
            for (int e = 0; e < 4; ++e) pk[(int64_t)(ci0 + 4 * g + e) * Cout + co0 + r16] = acc[u][e];
        }
    }
}

// other shapes and fp32: thread per (ci, co) of the workgroup's slice of offset k
template <int DT>
__global__ __launch_bounds__(256) void k_conv_wgrad_valu(const void* __restrict__ x, int64_t x_rows, int Cin,
                                                         const void* __restrict__ dy, int64_t dy_rows, int Cout,
                                                         const int32_t* __restrict__ off,
                                                         const int32_t* __restrict__ pairs, int64_t pair_bound,
                                                         int transposed, float* __restrict__ partial) {
    const int k = blockIdx.y, S = gridDim.x, sl = blockIdx.x;
    int64_t lo, hi;
    pair_range(off, k, pair_bound, lo, hi);
    const int isel = transposed ? 1 : 0;
    float* pk = partial + ((int64_t)k * S + sl) * Cin * Cout;
    for (int e = threadIdx.x; e < Cin * Cout; e += blockDim.x) {
        const int ci = e / Cout, co = e - ci * Cout;
        float s = 0.f;
        for (int64_t p = lo + sl; p < hi; p += S) {
            const int64_t i = pairs[2 * p + isel], j = pairs[2 * p + 1 - isel];
            if (i >= 0 && i < x_rows && j >= 0 && j < dy_rows)
                s += ld_feat<DT>(x, i * Cin + ci) * ld_feat<DT>(dy, j * Cout + co);
        }
        pk[e] = s;
    }
}

// dW[k][e] = sum over s of partial[k][s][e], in s order
__global__ void k_wgrad_reduce(const float* __restrict__ partial, int S, int64_t per_k, int K3, float* __restrict__ dW) {
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t >= (int64_t)K3 * per_k) return;
    const int64_t k = t / per_k, e = t - k * per_k;
    float s = 0.f;
    for (int q = 0; q < S; ++q) s += partial[(k * S + q) * per_k + e];
    dW[t] = s;
}

template <int DT, int TPW, int PPT>
static void launch_wgrad_mfma3(hipStream_t s, dim3 grid, const WgradArgs& a, float* partial) {
    const size_t lds = (size_t)(a.Cin + a.Cout) * kWgLd * 2;
    static const bool lds_ok = hipFuncSetAttribute((const void*)k_conv_wgrad_mfma<DT, TPW, PPT>,
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024) ==
                               hipSuccess;
    (void)lds_ok;
    k_conv_wgrad_mfma<DT, TPW, PPT><<<grid, 64 * kWgWaves, lds, s>>>((const uint16_t*)a.x, a.x_rows, a.Cin,
                                                                     (const uint16_t*)a.dy, a.dy_rows, a.Cout, a.off,
                                                                     a.pairs, a.pair_bound, a.transposed, partial);
}

template <int DT, int TPW>
static void launch_wgrad_mfma(hipStream_t s, dim3 grid, const WgradArgs& a, float* partial) {
    // pieces per thread: 64 pairs x (Cin + Cout) / 8 pieces over 512 threads
    const int ppt = (kWgChunk * ((a.Cin + a.Cout) / 8) + 64 * kWgWaves - 1) / (64 * kWgWaves);
    if (ppt <= 1) launch_wgrad_mfma3<DT, TPW, 1>(s, grid, a, partial);
    else if (ppt <= 2) launch_wgrad_mfma3<DT, TPW, 2>(s, grid, a, partial);
    else if (ppt <= 4) launch_wgrad_mfma3<DT, TPW, 4>(s, grid, a, partial);
    else launch_wgrad_mfma3<DT, TPW, 8>(s, grid, a, partial);  // Cin + Cout <= kWgMaxRowPair
}

template <int DT>
static void launch_wgrad_tpw(hipStream_t s, dim3 grid, const WgradArgs& a, float* partial) {
    const int nt = (a.Cin / 16) * (a.Cout / 16);
    const int tpw = (nt + kWgWaves - 1) / kWgWaves;
    if (tpw <= 1) launch_wgrad_mfma<DT, 1>(s, grid, a, partial);
    else if (tpw <= 2) launch_wgrad_mfma<DT, 2>(s, grid, a, partial);
    else if (tpw <= 4) launch_wgrad_mfma<DT, 4>(s, grid, a, partial);
    else if (tpw <= 8) launch_wgrad_mfma<DT, 8>(s, grid, a, partial);
    else if (tpw <= 16) launch_wgrad_mfma<DT, 16>(s, grid, a, partial);
    else launch_wgrad_mfma<DT, 32>(s, grid, a, partial);
}

void launch_wgrad(hipStream_t s, const WgradArgs& a, float* partial, float* dW) {
    const int S = wgrad_slices(a.Cin, a.Cout);
    const dim3 grid((unsigned)S, (unsigned)a.K3);
    // the MFMA kernel gathers at most 8 pieces of 16 bytes per thread, i.e. 64
    // pieces (512 channels) of a pair's two rows, and holds both rows of 64
    // pairs in LDS: wider pairs run on the vector-ALU kernel
    const bool mfma = a.dt != SPV_F32 && a.Cin % 16 == 0 && a.Cout % 16 == 0 && a.Cin + a.Cout <= kWgMaxRowPair;
    if (mfma) {
        if (a.dt == SPV_BF16) launch_wgrad_tpw<SPV_BF16>(s, grid, a, partial);
        else launch_wgrad_tpw<SPV_F16>(s, grid, a, partial);
    } else if (a.dt == SPV_F32) {
        k_conv_wgrad_valu<SPV_F32><<<grid, 256, 0, s>>>(a.x, a.x_rows, a.Cin, a.dy, a.dy_rows, a.Cout, a.off, a.pairs,
                                                        a.pair_bound, a.transposed, partial);
    } else if (a.dt == SPV_BF16) {
        k_conv_wgrad_valu<SPV_BF16><<<grid, 256, 0, s>>>(a.x, a.x_rows, a.Cin, a.dy, a.dy_rows, a.Cout, a.off,
                                                         a.pairs, a.pair_bound, a.transposed, partial);
    } else {
        k_conv_wgrad_valu<SPV_F16><<<grid, 256, 0, s>>>(a.x, a.x_rows, a.Cin, a.dy, a.dy_rows, a.Cout, a.off, a.pairs,
                                                        a.pair_bound, a.transposed, partial);
    }
    const int64_t per_k = (int64_t)a.Cin * a.Cout;
    k_wgrad_reduce<<<blocks_for((int64_t)a.K3 * per_k, 256), 256, 0, s>>>(partial, S, per_k, a.K3, dW);
}

// ---------------------------------------------------------------------------
// scatter-mean backward: thread per (point, channel); fp64 quotient, one rounding
// ---------------------------------------------------------------------------
template <int DT>
__global__ void k_vox_backward(const void* __restrict__ dv, int C, const int32_t* __restrict__ counts,
                               const int32_t* __restrict__ pt2vox, int64_t n, int64_t m, void* __restrict__ dfeat) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n * C; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = t / C;
        const int c = (int)(t - k * C);
        const int32_t v = pt2vox[k];
        const int32_t N = (v >= 0 && v < m) ? counts[v] : 0;
        const double q = N > 0 ? (double)ld_feat<DT>(dv, (int64_t)v * C + c) / (double)N : 0.0;
        if constexpr (DT == SPV_F32) ((float*)dfeat)[t] = (float)q;
        else ((uint16_t*)dfeat)[t] = to16<DT>(f64_to_f32_odd(q));
    }
}

// The same, one thread per (point, 16-byte chunk): the point's voxel and count
// are read once per chunk instead of once per channel, and the chunk moves in
// one load and one store.  VEC = 8 (16-bit storage) or 4 (fp32).
template <int DT, int VEC>
__global__ void k_vox_backward_vec(const void* __restrict__ dv, int C, const int32_t* __restrict__ counts,
                                   const int32_t* __restrict__ pt2vox, int64_t n, int64_t m,
                                   void* __restrict__ dfeat) {
    const int nch = C / VEC;
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t >= n * nch) return;
    const int64_t k = t / nch;
    const int c0 = (int)(t - k * nch) * VEC;
    const int32_t v = pt2vox[k];
    const int32_t N = (v >= 0 && v < m) ? counts[v] : 0;
    double q[VEC];
    if (N > 0) {
        if constexpr (VEC == 8) {
            const uint4 u = *(const uint4*)((const uint16_t*)dv + (int64_t)v * C + c0);
            const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                q[2 * j] = (double)from16<DT>(w[j] & 0xFFFF) / (double)N;
                q[2 * j + 1] = (double)from16<DT>(w[j] >> 16) / (double)N;
            }
        } else {
            const float4 f = *(const float4*)((const float*)dv + (int64_t)v * C + c0);
            q[0] = (double)f.x / (double)N;
            q[1] = (double)f.y / (double)N;
            q[2] = (double)f.z / (double)N;
            q[3] = (double)f.w / (double)N;
        }
    } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) q[j] = 0.0;
    }
    if constexpr (VEC == 8) {
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            w[j] = (uint32_t)to16<DT>(f64_to_f32_odd(q[2 * j])) | ((uint32_t)to16<DT>(f64_to_f32_odd(q[2 * j + 1])) << 16);
        *(uint4*)((uint16_t*)dfeat + k * C + c0) = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
        *(float4*)((float*)dfeat + k * C + c0) = make_float4((float)q[0], (float)q[1], (float)q[2], (float)q[3]);
    }
}

void launch_voxelize_backward(hipStream_t s, const void* dv, int C, const int32_t* counts, const int32_t* pt2vox,
                              int64_t n, int64_t m, void* dfeat, int dt) {
    if (n <= 0) return;
    // 16-byte chunks when the buffers and the rows allow them
    const bool a16 = (((uintptr_t)dv | (uintptr_t)dfeat) & 15u) == 0;
    if (a16 && dt != SPV_F32 && C % 8 == 0) {
        const unsigned g = (unsigned)blocks_for(n * (C / 8), 256);
        if (dt == SPV_BF16) k_vox_backward_vec<SPV_BF16, 8><<<g, 256, 0, s>>>(dv, C, counts, pt2vox, n, m, dfeat);
        else k_vox_backward_vec<SPV_F16, 8><<<g, 256, 0, s>>>(dv, C, counts, pt2vox, n, m, dfeat);
        return;
    }
    if (a16 && dt == SPV_F32 && C % 4 == 0) {
        const unsigned g = (unsigned)blocks_for(n * (C / 4), 256);
        k_vox_backward_vec<SPV_F32, 4><<<g, 256, 0, s>>>(dv, C, counts, pt2vox, n, m, dfeat);
        return;
    }
    int64_t g = blocks_for(n * C, 256);
    if (g > 8192) g = 8192;
    if (dt == SPV_F32) k_vox_backward<SPV_F32><<<(unsigned)g, 256, 0, s>>>(dv, C, counts, pt2vox, n, m, dfeat);
    else if (dt == SPV_BF16) k_vox_backward<SPV_BF16><<<(unsigned)g, 256, 0, s>>>(dv, C, counts, pt2vox, n, m, dfeat);
    else k_vox_backward<SPV_F16><<<(unsigned)g, 256, 0, s>>>(dv, C, counts, pt2vox, n, m, dfeat);
}

// ---------------------------------------------------------------------------
// devoxelization backward: zero dv, then thread per (point, channel) scatters
// to the point's present corners with the renormalized forward weights
// ---------------------------------------------------------------------------
__global__ void k_fill_zero_f32(float* p, int64_t n) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x)
        p[t] = 0.f;
}

template <int DT>
__global__ void k_devox_backward(const int32_t* __restrict__ cidx, const float* __restrict__ cw,
                                 const void* __restrict__ dout, int64_t n, int C, float* __restrict__ dv, int64_t m) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n * C; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = t / C;
        const int c = (int)(t - k * C);
        int32_t idx[8];
        float w[8];
        float den = 0.f;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            idx[q] = cidx[8 * k + q];
            w[q] = cw[8 * k + q];
            if (idx[q] >= 0 && idx[q] < m) den += w[q];
        }
        if (den <= 0.f) continue;
        const float g = ld_feat<DT>(dout, t) / den;
#pragma unroll
        for (int q = 0; q < 8; ++q)
            if (idx[q] >= 0 && idx[q] < m) atomicAdd(dv + (int64_t)idx[q] * C + c, w[q] * g);
    }
}

void launch_devoxelize_backward(hipStream_t s, const int32_t* cidx, const float* cw, const void* dout, int64_t n, int C,
                                float* dv, int64_t m, int dt) {
    if (m > 0) {
        int64_t gz = blocks_for(m * C, 256);
        if (gz > 8192) gz = 8192;
        k_fill_zero_f32<<<(unsigned)gz, 256, 0, s>>>(dv, m * C);
    }
    if (n <= 0) return;
    int64_t g = blocks_for(n * C, 256);
    if (g > 8192) g = 8192;
    if (dt == SPV_F32) k_devox_backward<SPV_F32><<<(unsigned)g, 256, 0, s>>>(cidx, cw, dout, n, C, dv, m);
    else if (dt == SPV_BF16) k_devox_backward<SPV_BF16><<<(unsigned)g, 256, 0, s>>>(cidx, cw, dout, n, C, dv, m);
    else k_devox_backward<SPV_F16><<<(unsigned)g, 256, 0, s>>>(cidx, cw, dout, n, C, dv, m);
}

}  // namespace spv
