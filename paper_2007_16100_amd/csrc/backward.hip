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
//   3.3): every voxel gathers the gradients of the points that have it as a
//   corner, weighted as the forward weighed them, in a fixed order (the same
//   bits on every run).
#include "conv_common.hpp"

namespace spv {

constexpr int kWgWaves = 8;
constexpr int kWgChunk = 64;  // pairs per LDS fill: two MFMA K-steps of 32
constexpr int kWgLd = kWgChunk + 8;  // LDS row length in 16-bit elements (padded)
constexpr int kWgMaxRowPair = 512;    // Cin + Cout the MFMA kernel takes (8 pieces per thread)

// slices per offset of the vector-ALU kernel: as many as a 64 MB partial-sum
// buffer holds (the centre offset of a submanifold map has ~15% of the pairs:
// more slices spread it over more compute units), a power of two in [8, 64];
// the buffer is sized by it for both kernels
static int wgrad_slices(int Cin, int Cout) {
    const int64_t per = (int64_t)27 * Cin * Cout * 4;
    int S = 64;
    while (S > 8 && per * S > ((int64_t)64 << 20)) S >>= 1;
    return S;
}

bool wgrad_supported(int Cin, int Cout) { return (int64_t)Cin * Cout <= 256 * 256; }

// The MFMA kernel splits the chunks of all offsets (64 pairs each, never
// across offsets; offset-major, as the map stores them) into G equal
// contiguous ranges, one per workgroup, so the centre offset's many pairs
// spread over as many workgroups as the rest.  A workgroup writes one
// partial sum per offset its range touches, to slot w + k: G + K3 - 1 slots
// at most, which the slice buffer (sized for slot_k3 * S slots) must hold.
constexpr int kWgMaxK3 = 27;
constexpr int kWgMaxGroups = 512;
__host__ __device__ inline int64_t wgrad_chunks_per_wg(int64_t chunks, int G) { return (chunks + G - 1) / G; }
// LDS of the MFMA kernel: the transposed chunk tiles, then the offsets' pair
// ranges and chunk prefix (27 + 27 + 28 int64)
__host__ __device__ inline size_t wgrad_tiles_bytes(int Cin, int Cout) {
    return ((size_t)(Cin + Cout) * kWgLd * 2 + 15) & ~(size_t)15;
}
static int wgrad_groups(int K3, int S) {
    const int g = K3 * (S - 1);
    return g < kWgMaxGroups ? g : kWgMaxGroups;
}

void* plan_wgrad_ws(Arena& a, int K3, int Cin, int Cout) {
    return a.take<float>((size_t)K3 * wgrad_slices(Cin, Cout) * Cin * Cout);
}

// The pairs of offset k, clamped to the pair buffer.  Without off and pairs
// the "map" is the identity on pair_bound rows, one offset: pair p = (p, p)
// (the weight gradient of a linear layer, x^T dy).
__device__ inline void pair_range(const int32_t* off, int k, int64_t pair_bound, int64_t& lo, int64_t& hi) {
    if (!off) {
        lo = 0;
        hi = k == 0 ? pair_bound : 0;
        return;
    }
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
    int K3, float* __restrict__ partial) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* xt = (uint16_t*)smem;             // [Cin][kWgLd]
    uint16_t* gt = xt + (size_t)Cin * kWgLd;    // [Cout][kWgLd]
    // then the offsets' pair ranges and chunk prefix (all LDS is dynamic: the
    // launch raises the dynamic limit to the whole 160 KB)
    int64_t* s_lo = (int64_t*)(smem + wgrad_tiles_bytes(Cin, Cout));
    int64_t* s_hi = s_lo + kWgMaxK3;
    int64_t* s_cpre = s_hi + kWgMaxK3;
    const int G = gridDim.x, w = blockIdx.x;
    if (threadIdx.x == 0) {
        int64_t c = 0;
        for (int k = 0; k < K3; ++k) {
            pair_range(off, k, pair_bound, s_lo[k], s_hi[k]);
            s_cpre[k] = c;
            c += (s_hi[k] - s_lo[k] + kWgChunk - 1) / kWgChunk;
        }
        s_cpre[K3] = c;
    }
    __syncthreads();
    const int64_t T = wgrad_chunks_per_wg(s_cpre[K3], G);
    const int64_t g0 = (int64_t)w * T, g1 = g0 + T < s_cpre[K3] ? g0 + T : s_cpre[K3];
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
    // global chunk gc: its offset (from kc upwards) and first pair
    auto locate = [&](int64_t gc, int& kc, int64_t& c0, int& np) {
        while (kc + 1 < K3 && gc >= s_cpre[kc + 1]) ++kc;
        c0 = s_lo[kc] + (gc - s_cpre[kc]) * kWgChunk;
        const int64_t left = s_hi[kc] - c0;
        np = left < kWgChunk ? (int)left : kWgChunk;
    };
    // a thread's pieces all belong to pair threadIdx.x % 64 of the chunk: its
    // two row indices are loaded one chunk before its rows (-1: no pair)
    auto load_idx = [&](int64_t c0, int np, int64_t& ii, int64_t& jj) {
        const int p = threadIdx.x & (kWgChunk - 1);
        ii = -1;
        jj = -1;
        if (p < np) {
            if (pairs) {
                ii = pairs[2 * (c0 + p) + isel];
                jj = pairs[2 * (c0 + p) + 1 - isel];
            } else {
                ii = jj = c0 + p;
            }
        }
    };
    auto gather = [&](int64_t ii, int64_t jj) {
#pragma unroll
        for (int r = 0; r < PPT; ++r) {
            const int q = (threadIdx.x + r * 64 * kWgWaves) / kWgChunk;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (q < qx) {
                if (ii >= 0 && ii < x_rows) v = *(const uint4*)(x + ii * Cin + q * 8);
            } else if (q < qq) {
                if (jj >= 0 && jj < dy_rows) v = *(const uint4*)(dy + jj * Cout + (q - qx) * 8);
            }
            pv[r] = v;
        }
    };
    // lane (r16, g) of tile (ci0, co0) holds dW[ci0 + 4g + e][co0 + r16]: the
    // workgroup's sums for offset k go to slot w + k (the offsets a workgroup
    // covers only grow with w, so the slots are distinct)
    auto flush = [&](int k) {
        float* pk = partial + ((int64_t)w + k) * Cin * Cout;
#pragma unroll
        for (int u = 0; u < TPW; ++u) {
            const int t = wave + u * kWgWaves;
            if (t < NT) {
                const int ci0 = (t / NTc) * 16, co0 = (t - (t / NTc) * NTc) * 16;
                // Cout through an opaque copy: left visible, the compiler hoists
                // all TPW * 4 store addresses out of the chunk loop (66 more
                // registers, half the waves per SIMD)
                int cv;
                asm volatile("s_mov_b32 %0, %1" : "=s"(cv) : "s"(Cout));
                float* q = pk + (int64_t)(ci0 + 4 * g) * cv + co0 + r16;
#pragma unroll
                for (int e = 0; e < 4; ++e) q[(int64_t)e * cv] = acc[u][e];
            }
            acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };
    // chunk gc's rows are in pv; chunk gc + 1's offset k1 and row indices
    // (i1, j1) are known
    int kcur = 0, k1 = 0;
    int64_t i1 = -1, j1 = -1;
    if (g0 < g1) {
        int64_t c0, ii, jj;
        int np;
        locate(g0, kcur, c0, np);
        load_idx(c0, np, ii, jj);
        gather(ii, jj);
        k1 = kcur;
        if (g0 + 1 < g1) {
            locate(g0 + 1, k1, c0, np);
            load_idx(c0, np, i1, j1);
        }
    }
    for (int64_t gc = g0; gc < g1; ++gc) {
        // the pieces in registers -> LDS, channel-major
#pragma unroll
        for (int r = 0; r < PPT; ++r) {
            const int e = threadIdx.x + r * 64 * kWgWaves;
            const int p = e & (kWgChunk - 1), q = e / kWgChunk;
            if (q < qq) {
                uint16_t* dst = (q < qx ? xt + (size_t)(q * 8) * kWgLd : gt + (size_t)((q - qx) * 8) * kWgLd) + p;
                const uint32_t wd[4] = {pv[r].x, pv[r].y, pv[r].z, pv[r].w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    dst[(2 * h) * kWgLd] = (uint16_t)(wd[h] & 0xFFFF);
                    dst[(2 * h + 1) * kWgLd] = (uint16_t)(wd[h] >> 16);
                }
            }
        }
        __syncthreads();
        // the next chunk's rows and the indices of the one after are in flight
        // while this one is multiplied
        gather(i1, j1);
        int k2 = k1;
        int64_t i2 = -1, j2 = -1;
        if (gc + 2 < g1) {
            int64_t c2;
            int n2;
            locate(gc + 2, k2, c2, n2);
            load_idx(c2, n2, i2, j2);
        }
#pragma unroll
        for (int ks = 0; ks < kWgChunk / 32; ++ks) {
#pragma unroll
            for (int u = 0; u < TPW; ++u) {
                // wave-uniform.  With 16 or more tiles per wave it goes through an
                // opaque copy, as Cout in flush: the LDS addresses of all tiles
                // would otherwise be hoisted out of the chunk loop and held,
                // and the wave would spill (with fewer tiles, recomputing them
                // every chunk costs more than holding them)
                int t = wave + u * kWgWaves;
                if constexpr (TPW >= 16) asm volatile("s_mov_b32 %0, %1" : "=s"(t) : "s"(wave + u * kWgWaves));
                if (t < NT) {
                    const int ci0 = (t / NTc) * 16, co0 = (t - (t / NTc) * NTc) * 16;
                    const uint4 a = *(const uint4*)(xt + (size_t)(ci0 + r16) * kWgLd + ks * 32 + 8 * g);
                    const uint4 b = *(const uint4*)(gt + (size_t)(co0 + r16) * kWgLd + ks * 32 + 8 * g);
                    acc[u] = mfma16x16x32<DT>(a, b, acc[u]);
                }
            }
        }
        __syncthreads();
        if (gc + 1 == g1 || k1 != kcur) flush(kcur);
        kcur = k1;
        k1 = k2;
        i1 = i2;
        j1 = j2;
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
            const int64_t i = pairs ? pairs[2 * p + isel] : p, j = pairs ? pairs[2 * p + 1 - isel] : p;
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

__device__ inline void acc_add(float& s, float v) { s += v; }
__device__ inline void acc_add(float4& s, const float4& v) {
    s.x += v.x;
    s.y += v.y;
    s.z += v.z;
    s.w += v.w;
}

// dW[k][e] = the sum of slots w + k over the workgroups w whose chunk ranges
// touch offset k (zero when offset k has no pairs).  V = float4 (four elements
// per lane) or float.  A workgroup of 4 waves takes 64 element groups of one
// offset: wave q sums the q-th quarter of the workgroups in order, and the
// four quarter sums are added in quarter order -- a fixed association, so the
// result does not depend on scheduling, with a quarter of the dependent loads
// per lane.  The chunk bounds of offset k are recomputed from off as the MFMA
// kernel computed them.
constexpr int kWgRedParts = 4;
template <class V>
__global__ __launch_bounds__(64 * kWgRedParts) void k_wgrad_reduce_bal(const V* __restrict__ partial, int G,
                                                                       int64_t per_kv, const int32_t* off,
                                                                       int64_t pair_bound, V* __restrict__ dW) {
    __shared__ V red[kWgRedParts][64];
    const int k = blockIdx.y, K3 = gridDim.y;
    const int lane = threadIdx.x & 63, part = threadIdx.x >> 6;
    const int64_t e = blockIdx.x * (int64_t)64 + lane;
    int64_t c = 0, ck = 0, nk = 0;
    for (int q = 0; q < K3; ++q) {
        int64_t lo, hi;
        pair_range(off, q, pair_bound, lo, hi);
        const int64_t n = (hi - lo + kWgChunk - 1) / kWgChunk;
        if (q == k) {
            ck = c;
            nk = n;
        }
        c += n;
    }
    V s{};
    if (nk > 0 && e < per_kv) {
        const int64_t T = wgrad_chunks_per_wg(c, G);
        const int64_t wlo = ck / T, nw = (ck + nk - 1) / T - wlo + 1;
        const int64_t pw = (nw + kWgRedParts - 1) / kWgRedParts;
        const int64_t wa = wlo + part * pw, wb = wa + pw < wlo + nw ? wa + pw : wlo + nw;
        int64_t w = wa;
        for (; w + 8 <= wb; w += 8) {  // the loads together, the additions in order
            V v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = partial[(w + u + k) * per_kv + e];
#pragma unroll
            for (int u = 0; u < 8; ++u) acc_add(s, v[u]);
        }
        for (; w < wb; ++w) acc_add(s, partial[(w + k) * per_kv + e]);
    }
    red[part][lane] = s;
    __syncthreads();
    if (part == 0 && e < per_kv) {
#pragma unroll
        for (int q = 1; q < kWgRedParts; ++q) acc_add(s, red[q][lane]);
        dW[(int64_t)k * per_kv + e] = s;
    }
}

// The same sums four elements per thread, the slices eight at a time (their
// loads issued together, then added in slice order: the same bits as above).
// Needs per_k % 4 == 0, S % 8 == 0 and a 16-byte aligned dW.
__global__ void k_wgrad_reduce4(const float4* __restrict__ partial, int S, int64_t per_k4, int K3,
                                float4* __restrict__ dW) {
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t >= (int64_t)K3 * per_k4) return;
    const int64_t k = t / per_k4, e = t - k * per_k4;
    const float4* p = partial + k * S * per_k4 + e;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int q = 0; q < S; q += 8) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = p[(int64_t)(q + u) * per_k4];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            s.x += v[u].x;
            s.y += v[u].y;
            s.z += v[u].z;
            s.w += v[u].w;
        }
    }
    dW[t] = s;
}

template <int DT, int TPW, int PPT>
static void launch_wgrad_mfma3(hipStream_t s, dim3 grid, const WgradArgs& a, float* partial) {
    const size_t lds = wgrad_tiles_bytes(a.Cin, a.Cout) + (3 * kWgMaxK3 + 1) * sizeof(int64_t);
    static const bool lds_ok = hipFuncSetAttribute((const void*)k_conv_wgrad_mfma<DT, TPW, PPT>,
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024) ==
                               hipSuccess;
    (void)lds_ok;
    k_conv_wgrad_mfma<DT, TPW, PPT><<<grid, 64 * kWgWaves, lds, s>>>((const uint16_t*)a.x, a.x_rows, a.Cin,
                                                                     (const uint16_t*)a.dy, a.dy_rows, a.Cout, a.off,
                                                                     a.pairs, a.pair_bound, a.transposed, a.K3,
                                                                     partial);
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
    // the buffer holds slot_k3 * S slots: G + K3 - 1 <= slot_k3 * S
    const int sk = a.slot_k3 > a.K3 ? a.slot_k3 : a.K3;
    int G = wgrad_groups(sk, S);
    if (G > sk * S - a.K3 + 1) G = sk * S - a.K3 + 1;
    if (!a.off) {
        // the identity map's chunk count is known here: about eight chunks per
        // workgroup, so that the reduction has fewer partial sums to add
        const int64_t ch = (a.pair_bound + kWgChunk - 1) / kWgChunk;
        const int64_t gi = ch / 8 > 1 ? ch / 8 : 1;
        if (gi < G) G = (int)gi;
    }
    // the MFMA kernel gathers at most 8 pieces of 16 bytes per thread, i.e. 64
    // pieces (512 channels) of a pair's two rows, and holds both rows of 64
    // pairs in LDS: wider pairs run on the vector-ALU kernel
    const bool mfma = a.dt != SPV_F32 && a.Cin % 16 == 0 && a.Cout % 16 == 0 && a.Cin + a.Cout <= kWgMaxRowPair;
    const int64_t per_k = (int64_t)a.Cin * a.Cout;
    if (mfma) {
        const dim3 gb((unsigned)G, 1);
        if (a.dt == SPV_BF16) launch_wgrad_tpw<SPV_BF16>(s, gb, a, partial);
        else launch_wgrad_tpw<SPV_F16>(s, gb, a, partial);
        // per_k is a multiple of 256 here (16-channel multiples)
        if (((uintptr_t)dW & 15u) == 0) {
            const dim3 gr(blocks_for(per_k / 4, 64), (unsigned)a.K3);
            k_wgrad_reduce_bal<float4><<<gr, 64 * kWgRedParts, 0, s>>>((const float4*)partial, G, per_k / 4, a.off,
                                                                       a.pair_bound, (float4*)dW);
        } else {
            const dim3 gr(blocks_for(per_k, 64), (unsigned)a.K3);
            k_wgrad_reduce_bal<float><<<gr, 64 * kWgRedParts, 0, s>>>(partial, G, per_k, a.off, a.pair_bound, dW);
        }
        return;
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
    if (per_k % 4 == 0 && S % 8 == 0 && ((uintptr_t)dW & 15u) == 0)
        k_wgrad_reduce4<<<blocks_for((int64_t)a.K3 * per_k / 4, 256), 256, 0, s>>>((const float4*)partial, S,
                                                                                    per_k / 4, a.K3, (float4*)dW);
    else
        k_wgrad_reduce<<<blocks_for((int64_t)a.K3 * per_k, 256), 256, 0, s>>>(partial, S, per_k, a.K3, dW);
}

// ---------------------------------------------------------------------------
// backward of the epilogue act(scale * a + shift (+ res)) (+ res) the convs and
// linear layers apply to their raw product a.  The activation's input is formed
// in float32 as fmaf(a, scale, shift) (+ res), the ReLU passes the gradient
// where it is > 0; da = gz * scale rounds once (an exact fp64 product), dres is
// dy or gz unchanged.  The per-channel sums dscale = sum gz * a and dshift =
// sum gz run in fp64 in a fixed association: within a workgroup of kEbRows
// rows, row lane q sums rows q, q + 4, ... in order and the four lanes are
// added in order; a second kernel adds the workgroups' sums in contiguous
// runs of the 256 threads, then the runs in order.
// ---------------------------------------------------------------------------
constexpr int kEbRows = 128;
constexpr int kEbLanes = 4;

size_t epilogue_backward_part_entries(int64_t m, int C) { return (size_t)blocks_for(m, kEbRows) * 2 * (size_t)C; }

template <int DT>
__global__ __launch_bounds__(64 * kEbLanes) void k_epi_backward(EpiBwdArgs a, double* part) {
    __shared__ double red[kEbLanes][2][64];
    const int cl = threadIdx.x & 63, rl = threadIdx.x >> 6;
    const int c = blockIdx.y * 64 + cl;
    const int64_t r0 = (int64_t)blockIdx.x * kEbRows;
    const int64_t r1 = r0 + kEbRows < a.m ? r0 + kEbRows : a.m;
    double ss = 0.0, sb = 0.0;
    if (c < a.C) {
        const float sc = a.scale ? a.scale[c] : 1.f, sh = a.shift ? a.shift[c] : 0.f;
        const bool rb = a.res && !a.res_after;
        // U rows per round: their loads first, then the rows in order
        constexpr int U = 4;
        for (int64_t i0 = r0 + rl; i0 < r1; i0 += U * kEbLanes) {
            float av[U], g[U], rv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t i = i0 + u * kEbLanes;
                const int64_t t = i * a.C + c;
                const bool in = i < r1;
                av[u] = in ? ld_feat<DT>(a.a, t) : 0.f;
                g[u] = in ? ld_feat<DT>(a.dy, t) : 0.f;
                rv[u] = (in && rb) ? ld_feat<DT>(a.res, t) : 0.f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t i = i0 + u * kEbLanes;
                if (i >= r1) break;
                const int64_t t = i * a.C + c;
                float z = fmaf(av[u], sc, sh);
                if (rb) z = z + rv[u];
                const float gz = (!a.relu || z > 0.f) ? g[u] : 0.f;
                if (a.da) {
                    const double d = (double)gz * (double)sc;
                    if constexpr (DT == SPV_F32) ((float*)a.da)[t] = (float)d;
                    else ((uint16_t*)a.da)[t] = to16<DT>(f64_to_f32_odd(d));
                }
                if (a.dres) st_feat<DT>(a.dres, t, a.res_after ? g[u] : gz);
                ss += (double)gz * (double)av[u];
                sb += (double)gz;
            }
        }
    }
    if (!part) return;  // the whole workgroup
    red[rl][0][cl] = ss;
    red[rl][1][cl] = sb;
    __syncthreads();
    if (rl == 0 && c < a.C) {
        for (int q = 1; q < kEbLanes; ++q) {
            ss += red[q][0][cl];
            sb += red[q][1][cl];
        }
        part[((int64_t)blockIdx.x * 2) * a.C + c] = ss;
        part[((int64_t)blockIdx.x * 2 + 1) * a.C + c] = sb;
    }
}

// The same, VEC channels per thread (16-byte loads and stores; C % VEC == 0,
// C / VEC <= 256, 16-byte aligned rows): thread (lane q, group g) of the
// L = 256 / G lanes takes rows q, q + L, ... of the workgroup's kEbRows; the
// lanes' sums are added in lane order.
template <int DT, int VEC>
__device__ inline void epi_ld(const void* p, int64_t i, float (&x)[VEC]) {
    if constexpr (DT == SPV_F32) {
        const float4 v = *(const float4*)((const float*)p + i);
        x[0] = v.x;
        x[1] = v.y;
        x[2] = v.z;
        x[3] = v.w;
    } else {
        const uint4 v = *(const uint4*)((const uint16_t*)p + i);
        const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            x[2 * j] = from16<DT>(u[j] & 0xffffu);
            x[2 * j + 1] = from16<DT>(u[j] >> 16);
        }
    }
}
template <int DT, int VEC>
__device__ inline void epi_st(void* p, int64_t i, const float (&x)[VEC]) {
    if constexpr (DT == SPV_F32) {
        *(float4*)((float*)p + i) = make_float4(x[0], x[1], x[2], x[3]);
    } else {
        uint32_t u[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) u[j] = (uint32_t)to16<DT>(x[2 * j]) | ((uint32_t)to16<DT>(x[2 * j + 1]) << 16);
        *(uint4*)((uint16_t*)p + i) = make_uint4(u[0], u[1], u[2], u[3]);
    }
}

template <int DT, int VEC>
__global__ __launch_bounds__(256) void k_epi_backward_vec(EpiBwdArgs a, double* part) {
    __shared__ double red[256][2 * VEC];
    const int G = a.C / VEC, L = 256 / G;
    const int q = threadIdx.x / G, g = threadIdx.x - q * G;
    const int64_t r0 = (int64_t)blockIdx.x * kEbRows;
    const int64_t r1 = r0 + kEbRows < a.m ? r0 + kEbRows : a.m;
    double ss[VEC], sb[VEC];
#pragma unroll
    for (int c = 0; c < VEC; ++c) ss[c] = sb[c] = 0.0;
    if (q < L) {
        float sc[VEC], sh[VEC];
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            sc[c] = a.scale ? a.scale[g * VEC + c] : 1.f;
            sh[c] = a.shift ? a.shift[g * VEC + c] : 0.f;
        }
        const bool rb = a.res && !a.res_after;
        for (int64_t i = r0 + q; i < r1; i += L) {
            const int64_t t = i * a.C + g * VEC;
            float av[VEC], gv[VEC], rv[VEC];
            epi_ld<DT, VEC>(a.a, t, av);
            epi_ld<DT, VEC>(a.dy, t, gv);
            if (rb) epi_ld<DT, VEC>(a.res, t, rv);
            float dz[VEC], dr[VEC];
#pragma unroll
            for (int c = 0; c < VEC; ++c) {
                float z = fmaf(av[c], sc[c], sh[c]);
                if (rb) z = z + rv[c];
                const float gz = (!a.relu || z > 0.f) ? gv[c] : 0.f;
                const double d = (double)gz * (double)sc[c];
                dz[c] = (DT == SPV_F32) ? (float)d : f64_to_f32_odd(d);  // one rounding below
                dr[c] = a.res_after ? gv[c] : gz;
                ss[c] += (double)gz * (double)av[c];
                sb[c] += (double)gz;
            }
            if (a.da) epi_st<DT, VEC>(a.da, t, dz);
            if (a.dres) epi_st<DT, VEC>(a.dres, t, dr);
        }
    }
    if (!part) return;  // the whole workgroup
#pragma unroll
    for (int c = 0; c < VEC; ++c) {
        red[threadIdx.x][c] = ss[c];
        red[threadIdx.x][VEC + c] = sb[c];
    }
    __syncthreads();
    if (q == 0) {
        for (int qq = 1; qq < L; ++qq)
#pragma unroll
            for (int c = 0; c < VEC; ++c) {
                ss[c] += red[qq * G + g][c];
                sb[c] += red[qq * G + g][VEC + c];
            }
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            part[((int64_t)blockIdx.x * 2) * a.C + g * VEC + c] = ss[c];
            part[((int64_t)blockIdx.x * 2 + 1) * a.C + g * VEC + c] = sb[c];
        }
    }
}

__global__ __launch_bounds__(256) void k_epi_reduce(const double* __restrict__ part, int64_t nblk, int C,
                                                    float* __restrict__ dscale, float* __restrict__ dshift) {
    __shared__ double rs[256], rb[256];
    const int c = blockIdx.x;
    const int64_t L = (nblk + 255) / 256;
    const int64_t b0 = threadIdx.x * L, b1 = b0 + L < nblk ? b0 + L : nblk;
    double ss = 0.0, sb = 0.0;
    for (int64_t b = b0; b < b1; ++b) {
        ss += part[(b * 2) * C + c];
        sb += part[(b * 2 + 1) * C + c];
    }
    rs[threadIdx.x] = ss;
    rb[threadIdx.x] = sb;
    __syncthreads();
    if (threadIdx.x == 0) {
        double s0 = 0.0, s1 = 0.0;
        for (int q = 0; q < 256; ++q) {
            s0 += rs[q];
            s1 += rb[q];
        }
        if (dscale) dscale[c] = (float)s0;
        if (dshift) dshift[c] = (float)s1;
    }
}

void launch_epilogue_backward(hipStream_t s, const EpiBwdArgs& a, double* part) {
    const bool sums = a.dscale || a.dshift;
    const dim3 g(blocks_for(a.m, kEbRows), (unsigned)((a.C + 63) / 64));
    double* p = sums ? part : nullptr;
    const int vec = a.dt == SPV_F32 ? 4 : 8;
    const bool al = (((uintptr_t)a.dy | (uintptr_t)a.a | (uintptr_t)a.res | (uintptr_t)a.da | (uintptr_t)a.dres) &
                     15u) == 0;
    if (al && a.C % vec == 0 && a.C / vec <= 256) {
        if (a.dt == SPV_F32) k_epi_backward_vec<SPV_F32, 4><<<g.x, 256, 0, s>>>(a, p);
        else if (a.dt == SPV_BF16) k_epi_backward_vec<SPV_BF16, 8><<<g.x, 256, 0, s>>>(a, p);
        else k_epi_backward_vec<SPV_F16, 8><<<g.x, 256, 0, s>>>(a, p);
    } else if (a.dt == SPV_F32) {
        k_epi_backward<SPV_F32><<<g, 64 * kEbLanes, 0, s>>>(a, p);
    } else if (a.dt == SPV_BF16) {
        k_epi_backward<SPV_BF16><<<g, 64 * kEbLanes, 0, s>>>(a, p);
    } else {
        k_epi_backward<SPV_F16><<<g, 64 * kEbLanes, 0, s>>>(a, p);
    }
    if (sums) k_epi_reduce<<<(unsigned)a.C, 256, 0, s>>>(part, (int64_t)g.x, a.C, a.dscale, a.dshift);
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
// devoxelization backward, deterministic.  An entry is one present corner c of
// one point k, numbered e = 8k + c, with the coefficient a = w_c / (sum of the
// point's present corner weights).  A counting sort groups the entries by
// voxel (count, scan, fill: inside a voxel the order is whatever the atomics
// of the count gave); every entry then takes its place in ascending e among its
// voxel's entries (it counts the smaller ones of its chunk of 256, then finds
// those of the other chunks by binary search); the gather sums a voxel's entries
// a * dout[k] in that order, one fp32 fma after another, so the result is the
// same bit for bit on every run.  Every voxel row is written, the empty ones
// with zeros.
// ---------------------------------------------------------------------------
DvbWs plan_devox_backward_ws(Arena& a, int64_t n, int64_t m) {
    DvbWs w;
    w.h = a.take<Header>(1);
    w.cnt = a.take<int32_t>((size_t)m + 1);
    w.off = a.take<int32_t>((size_t)m + 1);
    w.tmp = a.take<int32_t>(scan_tmp_entries(m));
    const size_t E = 8 * (size_t)n;
    w.slot = a.take<int32_t>(E);
    w.ent = a.take<int32_t>(E);
    w.coef = a.take<float>(E);
    w.vox = a.take<int32_t>(E);
    w.rec = a.take<int2>(E);
    w.chk = a.take<int2>(E);
    w.longv = a.take<int32_t>((size_t)m + 1);
    return w;
}

__global__ void k_dvb_zero(Header* h, int32_t* cnt, int64_t len) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        h->status = 0;
        h->m = 0;
        for (int i = 0; i < 4; ++i) h->aux[i] = 0;
    }
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < len; i += (int64_t)gridDim.x * blockDim.x)
        cnt[i] = 0;
}

// point k's present corners (0 <= idx < m; an index past m is reported and
// skipped) and their coefficients; false when the weights sum to <= 0
__device__ inline bool dvb_corners(const int32_t* cidx, const float* cw, int64_t k, int64_t m, Header* h,
                                   int32_t idx[8], float a[8]) {
    float den = 0.f;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        idx[q] = cidx[8 * k + q];
        a[q] = cw[8 * k + q];
        if (idx[q] >= m) {
            if (h) raise_flag(h, kFlagRange);
            idx[q] = -1;
        }
        if (idx[q] >= 0) den += a[q];
    }
    if (den <= 0.f) return false;
#pragma unroll
    for (int q = 0; q < 8; ++q) a[q] = a[q] / den;
    return true;
}

// Count every voxel's entries and give each entry its slot among them.  A
// workgroup first groups its points' entries by voxel in an LDS hash table
// (the points of a workgroup lie close together and share most corners), then
// claims each voxel's share with one global atomic; an entry's slot is the
// claimed base plus its rank in the workgroup.  slot[8k + c] = -1 marks an
// absent corner.
constexpr int kDvbThreads = 256;
constexpr int kDvbHash = 4096;  // at most 8 * kDvbThreads keys: the table stays at most half full

__global__ __launch_bounds__(kDvbThreads) void k_dvb_count(const int32_t* __restrict__ cidx,
                                                           const float* __restrict__ cw, int64_t n, int64_t m,
                                                           Header* h, int32_t* cnt, int32_t* __restrict__ slot) {
    __shared__ int32_t hkey[kDvbHash];
    __shared__ int32_t hval[kDvbHash];  // the workgroup's count of the key's entries, then the claimed base
    const int t = threadIdx.x;
    for (int i = t; i < kDvbHash; i += kDvbThreads) {
        hkey[i] = -1;
        hval[i] = 0;
    }
    __syncthreads();
    const int64_t k = (int64_t)blockIdx.x * kDvbThreads + t;
    int32_t idx[8];
    float a[8];
    const bool live = k < n && dvb_corners(cidx, cw, k, m, h, idx, a);
    int hs[8], lr[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        hs[q] = -1;
        lr[q] = 0;
        if (!live || idx[q] < 0) continue;
        uint32_t p = ((uint32_t)idx[q] * 2654435761u) >> 20;  // 12 bits
        while (true) {
            const int32_t old = atomicCAS(&hkey[p], -1, idx[q]);
            if (old == -1 || old == idx[q]) break;
            p = (p + 1) & (kDvbHash - 1);
        }
        hs[q] = (int)p;
        lr[q] = atomicAdd(&hval[p], 1);
    }
    __syncthreads();
    for (int i = t; i < kDvbHash; i += kDvbThreads) {
        const int32_t v = hkey[i];
        if (v >= 0) hval[i] = atomicAdd(cnt + v, hval[i]);
    }
    __syncthreads();
    if (k < n) {
        int32_t sl[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) sl[q] = hs[q] >= 0 ? hval[hs[q]] + lr[q] : -1;
        int4* o = (int4*)(slot + 8 * k);
        o[0] = make_int4(sl[0], sl[1], sl[2], sl[3]);
        o[1] = make_int4(sl[4], sl[5], sl[6], sl[7]);
    }
}

// every entry to its place in its voxel's range (no atomics: the count kernel
// gave the slots)
__global__ void k_dvb_fill(const int32_t* __restrict__ cidx, const float* __restrict__ cw, int64_t n, int64_t m,
                           Header* h, const int32_t* __restrict__ slot, const int32_t* __restrict__ off, int32_t* ent,
                           float* coef, int32_t* vox) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n; k += (int64_t)gridDim.x * blockDim.x) {
        int32_t idx[8];
        float a[8];
        if (!dvb_corners(cidx, cw, k, m, nullptr, idx, a)) continue;
        const int4* sp = (const int4*)(slot + 8 * k);
        const int4 s0 = sp[0], s1 = sp[1];
        const int32_t sl[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int32_t v = idx[q];
            if (v < 0) continue;
            const int32_t lo = off[v];
            if (sl[q] < 0 || sl[q] >= off[v + 1] - lo) {  // cannot happen: the count kernel saw the same corners
                raise_flag(h, kFlagInternal);
                continue;
            }
            const int64_t pos = lo + sl[q];
            ent[pos] = (int32_t)(8 * k + q);
            coef[pos] = a[q];
            vox[pos] = v;
        }
    }
}

// Entry i of voxel v goes to position off[v] + (the entries of v smaller than
// it); entries are distinct, so the positions are too.  A voxel's range (in
// fill order) is cut into chunks of kDvbChunk: every entry first counts the
// smaller entries of its own chunk.  A voxel of one chunk is then done (its
// entry goes straight to its place in rec); in a longer one the entry goes to
// that rank inside its chunk of chk (each chunk sorted), and the merge kernel
// adds, by a binary search of every other chunk, the smaller entries there --
// L * (kDvbChunk + (L / kDvbChunk) log kDvbChunk) comparisons for a voxel of L
// entries instead of L^2.
constexpr int kDvbChunk = 256;
constexpr int kDvbLong = 64;  // longer voxels are gathered by a workgroup each

__global__ void k_dvb_rank(const int32_t* __restrict__ off, int64_t m, int64_t cap, const int32_t* __restrict__ ent,
                           const float* __restrict__ coef, const int32_t* __restrict__ vox, int2* __restrict__ rec,
                           int2* __restrict__ chk, Header* h, int32_t* longv) {
    int64_t E = off[m];
    if (E > cap) E = cap;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < E; i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t v = vox[i], key = ent[i];
        if ((uint64_t)(uint32_t)v >= (uint64_t)m) continue;  // only after a fill that raised kFlagInternal
        const int32_t lo = off[v], hi = off[v + 1];
        const int32_t c0 = lo + ((int32_t)(i - lo) / kDvbChunk) * kDvbChunk;
        const int32_t c1 = c0 + kDvbChunk < hi ? c0 + kDvbChunk : hi;
        int32_t r = 0;
        for (int32_t j = c0; j < c1; ++j) r += ent[j] < key ? 1 : 0;
        const int2 e = make_int2(key, __float_as_int(coef[i]));
        if (hi - lo <= kDvbChunk) rec[lo + r] = e;
        else chk[c0 + r] = e;
        // the voxels whose gather takes a workgroup, once each (by the first entry in fill order)
        if (i == lo && hi - lo > kDvbLong)
            longv[atomicAdd((unsigned long long*)&h->aux[0], 1ull)] = v;
    }
}

__global__ void k_dvb_merge(const int32_t* __restrict__ off, int64_t m, int64_t cap, const int32_t* __restrict__ vox,
                            const int2* __restrict__ chk, int2* __restrict__ rec) {
    int64_t E = off[m];
    if (E > cap) E = cap;
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < E; p += (int64_t)gridDim.x * blockDim.x) {
        const int32_t v = vox[p];  // any position of a voxel's range holds that voxel
        if ((uint64_t)(uint32_t)v >= (uint64_t)m) continue;
        const int32_t lo = off[v], hi = off[v + 1];
        if (hi - lo <= kDvbChunk) continue;  // done by the rank kernel
        const int2 e = chk[p];
        const int32_t own = lo + ((int32_t)(p - lo) / kDvbChunk) * kDvbChunk;
        int32_t r = (int32_t)(p - own);  // the smaller entries of its own chunk
        for (int32_t c0 = lo; c0 < hi; c0 += kDvbChunk) {
            if (c0 == own) continue;
            // the entries of chunk [c0, c1) below e.x: a lower bound in the sorted chunk
            int32_t a = c0, b = c0 + kDvbChunk < hi ? c0 + kDvbChunk : hi;
            while (a < b) {
                const int32_t mid = (a + b) >> 1;
                if (chk[mid].x < e.x) a = mid + 1;
                else b = mid;
            }
            r += a - c0;
        }
        rec[lo + r] = e;
    }
}

template <int DT, int VEC>
__device__ inline void dvb_load(const void* p, int64_t i, float x[VEC]) {
    if constexpr (VEC == 1) {
        x[0] = ld_feat<DT>(p, i);
    } else if constexpr (DT == SPV_F32) {
        static_assert(VEC == 4, "four fp32 channels per 16 bytes");
        const float4 v = *(const float4*)((const float*)p + i);
        x[0] = v.x;
        x[1] = v.y;
        x[2] = v.z;
        x[3] = v.w;
    } else {
        static_assert(VEC == 8, "eight 16-bit channels per 16 bytes");
        const uint4 v = *(const uint4*)((const uint16_t*)p + i);
        const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            x[2 * j] = from16<DT>(u[j] & 0xffffu);
            x[2 * j + 1] = from16<DT>(u[j] >> 16);
        }
    }
}

// the entries [lo, hi) of one voxel into acc for channels c0 .. c0 + VEC - 1,
// four at a time (the loads first, then the fmas in entry order).  An entry
// past the points (left only by a fill that raised kFlagInternal) reads point
// 0 with weight 0.
template <int DT, int VEC>
__device__ inline void dvb_sum_range(const int2* __restrict__ rec, const void* __restrict__ dout, int64_t n, int C,
                                     int c0, int32_t lo, int32_t hi, float (&acc)[VEC]) {
    int32_t i = lo;
    for (; i + 4 <= hi; i += 4) {
        int2 r[4];
        float x[4][VEC];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            r[u] = rec[i + u];
            if ((uint64_t)(uint32_t)(r[u].x >> 3) >= (uint64_t)n) r[u] = make_int2(0, 0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) dvb_load<DT, VEC>(dout, (int64_t)(r[u].x >> 3) * C + c0, x[u]);
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int c = 0; c < VEC; ++c) acc[c] = fmaf(__int_as_float(r[u].y), x[u][c], acc[c]);
    }
    for (; i < hi; ++i) {
        int2 r = rec[i];
        if ((uint64_t)(uint32_t)(r.x >> 3) >= (uint64_t)n) r = make_int2(0, 0);
        float x[VEC];
        dvb_load<DT, VEC>(dout, (int64_t)(r.x >> 3) * C + c0, x);
#pragma unroll
        for (int c = 0; c < VEC; ++c) acc[c] = fmaf(__int_as_float(r.y), x[c], acc[c]);
    }
}

template <int VEC>
__device__ inline void dvb_store(float* o, const float (&acc)[VEC]) {
    if constexpr (VEC == 1) {
        o[0] = acc[0];
    } else {
#pragma unroll
        for (int c = 0; c < VEC; c += 4) *(float4*)(o + c) = make_float4(acc[c], acc[c + 1], acc[c + 2], acc[c + 3]);
    }
}

// thread per (voxel, VEC consecutive channels) of the voxels of at most
// kDvbLong entries (the others are the long kernel's)
template <int DT, int VEC>
__global__ void k_dvb_gather(const int32_t* __restrict__ off, const int2* __restrict__ rec, const void* __restrict__ dout,
                             int64_t n, int C, int64_t m, float* __restrict__ dv) {
    const int G = C / VEC;
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < m * G; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t v = t / G;
        const int c0 = (int)(t - v * G) * VEC;
        const int32_t lo = off[v], hi = off[v + 1];
        if (hi - lo > kDvbLong) continue;
        float acc[VEC];
#pragma unroll
        for (int c = 0; c < VEC; ++c) acc[c] = 0.f;
        dvb_sum_range<DT, VEC>(rec, dout, n, C, c0, lo, hi, acc);
        dvb_store<VEC>(dv + v * C + c0, acc);
    }
}

// a workgroup per voxel of more than kDvbLong entries (listed by the rank
// kernel): with G channel groups, P = 256 / G parts of the entry range are
// summed by their own threads, each in entry order, and the parts are added
// in part order -- a fixed association for the voxel's length and C
template <int DT, int VEC>
__global__ __launch_bounds__(256) void k_dvb_gather_long(const Header* h, const int32_t* __restrict__ longv, int64_t m,
                                                         const int32_t* __restrict__ off,
                                                         const int2* __restrict__ rec, const void* __restrict__ dout,
                                                         int64_t n, int C, float* __restrict__ dv) {
    __shared__ float red[256][VEC];
    int64_t nl = h->aux[0];
    if (nl > m) nl = m;
    const int G = C / VEC;
    const int P = G >= 256 ? 1 : 256 / G;
    const int q = threadIdx.x / G, g = threadIdx.x - q * G;  // G >= 256: q = 0, g = threadIdx.x
    for (int64_t e = blockIdx.x; e < nl; e += gridDim.x) {
        const int32_t v = longv[e];
        if ((uint64_t)(uint32_t)v >= (uint64_t)m) continue;  // the whole workgroup
        const int32_t lo = off[v], hi = off[v + 1];
        if (G >= 256) {
            for (int gg = threadIdx.x; gg < G; gg += 256) {
                float acc[VEC];
#pragma unroll
                for (int c = 0; c < VEC; ++c) acc[c] = 0.f;
                dvb_sum_range<DT, VEC>(rec, dout, n, C, gg * VEC, lo, hi, acc);
                dvb_store<VEC>(dv + (int64_t)v * C + gg * VEC, acc);
            }
            continue;
        }
        const int32_t len = (hi - lo + P - 1) / P;
        float acc[VEC];
#pragma unroll
        for (int c = 0; c < VEC; ++c) acc[c] = 0.f;
        if (q < P) {
            const int32_t a = lo + q * len, b = a + len < hi ? a + len : hi;
            if (a < b) dvb_sum_range<DT, VEC>(rec, dout, n, C, g * VEC, a, b, acc);
        }
#pragma unroll
        for (int c = 0; c < VEC; ++c) red[threadIdx.x][c] = acc[c];
        __syncthreads();
        if (q == 0) {
            for (int qq = 1; qq < P; ++qq)
#pragma unroll
                for (int c = 0; c < VEC; ++c) acc[c] += red[qq * G + g][c];
            dvb_store<VEC>(dv + (int64_t)v * C + g * VEC, acc);
        }
        __syncthreads();
    }
}

template <int DT, int VEC>
static void launch_dvb_gather(hipStream_t s, const DvbWs& w, const void* dout, int64_t n, int C, int64_t m,
                              float* dv) {
    int64_t g = blocks_for(m * (C / VEC), 256);
    if (g > 16384) g = 16384;
    k_dvb_gather<DT, VEC><<<(unsigned)g, 256, 0, s>>>(w.off, w.rec, dout, n, C, m, dv);
    const int64_t gl = m < 1024 ? m : 1024;
    k_dvb_gather_long<DT, VEC><<<(unsigned)gl, 256, 0, s>>>(w.h, w.longv, m, w.off, w.rec, dout, n, C, dv);
}

void launch_devoxelize_backward(hipStream_t s, const DvbWs& w, const int32_t* cidx, const float* cw, const void* dout,
                                int64_t n, int C, float* dv, int64_t m, int dt) {
    int64_t gz = blocks_for(m + 1, 256 * 4);
    if (gz > 4096) gz = 4096;
    k_dvb_zero<<<(unsigned)gz, 256, 0, s>>>(w.h, w.cnt, m + 1);
    if (m == 0) return;
    if (n > 0) k_dvb_count<<<blocks_for(n, kDvbThreads), kDvbThreads, 0, s>>>(cidx, cw, n, m, w.h, w.cnt, w.slot);
    launch_exclusive_scan(s, w.cnt, w.off, nullptr, m, w.tmp);
    if (n > 0) {
        int64_t gp = blocks_for(n, 256);
        if (gp > 8192) gp = 8192;
        k_dvb_fill<<<(unsigned)gp, 256, 0, s>>>(cidx, cw, n, m, w.h, w.slot, w.off, w.ent, w.coef, w.vox);
        int64_t gr = blocks_for(8 * n, 256);
        if (gr > 16384) gr = 16384;
        k_dvb_rank<<<(unsigned)gr, 256, 0, s>>>(w.off, m, 8 * n, w.ent, w.coef, w.vox, w.rec, w.chk, w.h, w.longv);
        k_dvb_merge<<<(unsigned)gr, 256, 0, s>>>(w.off, m, 8 * n, w.vox, w.chk, w.rec);
    }
    const bool vec = (((uintptr_t)dout | (uintptr_t)dv) & 15u) == 0;
    if (dt == SPV_F32) {
        if (vec && C % 4 == 0) launch_dvb_gather<SPV_F32, 4>(s, w, dout, n, C, m, dv);
        else launch_dvb_gather<SPV_F32, 1>(s, w, dout, n, C, m, dv);
    } else if (dt == SPV_BF16) {
        if (vec && C % 8 == 0) launch_dvb_gather<SPV_BF16, 8>(s, w, dout, n, C, m, dv);
        else launch_dvb_gather<SPV_BF16, 1>(s, w, dout, n, C, m, dv);
    } else {
        if (vec && C % 8 == 0) launch_dvb_gather<SPV_F16, 8>(s, w, dout, n, C, m, dv);
        else launch_dvb_gather<SPV_F16, 1>(s, w, dout, n, C, m, dv);
    }
}

}  // namespace spv
