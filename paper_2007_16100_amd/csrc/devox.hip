// devox.hip -- sparse devoxelization (Sec. 3.3 "Sparse Devoxelization": trilinear
// interpolation from the 8 neighbouring voxels, looked up in the voxel hash) fused
// with the point-branch MLP and the fusion by addition ("Point Transformation and
// Feature Fusion").
//
// MFMA path (bf16/f16): a wave owns 16 points.  Each lane computes two of the
// 8 corners of one point (hash probes + raw trilinear weights), the weights are
// renormalized over the present corners with two cross-lane sums, the point MLP
// runs as a 16 x C x Cp MFMA GEMM with the point rows as the A operand, and the
// epilogue blends the 8 corner rows into each output element before the single
// write of the fused result.
#include "spv_internal.hpp"

namespace spv {

// corner geometry of one point; the float arithmetic is kept in this exact order
// (no contraction) so corner indices and raw weights are reproducible bit for bit
struct Corners {
    int b;
    int base[3];
    float t[3];
    bool ok;
};

#pragma clang fp contract(off)
__device__ inline Corners corners_of(const float (&p)[3], int b, float v, float sfac, int mode) {
    Corners c;
    c.b = b;
    c.ok = c.b >= 0 && c.b <= kBatchMax;
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        const float x = p[d];
        const float a = x / v;  // the same quantity as Eq. 1 before the floor
        const float fa = floorf(a);
        c.ok = c.ok && isfinite(x) && isfinite(a) && fa >= (float)kCoordMin && fa <= (float)kCoordMax;
        const float as = a * sfac;  // exact scaling by 2^-stride_log2
        const float u = (mode == SPV_DEVOX_CENTER) ? as - 0.5f : as;
        const float fb = floorf(u);
        c.base[d] = c.ok ? (int)fb : 0;
        // NEAREST: the voxel containing the point (corner 0) takes all the weight
        c.t[d] = (c.ok && mode != SPV_DEVOX_NEAREST) ? u - fb : 0.f;
    }
    return c;
}
__device__ inline Corners point_corners(const float* xyz, const int32_t* batch, int64_t k, float v, float sfac,
                                        int mode) {
    const float p[3] = {xyz[3 * k], xyz[3 * k + 1], xyz[3 * k + 2]};
    return corners_of(p, batch ? batch[k] : 0, v, sfac, mode);
}

__device__ inline float corner_weight(const Corners& c, int cc) {
    const int cx = (cc >> 2) & 1, cy = (cc >> 1) & 1, cz = cc & 1;
    const float wx = cx ? c.t[0] : 1.0f - c.t[0];
    const float wy = cy ? c.t[1] : 1.0f - c.t[1];
    const float wz = cz ? c.t[2] : 1.0f - c.t[2];
    float w = wx * wy;
    w = w * wz;
    return w;
}
#pragma clang fp contract(on)

__device__ inline int32_t corner_lookup(Table t, const Corners& c, int cc) {
    if (!c.ok) return -1;
    return table_find(t, pack_key(c.b, c.base[0] + ((cc >> 2) & 1), c.base[1] + ((cc >> 1) & 1), c.base[2] + (cc & 1)));
}

// ---------------------------------------------------------------------------
// generic path: corners per point, then one thread per output element
// ---------------------------------------------------------------------------
__global__ void k_devox_corners(DevoxArgs a, int32_t* cidx, float* cw) {
    int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (k >= a.n) return;
    const float sfac = __builtin_ldexpf(1.0f, -a.stride_log2);
    Corners c = point_corners(a.xyz, a.batch, k, a.voxel_size, sfac, a.mode);
    if (!c.ok) raise_flag(a.h, isfinite(a.xyz[3 * k]) && isfinite(a.xyz[3 * k + 1]) && isfinite(a.xyz[3 * k + 2])
                                   ? kFlagRange
                                   : kFlagNonfinite);
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
        cidx[8 * k + cc] = corner_lookup(a.table, c, cc);
        cw[8 * k + cc] = c.ok ? corner_weight(c, cc) : 0.f;
    }
}

template <int DT>
__global__ void k_devox_generic(DevoxArgs a, const int32_t* cidx, const float* cw) {
    int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t k = t / a.C;
    int col = (int)(t - k * a.C);
    if (k >= a.n) return;
    float den = 0.f, num = 0.f;
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
        int32_t i = cidx[8 * k + cc];
        if (i < 0) continue;
        float w = cw[8 * k + cc];
        den += w;
        num += w * ld_feat<DT>(a.vfeat, (int64_t)i * a.C + col);
    }
    float y = den > 0.f ? num / den : 0.f;
    if (a.pfeat) {
        float s = 0.f;
        for (int ci = 0; ci < a.Cp; ++ci)
            s += ld_feat<DT>(a.pfeat, k * a.Cp + ci) * ld_feat<DT>(a.Wp, (int64_t)ci * a.C + col);
        if (a.scale_p) s *= a.scale_p[col];
        if (a.shift_p) s += a.shift_p[col];
        if (a.relu_p) s = fmaxf(s, 0.f);
        y += s;
    }
    st_feat<DT>(a.out, k * a.C + col, y);
}

// ---------------------------------------------------------------------------
// MFMA path: a wave owns PB blocks of 16 points.
//  1. corner probes of all its points issued together (lane (r16, g) takes
//     corners 2g, 2g+1 of point r16 of each block), weights renormalized over
//     the present corners, kept in LDS;
//  2. point MLP D = Wp^T P^T on matrix cores (Wp fragments staged once per
//     workgroup in LDS): lane (r16, g) ends with channels nb*16 + 4g .. 4g+3 of
//     point r16, activated and parked in an LDS row tile;
//  3. blend: one lane per (point, 8-channel chunk) gathers that chunk of the 8
//     corner voxels (16-byte loads), adds the MLP row chunk and writes the
//     fused 16 bytes once.
// ---------------------------------------------------------------------------
constexpr int kDevoxPB = 4;  // 16-point blocks per wave

// NBR: corners read from the grid's neighbour table (a.nbr), else probed
template <int DT, int KCH, int NB, bool NBR>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_devox_mfma(DevoxArgs a,
                                                                                            const uint4* __restrict__ wpack) {
    constexpr int PB = kDevoxPB;
    constexpr int C = NB * 16;
    // above 128 channels the row tile holds half the channels at a time (LDS for
    // two workgroups per CU) and each lane keeps the corner rows of 2 of its
    // tasks in flight at once instead of all of them
    constexpr int HV = NB > 8 ? 2 : 1;
    constexpr int CH = C / HV;   // channels per half
    constexpr int NCH = CH / 8;  // 16-byte chunks per half row
    __shared__ __align__(16) uint4 wl[KCH * NB * 64];
    __shared__ __align__(16) int32_t sidx[4][PB * 16][8];
    __shared__ __align__(16) float sw[4][PB * 16][8];
    __shared__ __align__(16) float ys[4][16][CH + 4];
    __shared__ float ssc[C], ssh[C];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r16 = lane & 15, g = lane >> 4;
    const int64_t p0 = ((int64_t)blockIdx.x * 4 + wave) * (PB * 16);
    const float sfac = __builtin_ldexpf(1.0f, -a.stride_log2);
    const bool mlp = a.pfeat != nullptr;

    // Wp fragments, scale and shift into LDS (the whole workgroup)
    if (mlp) {
        for (int f = threadIdx.x; f < KCH * NB * 64; f += blockDim.x) wl[f] = wpack[f];
        for (int c = threadIdx.x; c < C; c += blockDim.x) {
            ssc[c] = a.scale_p ? a.scale_p[c] : 1.f;
            ssh[c] = a.shift_p ? a.shift_p[c] : 0.f;
        }
    }

    // 1. corners: coordinates of the wave's points loaded together, then the
    // probes of all its blocks together
    float px[PB][3];
    int pb[PB];
#pragma unroll
    for (int b = 0; b < PB; ++b) {
        const int64_t k = p0 + b * 16 + r16;
        const int64_t kc = k < a.n ? k : 0;
#pragma unroll
        for (int d = 0; d < 3; ++d) px[b][d] = a.xyz[3 * kc + d];
        pb[b] = a.batch ? a.batch[kc] : 0;
    }
    Corners cn[PB];
    uint64_t key[2 * PB];
    bool act[2 * PB];
    int32_t idx[2 * PB];
#pragma unroll
    for (int b = 0; b < PB; ++b) {
        const int64_t k = p0 + b * 16 + r16;
        cn[b] = corners_of(px[b], pb[b], a.voxel_size, sfac, a.mode);
        if (k >= a.n) cn[b].ok = false;
        if (k < a.n && !cn[b].ok && g == 0)
            raise_flag(a.h, isfinite(px[b][0]) && isfinite(px[b][1]) && isfinite(px[b][2]) ? kFlagRange
                                                                                        : kFlagNonfinite);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int cc = 2 * g + h;
            act[2 * b + h] = cn[b].ok;
            key[2 * b + h] = pack_key(cn[b].b, cn[b].base[0] + ((cc >> 2) & 1), cn[b].base[1] + ((cc >> 1) & 1),
                                      cn[b].base[2] + (cc & 1));
        }
    }
    if constexpr (NBR) {
        // the grid is the points' own voxelization with its 3x3x3 neighbour
        // table: every corner lies in the neighbourhood of the point's voxel j,
        // so corner c is entry 9(dx+1) + 3(dy+1) + (dz+1) of row j, with
        // d = base + c - (voxel j's coordinates) in {-1, 0, 1} per axis
        // rows of the grid that exist: the live count when given, else the capacity
        int64_t rows = a.nbr_rows;
        if (a.nbr_m_dev) {
            const int64_t md = *a.nbr_m_dev;
            rows = md < 0 ? 0 : (md < rows ? md : rows);
        }
        int32_t j[PB];
#pragma unroll
        for (int b = 0; b < PB; ++b) {
            const int64_t k = p0 + b * 16 + r16;
            j[b] = (cn[b].ok && k < a.n) ? a.pt2vox[k] : -1;
            if (j[b] >= rows) j[b] = -1;
        }
        int own[PB][3];
#pragma unroll
        for (int b = 0; b < PB; ++b)
#pragma unroll
            for (int d = 0; d < 3; ++d) own[b][d] = j[b] >= 0 ? a.grid_coords[4 * (int64_t)j[b] + 1 + d] : 0;
#pragma unroll
        for (int b = 0; b < PB; ++b) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int cc = 2 * g + h;
                const int dx = cn[b].base[0] + ((cc >> 2) & 1) - own[b][0];
                const int dy = cn[b].base[1] + ((cc >> 1) & 1) - own[b][1];
                const int dz = cn[b].base[2] + (cc & 1) - own[b][2];
                const bool in = j[b] >= 0 && dx >= -1 && dx <= 1 && dy >= -1 && dy <= 1 && dz >= -1 && dz <= 1;
                idx[2 * b + h] = in ? a.nbr[27 * (int64_t)j[b] + 9 * (dx + 1) + 3 * (dy + 1) + (dz + 1)] - 1 : -1;
                // outside the neighbourhood (not expected): the hash decides
                if (act[2 * b + h] && !in) idx[2 * b + h] = table_find(a.table, key[2 * b + h]);
            }
        }
    } else {
        table_find_n<2 * PB>(a.table, key, act, idx);
    }
#pragma unroll
    for (int b = 0; b < PB; ++b) {
        const int64_t k = p0 + b * 16 + r16;
        const int32_t i0 = idx[2 * b], i1 = idx[2 * b + 1];
        const float w0 = cn[b].ok ? corner_weight(cn[b], 2 * g) : 0.f;
        const float w1 = cn[b].ok ? corner_weight(cn[b], 2 * g + 1) : 0.f;
        if (k < a.n && a.corner_idx) {
            a.corner_idx[8 * k + 2 * g] = i0;
            a.corner_idx[8 * k + 2 * g + 1] = i1;
            a.corner_w[8 * k + 2 * g] = w0;
            a.corner_w[8 * k + 2 * g + 1] = w1;
        }
        float wp = (i0 >= 0 ? w0 : 0.f) + (i1 >= 0 ? w1 : 0.f);
        wp += __shfl_xor(wp, 16, 64);
        wp += __shfl_xor(wp, 32, 64);
        const float inv = wp > 0.f ? 1.0f / wp : 0.f;
        sidx[wave][b * 16 + r16][2 * g] = i0;
        sidx[wave][b * 16 + r16][2 * g + 1] = i1;
        sw[wave][b * 16 + r16][2 * g] = (i0 >= 0) ? w0 * inv : 0.f;
        sw[wave][b * 16 + r16][2 * g + 1] = (i1 >= 0) ? w1 * inv : 0.f;
    }

    __syncthreads();  // Wp fragments in LDS

    const uint16_t* V = (const uint16_t*)a.vfeat;
    uint16_t* out = (uint16_t*)a.out;
    // point rows for the MLP: B operand, lane (r16, g) = point r16, channels kc*32 + 8g ..
    auto load_p = [&](int b, i32x4v (&pv)[KCH]) __attribute__((always_inline)) {
        const int64_t k = p0 + b * 16 + r16;
        const uint16_t* prow = (const uint16_t*)a.pfeat + (k < a.n ? k : 0) * a.Cp + 8 * g;
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc) {
            pv[kc] = i32x4v{0, 0, 0, 0};
            if (mlp && k < a.n && kc * 32 + 8 * g < a.Cp) pv[kc] = *(const i32x4v*)(prow + kc * 32);
        }
    };
    i32x4v pv[2][KCH];
    load_p(0, pv[0]);
#pragma unroll
    for (int b = 0; b < PB; ++b) {
        if (b + 1 < PB) load_p(b + 1, pv[(b + 1) & 1]);
        f32x4 acc[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (mlp) {
#pragma unroll
            for (int kc = 0; kc < KCH; ++kc) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    acc[nb] = mfma16x16x32<DT>(wl[(kc * NB + nb) * 64 + lane], __builtin_bit_cast(uint4, pv[b & 1][kc]),
                                               acc[nb]);
            }
        }
#pragma unroll
        for (int hv = 0; hv < HV; ++hv) {
            // 2. activated MLP rows of block b (this half's channels) into the wave's row tile
#pragma unroll
            for (int nb = hv * (NB / HV); nb < (hv + 1) * (NB / HV); ++nb) {
                float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
                if (mlp) {
                    const int col = nb * 16 + 4 * g;
                    float sc[4], sh[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        sc[e] = ssc[col + e];
                        sh[e] = ssh[col + e];
                    }
                    y.x = acc[nb][0] * sc[0] + sh[0];
                    y.y = acc[nb][1] * sc[1] + sh[1];
                    y.z = acc[nb][2] * sc[2] + sh[2];
                    y.w = acc[nb][3] * sc[3] + sh[3];
                    if (a.relu_p) {
                        y.x = fmaxf(y.x, 0.f);
                        y.y = fmaxf(y.y, 0.f);
                        y.z = fmaxf(y.z, 0.f);
                        y.w = fmaxf(y.w, 0.f);
                    }
                }
                *(float4*)&ys[wave][r16][nb * 16 - hv * CH + 4 * g] = y;
            }
            __builtin_amdgcn_wave_barrier();
            // 3. blend: tasks (point, chunk) of block b; the corner rows of a group of
            // a lane's tasks are requested before any of them is used
            constexpr int NT = (16 * NCH + 63) / 64;
            constexpr int G = HV > 1 ? 2 : NT;
#pragma unroll
            for (int j0 = 0; j0 < NT; j0 += G) {
                int32_t ci[G][8];
                float cw[G][8];
                uint4 v[G][8];
#pragma unroll
                for (int j = 0; j < G; ++j) {
                    const int t = lane + 64 * (j0 + j);
                    const int pt = (t < 16 * NCH ? t : 0) / NCH, ch = (t < 16 * NCH ? t : 0) % NCH;
                    const i32x4v ia = *(const i32x4v*)&sidx[wave][b * 16 + pt][0];
                    const i32x4v ib = *(const i32x4v*)&sidx[wave][b * 16 + pt][4];
                    const float4 wa = *(const float4*)&sw[wave][b * 16 + pt][0];
                    const float4 wb = *(const float4*)&sw[wave][b * 16 + pt][4];
                    const int32_t ii[8] = {ia.x, ia.y, ia.z, ia.w, ib.x, ib.y, ib.z, ib.w};
                    const float ww[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
#pragma unroll
                    for (int cc = 0; cc < 8; ++cc) {
                        ci[j][cc] = t < 16 * NCH ? ii[cc] : -1;
                        cw[j][cc] = ww[cc];
                        v[j][cc] = make_uint4(0, 0, 0, 0);
                        if (ci[j][cc] >= 0) v[j][cc] = *(const uint4*)(V + (int64_t)ci[j][cc] * C + hv * CH + ch * 8);
                    }
                }
#pragma unroll
                for (int j = 0; j < G; ++j) {
                    const int t = lane + 64 * (j0 + j);
                    if (t >= 16 * NCH) break;
                    const int pt = t / NCH, ch = t - pt * NCH;
                    const int64_t k = p0 + b * 16 + pt;
                    float dv[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) dv[e] = 0.f;
#pragma unroll
                    for (int cc = 0; cc < 8; ++cc) {
                        if (ci[j][cc] < 0) continue;
                        const uint32_t u[4] = {v[j][cc].x, v[j][cc].y, v[j][cc].z, v[j][cc].w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            dv[2 * e] += cw[j][cc] * from16<DT>(u[e] & 0xFFFF);
                            dv[2 * e + 1] += cw[j][cc] * from16<DT>(u[e] >> 16);
                        }
                    }
                    const float4 y0 = *(const float4*)&ys[wave][pt][ch * 8];
                    const float4 y1 = *(const float4*)&ys[wave][pt][ch * 8 + 4];
                    const float yy[8] = {y0.x, y0.y, y0.z, y0.w, y1.x, y1.y, y1.z, y1.w};
                    uint32_t o[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        o[e] = (uint32_t)to16<DT>(yy[2 * e] + dv[2 * e]) |
                               ((uint32_t)to16<DT>(yy[2 * e + 1] + dv[2 * e + 1]) << 16);
                    if (k < a.n) *(uint4*)(out + k * C + hv * CH + ch * 8) = make_uint4(o[0], o[1], o[2], o[3]);
                }
            }
            __builtin_amdgcn_wave_barrier();
        }
    }
}

// 16-bit features, C in {16, 32, 64, 96, 128, 256} and Cp <= 128 (LDS: the Wp
// fragments plus each wave's row tile); everything else takes the generic path
bool devox_mfma_supported(int C, int Cp, int dt) {
    if (dt == SPV_F32 || C % 16 != 0) return false;
    int NB = C / 16;
    if (!(NB == 1 || NB == 2 || NB == 4 || NB == 6 || NB == 8 || NB == 16)) return false;
    return Cp == 0 || (Cp % 8 == 0 && Cp <= 128);
}

void* plan_devox_ws(Arena& a, int C, int Cp) {
    int KCH = (Cp + 31) / 32, NB = C / 16;
    if (KCH < 1) KCH = 1;
    if (NB < 1) NB = 1;
    return a.take<uint4>((size_t)KCH * NB * 64);
}

template <int DT, int KCH, int NB>
static void launch_devox_mfma(hipStream_t s, const DevoxArgs& a, const void* wpack) {
    int64_t waves = (a.n + 16 * kDevoxPB - 1) / (16 * kDevoxPB);
    if (a.nbr && a.pt2vox && a.grid_coords)
        k_devox_mfma<DT, KCH, NB, true><<<blocks_for(waves, 4), 256, 0, s>>>(a, (const uint4*)wpack);
    else
        k_devox_mfma<DT, KCH, NB, false><<<blocks_for(waves, 4), 256, 0, s>>>(a, (const uint4*)wpack);
}

template <int DT, int NB>
static void launch_devox_kch(hipStream_t s, const DevoxArgs& a, const void* wpack) {
    switch (a.pfeat ? (a.Cp + 31) / 32 : 0) {
        case 0:
        case 1: launch_devox_mfma<DT, 1, NB>(s, a, wpack); break;
        case 2: launch_devox_mfma<DT, 2, NB>(s, a, wpack); break;
        case 3: launch_devox_mfma<DT, 3, NB>(s, a, wpack); break;
        case 4: launch_devox_mfma<DT, 4, NB>(s, a, wpack); break;
    }
}

template <int DT>
static void launch_devox_dt(hipStream_t s, const DevoxArgs& a, const void* wpack) {
    switch (a.C / 16) {
        case 1: launch_devox_kch<DT, 1>(s, a, wpack); break;
        case 2: launch_devox_kch<DT, 2>(s, a, wpack); break;
        case 4: launch_devox_kch<DT, 4>(s, a, wpack); break;
        case 6: launch_devox_kch<DT, 6>(s, a, wpack); break;
        case 8: launch_devox_kch<DT, 8>(s, a, wpack); break;
        case 16: launch_devox_kch<DT, 16>(s, a, wpack); break;
    }
}

__global__ void k_pack_wp(const uint16_t* W, int Cin, int Cout, int KCH, int NB, uint4* wpack);

// the point-MLP weight [Cp][C] packed like a single-offset conv weight, when
// the MFMA kernel runs with point features
PackJob devox_pack_job(const DevoxArgs& a, void* wpack) {
    PackJob q{(const uint16_t*)a.Wp, (uint4*)wpack, 1, a.Cp, a.C, 0, 0, 0, a.C, (int64_t)a.Cp * a.C, 1};
    if (a.n <= 0 || !a.pfeat || !devox_mfma_supported(a.C, a.Cp, a.dt)) return q;
    q.KCH = (a.Cp + 31) / 32;
    q.NB = a.C / 16;
    q.total = (int64_t)q.KCH * q.NB * 64;
    return q;
}

void launch_devox(hipStream_t s, const DevoxArgs& a, void* wpack, int32_t* cidx_tmp, float* cw_tmp, bool wp_packed) {
    if (a.n <= 0) return;
    if (devox_mfma_supported(a.C, a.pfeat ? a.Cp : 0, a.dt)) {
        if (a.pfeat && !wp_packed) {
            int KCH = (a.Cp + 31) / 32, NB = a.C / 16;
            int64_t tot = (int64_t)KCH * NB * 64;
            k_pack_wp<<<blocks_for(tot, 256), 256, 0, s>>>((const uint16_t*)a.Wp, a.Cp, a.C, KCH, NB, (uint4*)wpack);
        }
        if (a.dt == SPV_BF16) launch_devox_dt<SPV_BF16>(s, a, wpack);
        else launch_devox_dt<SPV_F16>(s, a, wpack);
        return;
    }
    int32_t* ci = a.corner_idx ? a.corner_idx : cidx_tmp;
    float* cw = a.corner_w ? a.corner_w : cw_tmp;
    k_devox_corners<<<blocks_for(a.n, 256), 256, 0, s>>>(a, ci, cw);
    unsigned g = blocks_for(a.n * a.C, 256);
    if (a.dt == SPV_F32) k_devox_generic<SPV_F32><<<g, 256, 0, s>>>(a, ci, cw);
    else if (a.dt == SPV_BF16) k_devox_generic<SPV_BF16><<<g, 256, 0, s>>>(a, ci, cw);
    else k_devox_generic<SPV_F16><<<g, 256, 0, s>>>(a, ci, cw);
}

// the point-MLP weight [Cin][Cout] packed like a single-offset conv weight
__global__ void k_pack_wp(const uint16_t* W, int Cin, int Cout, int KCH, int NB, uint4* wpack) {
    int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t total = (int64_t)KCH * NB * 64;
    if (t >= total) return;
    int lane = (int)(t & 63);
    int64_t f = t >> 6;
    int nb = (int)(f % NB);
    int kc = (int)(f / NB);
    int col = nb * 16 + (lane & 15);
    int ci0 = kc * 32 + 8 * (lane >> 4);
    uint32_t w[4];
    for (int e = 0; e < 4; ++e) {
        uint32_t lo = 0, hi = 0;
        int c0 = ci0 + 2 * e, c1 = ci0 + 2 * e + 1;
        if (c0 < Cin) lo = W[(int64_t)c0 * Cout + col];
        if (c1 < Cin) hi = W[(int64_t)c1 * Cout + col];
        w[e] = lo | (hi << 16);
    }
    wpack[t] = make_uint4(w[0], w[1], w[2], w[3]);
}

}  // namespace spv
