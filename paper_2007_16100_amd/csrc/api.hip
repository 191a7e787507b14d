// api.hip -- the extern "C" entry points of libspv.so: argument validation,
// workspace layout and the launch sequences of each operation of the SPVConv
// hot path (Sec. 3.3 and Fig. 2 of the paper).  No entry point allocates memory
// or synchronizes unless a host read-back pointer is given.
#include <math.h>
#include <string.h>

#include <mutex>

#include "conv_common.hpp"

using namespace spv;

// Device-resident scratch of spv_sparse_conv_nbr_noalloc: the packed weights of
// one layer, up to 256 -> 256 channels (27 offsets x 8 input slabs x 16 output
// blocks x 64 lanes x 16 bytes).  Each device holds its own copy for the
// lifetime of the process; calls on one device share it.
constexpr size_t kNoAllocScratchBytes = (size_t)27 * 8 * 16 * 64 * 16;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

thread_local int g_last_hip_error = 0;

spv_status hip_check() {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return SPV_ERR_HIP;
    }
    return SPV_OK;
}

spv_status flags_to_status(uint32_t f) {
    if (f & kFlagNonfinite) return SPV_ERR_NONFINITE;
    if (f & kFlagRange) return SPV_ERR_RANGE;
    if (f & (kFlagCapacity | kFlagTableFull)) return SPV_ERR_CAPACITY;
    if (f & (kFlagDuplicate | kFlagUnsorted)) return SPV_ERR_INVALID_ARG;
    if (f & kFlagInternal) return SPV_ERR_HIP;
    return SPV_OK;
}

// synchronize and return the device status (and optionally the header)
spv_status sync_status(hipStream_t s, const Header* h, Header* out) {
    Header tmp;
    if (hipMemcpyAsync(&tmp, h, sizeof(Header), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return hip_check() == SPV_OK ? SPV_ERR_HIP : SPV_ERR_HIP;
    if (out) *out = tmp;
    return flags_to_status(tmp.status);
}

bool valid_dt(int dt) { return dt == SPV_F32 || dt == SPV_BF16 || dt == SPV_F16; }
// a workspace pointer every layout can carve from (its offsets are 256-byte multiples)
bool ws_ok(const void* ws) { return ws && ((uintptr_t)ws & 255u) == 0; }
size_t esize(int dt) { return dt == SPV_F32 ? 4 : 2; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
constexpr int kUpChildren = 8;  // offsets of a k=2 s=2 map
bool valid_v(float v) { return isfinite(v) && v > 0.0f; }

// --- workspace layouts (a null base gives the size) -----------------------------
// A call that records device-detected errors and has nothing to compute still
// clears the status word (at workspace offset 0), as its launches would.
static spv_status clear_status_only(hipStream_t s, void* ws) {
    launch_clear_header(s, (Header*)ws);
    return hip_check();
}

struct VoxLayout {
    Header* h;
    VoxelizeWs w;
};
size_t layout_voxelize(void* ws, size_t bytes, int64_t n, VoxLayout& L) {
    Arena a(ws, bytes);
    L.h = a.take<Header>(1);
    plan_voxelize_ws(a, L.w, n);
    L.w.h = L.h;
    return a.used;
}

struct MapLayout {
    Header* h;
    KmapWs w;
};
size_t layout_kmap(void* ws, size_t bytes, int64_t m_cap, int K, int stride, MapLayout& L) {
    Arena a(ws, bytes);
    L.h = a.take<Header>(1);
    plan_kmap_ws(a, L.w, m_cap, K, stride, true, true);
    L.w.h = L.h;
    return a.used;
}

struct ConvLayout {
    Header* h;
    ConvPlan p;
    void* wpack;
};
size_t layout_conv(void* ws, size_t bytes, int64_t m_out_cap, int K3, int Cin, int Cout, int dt, ConvLayout& L,
                   int64_t in_rows, bool sparse_transposed = false) {
    Arena a(ws, bytes);
    L.h = a.take<Header>(1);
    plan_conv_ws(a, L.p, m_out_cap, K3, Cin, Cout, dt, in_rows, sparse_transposed);
    L.p.h = L.h;
    L.wpack = plan_wpack_ws(a, K3, Cin, Cout > 16 ? Cout : 16);
    return a.used;
}

// every layout starts with the status header, which calls that record no device
// errors leave untouched
size_t layout_linear(void* ws, size_t bytes, int Cin, int Cout, void** wpack) {
    Arena a(ws, bytes);
    a.take<Header>(1);
    *wpack = plan_linear_ws(a, Cin, Cout);
    return a.used;
}

struct DevoxLayout {
    Header* h;
    Table t;
    void* wpack;
    int32_t* cidx;
    float* cw;
};
size_t layout_devox(void* ws, size_t bytes, int64_t m_cap, int64_t n, int C, int Cp, DevoxLayout& L) {
    Arena a(ws, bytes);
    L.h = a.take<Header>(1);
    uint32_t S = table_capacity(m_cap > 0 ? m_cap : 1);
    L.t = take_table(a, S);
    L.wpack = plan_devox_ws(a, C, Cp);
    int64_t nn = n > 0 ? n : 1;
    L.cidx = a.take<int32_t>(8 * nn);
    L.cw = a.take<float>(8 * nn);
    return a.used;
}

struct BlockLayout {
    Header* h;
    VoxelizeWs vox;
    KmapWs map;
    ConvPlan plan;
    int32_t* coords;
    int32_t* counts;
    int32_t* pt2vox;
    int64_t* m_dev;
    void* va;
    void* vb;
    void* vc;
    int32_t* off;
    int32_t* pairs;
    int64_t pair_cap;
    void* wpack_conv[2];
    void* wpack_mlp;
    int32_t* cidx;
    float* cw;
};
size_t layout_block(void* ws, size_t bytes, int64_t n, int C, int dt, BlockLayout& L) {
    Arena a(ws, bytes);
    const int64_t nn = n > 0 ? n : 1;
    L.h = a.take<Header>(1);
    plan_voxelize_ws(a, L.vox, nn);
    L.vox.h = L.h;
    L.map.h = L.h;
    L.map.fine = L.vox.table;  // the voxelization's table serves the kernel map and the devoxelization
    plan_kmap_ws(a, L.map, nn, 3, 1, false, false);
    plan_conv_ws(a, L.plan, nn, 27, C, C, dt, nn);
    L.plan.h = L.h;
    L.map.nbr = L.plan.nbr;  // the map's neighbour table is the 3x3x3 conv's plan
    L.coords = a.take<int32_t>(4 * nn);
    L.counts = a.take<int32_t>(nn);
    L.pt2vox = a.take<int32_t>(nn);
    L.m_dev = a.take<int64_t>(1);
    L.va = a.take<char>((size_t)nn * C * esize(dt));
    L.vb = a.take<char>((size_t)nn * C * esize(dt));
    L.vc = a.take<char>((size_t)nn * C * esize(dt));  // a residual block's last output (its input stays in va)
    L.off = a.take<int32_t>(28);
    L.pair_cap = 27 * nn;
    L.pairs = a.take<int32_t>(2 * L.pair_cap);
    L.wpack_conv[0] = plan_wpack_ws(a, 27, C, C > 16 ? C : 16);
    L.wpack_conv[1] = plan_wpack_ws(a, 27, C, C > 16 ? C : 16);
    L.wpack_mlp = plan_devox_ws(a, C, C);
    L.cidx = a.take<int32_t>(8 * nn);
    L.cw = a.take<float>(8 * nn);
    return a.used;
}

spv_status need(size_t needed, size_t have) { return needed <= have ? SPV_OK : SPV_ERR_CAPACITY; }

}  // namespace

extern "C" {

size_t spv_workspace_bytes(int64_t max_points, int32_t max_C) {
    if (max_points < 0) max_points = 0;
    if (max_C < 16) max_C = 16;
    VoxLayout v;
    MapLayout m;
    ConvLayout c;
    DevoxLayout d;
    size_t s = layout_voxelize(nullptr, 0, max_points, v);
    s = std::max(s, layout_kmap(nullptr, 0, max_points, 3, 1, m));
    s = std::max(s, layout_kmap(nullptr, 0, max_points, 2, 2, m));
    s = std::max(s, layout_kmap(nullptr, 0, max_points, 3, 2, m));
    s = std::max(s, layout_conv(nullptr, 0, max_points, 27, max_C, max_C, SPV_BF16, c, max_points));
    void* wl = nullptr;
    s = std::max(s, layout_linear(nullptr, 0, max_C, max_C, &wl));

    s = std::max(s, layout_devox(nullptr, 0, max_points, max_points, max_C, max_C, d));
    return s;
}

size_t spv_wgrad_workspace_bytes(int32_t K3, int32_t Cin, int32_t Cout) {
    if (K3 <= 0 || Cin <= 0 || Cout <= 0) return 0;
    Arena a(nullptr, 0);
    a.take<Header>(1);
    plan_wgrad_ws(a, K3, Cin, Cout);
    return a.used;
}

size_t spv_block_workspace_bytes(int64_t max_points, int32_t C) {
    BlockLayout L;
    return layout_block(nullptr, 0, max_points < 0 ? 0 : max_points, C < 16 ? 16 : C, SPV_F32, L);
}

const char* spv_status_string(spv_status s) {
    switch (s) {
        case SPV_OK: return "ok";
        case SPV_ERR_INVALID_ARG: return "invalid argument";
        case SPV_ERR_CAPACITY: return "capacity too small";
        case SPV_ERR_RANGE: return "coordinate out of range";
        case SPV_ERR_NONFINITE: return "non-finite coordinate";
        case SPV_ERR_UNSUPPORTED: return "unsupported";
        case SPV_ERR_HIP: return "HIP runtime error";
    }
    return "unknown";
}

int spv_last_hip_error(void) { return g_last_hip_error; }

spv_status spv_status_check(const void* ws, void* stream) {
    if (!ws_ok(ws)) return SPV_ERR_INVALID_ARG;
    return sync_status((hipStream_t)stream, (const Header*)ws, nullptr);
}

int32_t spv_conv_kernel(int32_t K3, int32_t Cin, int32_t Cout, spv_dtype dt, int64_t in_rows, int64_t m_out_cap,
                        int64_t pair_cap, int32_t transposed) {
    if (!(K3 == 27 || K3 == 8) || Cin <= 0 || Cout <= 0 || !valid_dt(dt) || in_rows < 0 || m_out_cap < 0 ||
        pair_cap < 0)
        return -1;
    return conv_kernel_choice(K3, Cin, Cout, dt, m_out_cap > 0 ? m_out_cap : 1, in_rows, pair_cap,
                              transposed && in_rows != m_out_cap);
}

int32_t spv_block_conv_kernel(int64_t n, int32_t C, spv_dtype dt) {
    if (n < 0 || C <= 0 || !valid_dt(dt)) return -1;
    // the block's plan makes this choice (its pair list holds 27 n pairs)
    const int64_t nn = n > 0 ? n : 1;
    return conv_kernel_choice(27, C, C, dt, nn, nn, 27 * nn, false);
}

spv_status spv_voxelize(void* stream, void* ws, size_t ws_bytes, const float* xyz, const int32_t* batch, int64_t n,
                        float voxel_size, const void* feat, int32_t C, spv_dtype dt, int32_t* coords, void* vfeat,
                        int32_t* counts, int32_t* pt2vox, int64_t* m_dev, int64_t* m_host) {
    if (!ws_ok(ws) || n < 0 || n >= ((int64_t)1 << 31) || !valid_v(voxel_size)) return SPV_ERR_INVALID_ARG;
    if (n > 0 && (!xyz || !coords || !counts || !pt2vox)) return SPV_ERR_INVALID_ARG;
    if (feat && (C <= 0 || !vfeat || !valid_dt(dt))) return SPV_ERR_INVALID_ARG;
    VoxLayout L;
    if (need(layout_voxelize(nullptr, 0, n, L), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_voxelize(ws, ws_bytes, n, L);
    if (feat && (!aligned16(feat) || !aligned16(vfeat))) return SPV_ERR_INVALID_ARG;
    hipStream_t s = (hipStream_t)stream;
    launch_voxelize(s, L.w, xyz, batch, n, voxel_size, feat, C, dt, coords, vfeat, counts, pt2vox, m_dev);
    spv_status st = hip_check();
    if (st || !m_host) return st;
    Header h;
    st = sync_status(s, L.h, &h);
    *m_host = st ? 0 : (h.m > n ? n : h.m);
    return st;
}

spv_status spv_voxelize_onto(void* stream, void* ws, size_t ws_bytes, const int32_t* coords, const int64_t* m_dev,
                             int64_t m_cap, const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                             const void* feat, int32_t C, spv_dtype dt, void* vfeat, int32_t* counts,
                             int32_t* pt2vox) {
    if (!ws_ok(ws) || n < 0 || n >= ((int64_t)1 << 31) || m_cap < 0 || m_cap >= ((int64_t)1 << 31) || !valid_v(voxel_size))
        return SPV_ERR_INVALID_ARG;
    if (n > 0 && (!xyz || !pt2vox)) return SPV_ERR_INVALID_ARG;
    if (m_cap > 0 && (!coords || !counts)) return SPV_ERR_INVALID_ARG;
    if (feat && (C <= 0 || !valid_dt(dt))) return SPV_ERR_INVALID_ARG;
    if (feat && m_cap > 0 && !vfeat) return SPV_ERR_INVALID_ARG;
    VoxLayout L;
    const int64_t cap = n > m_cap ? n : m_cap;
    if (need(layout_voxelize(nullptr, 0, cap, L), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_voxelize(ws, ws_bytes, cap, L);
    if (feat && (!aligned16(feat) || (m_cap > 0 && !aligned16(vfeat)))) return SPV_ERR_INVALID_ARG;
    launch_voxelize_onto((hipStream_t)stream, L.w, coords, m_dev, m_cap, xyz, batch, n, voxel_size, feat, C, dt, vfeat,
                         counts, pt2vox);
    return hip_check();
}

spv_status spv_lookup(void* stream, void* ws, size_t ws_bytes, const int32_t* table_coords, const int64_t* m_dev,
                      int64_t m_cap, const int32_t* qcoords, int64_t q, int32_t* idx) {
    if (!ws_ok(ws) || m_cap < 0 || q < 0 || (m_cap > 0 && !table_coords) || (q > 0 && (!qcoords || !idx)))
        return SPV_ERR_INVALID_ARG;
    Arena probe(nullptr, 0);
    probe.take<Header>(1);
    uint32_t S = table_capacity(m_cap > 0 ? m_cap : 1);
    take_table(probe, S);
    if (need(probe.used, ws_bytes)) return SPV_ERR_CAPACITY;
    Arena a(ws, ws_bytes);
    Header* h = a.take<Header>(1);
    Table t = take_table(a, S);
    hipStream_t s = (hipStream_t)stream;
    launch_clear(s, h, t, true);
    if (m_cap > 0) launch_table_build(s, h, t, table_coords, m_dev, m_cap);
    launch_table_lookup(s, t, qcoords, q, idx);
    return hip_check();
}

spv_status spv_voxel_lookup(void* stream, const void* ws, size_t ws_bytes, int64_t n, const int32_t* qcoords,
                            int64_t q, int32_t* idx) {
    if (!ws_ok(ws) || n < 0 || n >= ((int64_t)1 << 31) || q < 0 || (q > 0 && (!qcoords || !idx)))
        return SPV_ERR_INVALID_ARG;
    VoxLayout L;
    if (need(layout_voxelize(nullptr, 0, n, L), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_voxelize(const_cast<void*>(ws), ws_bytes, n, L);
    launch_table_lookup((hipStream_t)stream, L.w.table, qcoords, q, idx);
    return hip_check();
}

spv_status spv_kernel_map(void* stream, void* ws, size_t ws_bytes, const int32_t* in_coords, const int64_t* m_in_dev,
                          int64_t m_cap, int32_t K, int32_t stride, int32_t* out_coords, int64_t* m_out_dev,
                          int32_t* off, int32_t* pairs, int64_t pair_cap, int64_t* total_host) {
    if (!ws_ok(ws) || m_cap < 0 || m_cap >= ((int64_t)1 << 31) || !off || pair_cap < 0) return SPV_ERR_INVALID_ARG;
    if (m_cap > 0 && !in_coords) return SPV_ERR_INVALID_ARG;
    if (!((K == 3 && (stride == 1 || stride == 2)) || (K == 2 && stride == 2))) return SPV_ERR_UNSUPPORTED;
    if (stride == 2 && !out_coords) return SPV_ERR_INVALID_ARG;
    if (pair_cap > 0 && !pairs) return SPV_ERR_INVALID_ARG;
    MapLayout L;
    if (need(layout_kmap(nullptr, 0, m_cap, K, stride, L), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_kmap(ws, ws_bytes, m_cap, K, stride, L);
    hipStream_t s = (hipStream_t)stream;
    // the map's first launch clears the status header
    launch_kernel_map(s, L.w, true, in_coords, m_in_dev, m_cap, K, stride, out_coords, m_out_dev, off, pairs,
                      pair_cap, true);
    spv_status st = hip_check();
    if (st || !total_host) return st;
    const int K3 = K * K * K;
    int32_t tot = 0;
    if (hipMemcpyAsync(&tot, off + K3, sizeof(int32_t), hipMemcpyDeviceToHost, s) != hipSuccess) return hip_check();
    st = sync_status(s, L.h, nullptr);
    *total_host = tot;
    if (st == SPV_OK && tot > pair_cap) st = SPV_ERR_CAPACITY;
    return st;
}

// W[k][c][col] (c < Cin, col < Cout) at W[k * ldk + c * ldc + col * ldcol]
struct WStrides {
    int ldc, ldcol;
    int64_t ldk;
};

static spv_status sparse_conv_call(void* stream, void* ws, size_t ws_bytes, const void* in, int64_t in_rows,
                                   int32_t Cin, const int32_t* off, const int32_t* pairs, int64_t pair_cap, int32_t K3,
                                   int32_t transposed, const void* W, WStrides wst, const float* scale,
                                   const float* shift, const void* res, int32_t relu, void* out,
                                   const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout, spv_dtype dt) {
    if (!ws_ok(ws) || in_rows < 0 || m_out_cap < 0 || m_out_cap >= ((int64_t)1 << 31) || Cin <= 0 || Cout <= 0 || !off ||
        !W || pair_cap < 0 || !valid_dt(dt))
        return SPV_ERR_INVALID_ARG;
    if (!(K3 == 27 || K3 == 8)) return SPV_ERR_UNSUPPORTED;
    if ((in_rows > 0 && !in) || (m_out_cap > 0 && !out) || (pair_cap > 0 && !pairs)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(in) || !aligned16(out) || !aligned16(W) || !aligned16(res) || (res && res == out))
        return SPV_ERR_INVALID_ARG;
    // A transposed stride-2 map gives an output few of the 27 offsets (at most
    // 8, 2-3 on a sweep), which the neighbour-table kernel would still step
    // through for every block: the tile kernel, which only visits pairs, takes
    // it.  A transposed map with as many inputs as outputs (a submanifold map
    // read backwards, as in the input gradient) is as dense as the forward one.
    const bool sparse_tr = transposed && in_rows != m_out_cap;
    ConvLayout L;
    if (need(layout_conv(nullptr, 0, m_out_cap, K3, Cin, Cout, dt, L, in_rows, sparse_tr), ws_bytes))
        return SPV_ERR_CAPACITY;
    layout_conv(ws, ws_bytes, m_out_cap, K3, Cin, Cout, dt, L, in_rows, sparse_tr);
    hipStream_t s = (hipStream_t)stream;
    if (m_out_cap == 0) return clear_status_only(s, ws);
    L.p.m_out_dev = m_out_dev;
    L.p.res = res;
    L.p.w_ldc = wst.ldc;
    L.p.w_ldcol = wst.ldcol;
    L.p.w_ldk = wst.ldk;
    // the plan clears the status header first and packs W in one of its launches
    launch_conv_plan(s, L.p, off, pairs, K3, transposed, pair_cap, in_rows,
                     conv_pack_job(K3, W, L.wpack, Cin, Cout, dt, wst.ldc, wst.ldk, wst.ldcol), true);
    launch_conv_run(s, L.p, in, Cin, in_rows, pairs, pair_cap, transposed, W, L.wpack, scale, shift, relu, out, Cout,
                    dt);
    return hip_check();
}

spv_status spv_sparse_conv(void* stream, void* ws, size_t ws_bytes, const void* in, int64_t in_rows, int32_t Cin,
                           const int32_t* off, const int32_t* pairs, int64_t pair_cap, int32_t K3, int32_t transposed,
                           const void* W, const float* scale, const float* shift, int32_t relu, void* out,
                           const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout, spv_dtype dt) {
    return sparse_conv_call(stream, ws, ws_bytes, in, in_rows, Cin, off, pairs, pair_cap, K3, transposed, W,
                            WStrides{Cout, 1, (int64_t)Cin * Cout}, scale, shift, nullptr, relu, out, m_out_dev,
                            m_out_cap, Cout, dt);
}

spv_status spv_sparse_conv_sliced(void* stream, void* ws, size_t ws_bytes, const void* in, int64_t in_rows,
                                  int32_t Cin, const int32_t* off, const int32_t* pairs, int64_t pair_cap, int32_t K3,
                                  int32_t transposed, const void* W, int32_t Cin_full, int32_t Cout_full,
                                  const float* scale, const float* shift, const void* res, int32_t relu, void* out,
                                  const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout, spv_dtype dt) {
    if (Cin > Cin_full || Cout > Cout_full) return SPV_ERR_INVALID_ARG;
    return sparse_conv_call(stream, ws, ws_bytes, in, in_rows, Cin, off, pairs, pair_cap, K3, transposed, W,
                            WStrides{Cout_full, 1, (int64_t)Cin_full * Cout_full}, scale, shift, res, relu, out,
                            m_out_dev, m_out_cap, Cout, dt);
}

spv_status spv_kernel_map_nbr(void* stream, void* ws, size_t ws_bytes, const int32_t* in_coords,
                              const int64_t* m_in_dev, int64_t m_cap, int32_t* nbr) {
    if (!ws_ok(ws) || m_cap < 0 || m_cap >= ((int64_t)1 << 31) || (m_cap > 0 && (!in_coords || !nbr)))
        return SPV_ERR_INVALID_ARG;
    if (m_cap * 27 * 4 > (int64_t)0xFFFFE000) return SPV_ERR_UNSUPPORTED;
    MapLayout L;
    if (need(layout_kmap(nullptr, 0, m_cap, 3, 1, L), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_kmap(ws, ws_bytes, m_cap, 3, 1, L);
    hipStream_t s = (hipStream_t)stream;
    if (m_cap == 0) return clear_status_only(s, ws);
    launch_clear(s, L.h, L.w.fine, true);
    launch_table_build(s, L.h, L.w.fine, in_coords, m_in_dev, m_cap, nullptr, nullptr, nbr);
    launch_kernel_map_nbr(s, L.w, in_coords, m_in_dev, m_cap, nbr);
    return hip_check();
}

// W: the weights to pack into the workspace, or (packed != NULL) unused
static spv_status conv_nbr_call(void* stream, void* ws, size_t ws_bytes, const void* in, int64_t in_rows, int32_t Cin,
                                const int32_t* nbr, const void* W, int32_t Cin_full, int32_t Cout_full,
                                const void* packed, const float* scale, const float* shift, const void* res,
                                int32_t relu, void* out, const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout,
                                spv_dtype dt) {
    if (!ws_ok(ws) || in_rows < 0 || m_out_cap < 0 || m_out_cap >= ((int64_t)1 << 31) || Cin <= 0 || Cout <= 0 || !W ||
        !valid_dt(dt) || Cin > Cin_full || Cout > Cout_full)
        return SPV_ERR_INVALID_ARG;
    if (!union_supported(27, Cin, Cout, dt) || m_out_cap * 27 * 4 > (int64_t)0xFFFFE000 ||
        in_rows * (int64_t)Cin * 2 > (int64_t)0xFFFFE000)
        return SPV_ERR_UNSUPPORTED;
    if ((in_rows > 0 && !in) || (m_out_cap > 0 && (!out || !nbr))) return SPV_ERR_INVALID_ARG;
    if (!aligned16(in) || !aligned16(out) || !aligned16(W) || !aligned16(res) || (res && res == out))
        return SPV_ERR_INVALID_ARG;
    ConvLayout L;
    if (need(layout_conv(nullptr, 0, m_out_cap, 27, Cin, Cout, dt, L, in_rows), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_conv(ws, ws_bytes, m_out_cap, 27, Cin, Cout, dt, L, in_rows);
    if (m_out_cap == 0) return SPV_OK;
    hipStream_t s = (hipStream_t)stream;
    ConvPlan p = L.p;
    p.nbr = const_cast<int32_t*>(nbr);  // read only
    p.m_out_dev = m_out_dev;
    p.res = res;
    void* wpack = packed ? const_cast<void*>(packed) : L.wpack;
    if (!packed)
        launch_pack_job(s, conv_pack_job(27, W, L.wpack, Cin, Cout, dt, Cout_full, (int64_t)Cin_full * Cout_full));
    launch_conv_union(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out, dt);
    return hip_check();
}

spv_status spv_sparse_conv_nbr(void* stream, void* ws, size_t ws_bytes, const void* in, int64_t in_rows, int32_t Cin,
                               const int32_t* nbr, const void* W, int32_t Cin_full, int32_t Cout_full,
                               const float* scale, const float* shift, const void* res, int32_t relu, void* out,
                               const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout, spv_dtype dt) {
    return conv_nbr_call(stream, ws, ws_bytes, in, in_rows, Cin, nbr, W, Cin_full, Cout_full, nullptr, scale, shift,
                         res, relu, out, m_out_dev, m_out_cap, Cout, dt);
}

spv_status spv_sparse_conv_nbr_packed(void* stream, void* ws, size_t ws_bytes, const void* in, int64_t in_rows,
                                      int32_t Cin, const int32_t* nbr, const void* Wpacked, const float* scale,
                                      const float* shift, const void* res, int32_t relu, void* out,
                                      const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout, spv_dtype dt) {
    if (!Wpacked) return SPV_ERR_INVALID_ARG;
    return conv_nbr_call(stream, ws, ws_bytes, in, in_rows, Cin, nbr, Wpacked, Cin, Cout, Wpacked, scale, shift, res,
                         relu, out, m_out_dev, m_out_cap, Cout, dt);
}

// The device address of `scratch` on the current device, looked up once per
// device (host code never passes the symbol itself to a kernel).
static spv_status noalloc_scratch(void** out) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        g_last_hip_error = (int)hipGetLastError();
        return SPV_ERR_HIP;
    }
    if (dev < 0 || dev >= kMaxDevices) return SPV_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            g_last_hip_error = (int)hipGetLastError();
            return SPV_ERR_HIP;
        }
        addr[dev] = p;
    }
    *out = addr[dev];
    return SPV_OK;
}

spv_status spv_sparse_conv_nbr_noalloc(void* stream, const void* in, int64_t in_rows, int32_t Cin, const int32_t* nbr,
                                       const void* W, int32_t Cin_full, int32_t Cout_full, const float* scale,
                                       const float* shift, const void* res, int32_t relu, void* out,
                                       const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout, spv_dtype dt) {
    if (in_rows < 0 || m_out_cap < 0 || m_out_cap >= ((int64_t)1 << 31) || Cin <= 0 || Cout <= 0 || !W ||
        !valid_dt(dt) || Cin > Cin_full || Cout > Cout_full)
        return SPV_ERR_INVALID_ARG;
    if (!union_supported(27, Cin, Cout, dt) || m_out_cap * 27 * 4 > (int64_t)0xFFFFE000 ||
        in_rows * (int64_t)Cin * 2 > (int64_t)0xFFFFE000)
        return SPV_ERR_UNSUPPORTED;
    if ((in_rows > 0 && !in) || (m_out_cap > 0 && (!out || !nbr))) return SPV_ERR_INVALID_ARG;
    if (!aligned16(in) || !aligned16(out) || !aligned16(W) || !aligned16(res) || (res && res == out))
        return SPV_ERR_INVALID_ARG;
    // the packed weights are the only scratch; more than the array holds is refused
    Arena probe(nullptr, 0);
    plan_wpack_ws(probe, 27, Cin, Cout);
    if (probe.used > kNoAllocScratchBytes) return SPV_ERR_CAPACITY;
    if (m_out_cap == 0) return SPV_OK;
    void* wpack = nullptr;
    spv_status st = noalloc_scratch(&wpack);
    if (st) return st;
    hipStream_t s = (hipStream_t)stream;
    ConvPlan p;
    p.m_cap = m_out_cap;
    p.K3 = 27;
    p.use_union = 1;
    p.nbr = const_cast<int32_t*>(nbr);  // read only
    p.m_out_dev = m_out_dev;
    p.h = nullptr;
    p.res = res;
    launch_pack_job(s, conv_pack_job(27, W, wpack, Cin, Cout, dt, Cout_full, (int64_t)Cin_full * Cout_full));
    launch_conv_union(s, p, in, Cin, in_rows, Cout, wpack, scale, shift, relu, out, dt);
    return hip_check();
}

spv_status spv_map_children(void* stream, void* ws, size_t ws_bytes, const int32_t* off, const int32_t* pairs,
                            int64_t pair_cap, int64_t fine_rows, const int64_t* m_coarse_dev, int64_t m_coarse_cap,
                            int32_t* children) {
    if (!ws_ok(ws) || !off || pair_cap < 0 || fine_rows < 0 || m_coarse_cap < 0 || m_coarse_cap >= ((int64_t)1 << 31))
        return SPV_ERR_INVALID_ARG;
    if ((pair_cap > 0 && !pairs) || (m_coarse_cap > 0 && !children) || !aligned16(children)) return SPV_ERR_INVALID_ARG;
    if (need(sizeof(Header), ws_bytes)) return SPV_ERR_CAPACITY;
    if (m_coarse_cap == 0) return clear_status_only((hipStream_t)stream, ws);
    launch_nbr_table((hipStream_t)stream, off, pairs, kUpChildren, pair_cap, m_coarse_dev, m_coarse_cap, fine_rows,
                     children, (Header*)ws);
    return hip_check();
}

static spv_status conv_up_call(void* stream, void* ws, size_t ws_bytes, const void* in, const int64_t* m_in_dev,
                               int64_t m_in_cap, int32_t Cin, const int32_t* children, const void* W, int32_t Cin_full,
                               int32_t Cout_full, const void* packed, const float* scale, const float* shift,
                               const void* res, int32_t relu, void* out, int64_t out_rows, int32_t Cout,
                               spv_dtype dt) {
    if (!ws_ok(ws) || m_in_cap < 0 || m_in_cap >= ((int64_t)1 << 31) || out_rows < 0 || Cin <= 0 || Cout <= 0 || !W ||
        !valid_dt(dt) || Cin > Cin_full || Cout > Cout_full)
        return SPV_ERR_INVALID_ARG;
    if (!up_supported(Cin, Cout, dt)) return SPV_ERR_UNSUPPORTED;
    if ((m_in_cap > 0 && (!in || !children)) || (out_rows > 0 && !out)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(in) || !aligned16(out) || !aligned16(W) || !aligned16(res) || (res && res == out) || in == out)
        return SPV_ERR_INVALID_ARG;
    Arena probe(nullptr, 0);
    probe.take<Header>(1);
    plan_wpack_ws(probe, kUpChildren, Cin, Cout);
    if (need(probe.used, ws_bytes)) return SPV_ERR_CAPACITY;
    Arena a(ws, ws_bytes);
    a.take<Header>(1);
    void* wpack = plan_wpack_ws(a, kUpChildren, Cin, Cout);
    if (m_in_cap == 0) return SPV_OK;
    hipStream_t s = (hipStream_t)stream;
    if (packed)
        wpack = const_cast<void*>(packed);
    else
        launch_pack_job(s, conv_pack_job(kUpChildren, W, wpack, Cin, Cout, dt, Cout_full,
                                         (int64_t)Cin_full * Cout_full));
    UpArgs u{children, m_in_dev, m_in_cap, in, Cin, Cout, (int)dt, scale, shift, relu, res, out, out_rows};
    launch_conv_up(s, u, wpack);
    return hip_check();
}

spv_status spv_sparse_conv_up(void* stream, void* ws, size_t ws_bytes, const void* in, const int64_t* m_in_dev,
                              int64_t m_in_cap, int32_t Cin, const int32_t* children, const void* W, int32_t Cin_full,
                              int32_t Cout_full, const float* scale, const float* shift, const void* res, int32_t relu,
                              void* out, int64_t out_rows, int32_t Cout, spv_dtype dt) {
    return conv_up_call(stream, ws, ws_bytes, in, m_in_dev, m_in_cap, Cin, children, W, Cin_full, Cout_full, nullptr,
                        scale, shift, res, relu, out, out_rows, Cout, dt);
}

spv_status spv_sparse_conv_up_packed(void* stream, void* ws, size_t ws_bytes, const void* in, const int64_t* m_in_dev,
                                     int64_t m_in_cap, int32_t Cin, const int32_t* children, const void* Wpacked,
                                     const float* scale, const float* shift, const void* res, int32_t relu, void* out,
                                     int64_t out_rows, int32_t Cout, spv_dtype dt) {
    if (!Wpacked) return SPV_ERR_INVALID_ARG;
    return conv_up_call(stream, ws, ws_bytes, in, m_in_dev, m_in_cap, Cin, children, Wpacked, Cin, Cout, Wpacked,
                        scale, shift, res, relu, out, out_rows, Cout, dt);
}

spv_status spv_sparse_conv_dgrad(void* stream, void* ws, size_t ws_bytes, const void* dy, int64_t dy_rows,
                                 int32_t Cout, const int32_t* off, const int32_t* pairs, int64_t pair_cap, int32_t K3,
                                 int32_t transposed, const void* W, void* dx, const int64_t* m_in_dev, int64_t m_in_cap,
                                 int32_t Cin, spv_dtype dt) {
    // dx[i] = sum over the pairs (i, j, k) of dy[j] @ W[k]^T: the conv over the
    // same map with each pair's roles swapped, reading W[k] transposed in place
    return sparse_conv_call(stream, ws, ws_bytes, dy, dy_rows, Cout, off, pairs, pair_cap, K3, transposed ? 0 : 1, W,
                            WStrides{1, Cout, (int64_t)Cin * Cout}, nullptr, nullptr, nullptr, 0, dx, m_in_dev,
                            m_in_cap, Cin, dt);
}

spv_status spv_sparse_conv_dgrad_nbr(void* stream, void* ws, size_t ws_bytes, const void* dy, int32_t Cout,
                                     const int32_t* nbr, const void* W, void* dx, const int64_t* m_dev, int64_t m_cap,
                                     int32_t Cin, spv_dtype dt) {
    if (!ws_ok(ws) || m_cap < 0 || m_cap >= ((int64_t)1 << 31) || Cin <= 0 || Cout <= 0 || !W || !valid_dt(dt))
        return SPV_ERR_INVALID_ARG;
    // the conv with Cout inputs and Cin outputs on the same table
    if (!union_supported(27, Cout, Cin, dt) || m_cap * 27 * 4 > (int64_t)0xFFFFE000 ||
        m_cap * (int64_t)Cout * 2 > (int64_t)0xFFFFE000)
        return SPV_ERR_UNSUPPORTED;
    if (m_cap > 0 && (!dy || !dx || !nbr)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(dy) || !aligned16(dx) || !aligned16(W) || dx == dy) return SPV_ERR_INVALID_ARG;
    ConvLayout L;
    if (need(layout_conv(nullptr, 0, m_cap, 27, Cout, Cin, dt, L, m_cap), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_conv(ws, ws_bytes, m_cap, 27, Cout, Cin, dt, L, m_cap);
    if (m_cap == 0) return SPV_OK;
    hipStream_t s = (hipStream_t)stream;
    ConvPlan p = L.p;
    p.nbr = const_cast<int32_t*>(nbr);  // read only
    p.m_out_dev = m_dev;
    p.res = nullptr;
    launch_pack_job(s, conv_pack_job_mirrored(W, L.wpack, Cin, Cout, dt));
    launch_conv_union(s, p, dy, Cout, m_cap, Cin, L.wpack, nullptr, nullptr, 0, dx, dt);
    return hip_check();
}

spv_status spv_sparse_conv_wgrad(void* stream, void* ws, size_t ws_bytes, const void* x, int64_t x_rows, int32_t Cin,
                                 const void* dy, int64_t dy_rows, int32_t Cout, const int32_t* off, const int32_t* pairs,
                                 int64_t pair_cap, int32_t K3, int32_t transposed, float* dW, spv_dtype dt) {
    if (!ws_ok(ws) || x_rows < 0 || dy_rows < 0 || Cin <= 0 || Cout <= 0 || !off || !dW || pair_cap < 0 || !valid_dt(dt))
        return SPV_ERR_INVALID_ARG;
    if (!(K3 == 27 || K3 == 8) || !wgrad_supported(Cin, Cout)) return SPV_ERR_UNSUPPORTED;
    if ((x_rows > 0 && !x) || (dy_rows > 0 && !dy) || (pair_cap > 0 && !pairs)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(dy)) return SPV_ERR_INVALID_ARG;
    Arena probe(nullptr, 0);
    probe.take<Header>(1);
    plan_wgrad_ws(probe, K3, Cin, Cout);
    if (need(probe.used, ws_bytes)) return SPV_ERR_CAPACITY;
    Arena a(ws, ws_bytes);
    a.take<Header>(1);
    float* partial = (float*)plan_wgrad_ws(a, K3, Cin, Cout);
    WgradArgs w{x, x_rows, Cin, dy, dy_rows, Cout, off, pairs, pair_cap, K3, transposed ? 1 : 0, (int)dt};
    launch_wgrad((hipStream_t)stream, w, partial, dW);
    return hip_check();
}

spv_status spv_voxelize_backward(void* stream, const void* dvfeat, int64_t m, int32_t C, const int32_t* counts,
                                 const int32_t* pt2vox, int64_t n, void* dfeat, spv_dtype dt) {
    if (m < 0 || n < 0 || C <= 0 || !valid_dt(dt)) return SPV_ERR_INVALID_ARG;
    if (n > 0 && (!dvfeat || !counts || !pt2vox || !dfeat)) return SPV_ERR_INVALID_ARG;
    launch_voxelize_backward((hipStream_t)stream, dvfeat, C, counts, pt2vox, n, m, dfeat, (int)dt);
    return hip_check();
}

size_t spv_epilogue_backward_workspace_bytes(int64_t m, int32_t C) {
    if (m < 0 || C <= 0) return 0;
    Arena a(nullptr, 0);
    a.take<double>(epilogue_backward_part_entries(m, C));
    return a.used;
}

spv_status spv_epilogue_backward(void* stream, void* ws, size_t ws_bytes, const void* dy, const void* a,
                                 const float* scale, const float* shift, int32_t relu, const void* res,
                                 int32_t res_after_act, int64_t m, int32_t C, void* da, void* dres, float* dscale,
                                 float* dshift, spv_dtype dt) {
    if (m < 0 || C <= 0 || !valid_dt(dt)) return SPV_ERR_INVALID_ARG;
    if (m > 0 && (!dy || !a)) return SPV_ERR_INVALID_ARG;
    const bool sums = dscale || dshift;
    if (sums) {
        if (!ws_ok(ws)) return SPV_ERR_INVALID_ARG;
        if (need(spv_epilogue_backward_workspace_bytes(m, C), ws_bytes)) return SPV_ERR_CAPACITY;
    }
    if (m == 0 && !sums) return SPV_OK;
    EpiBwdArgs e{dy, a, scale, shift, relu ? 1 : 0, res, res_after_act ? 1 : 0, m, C, (int)dt, da, dres, dscale, dshift};
    launch_epilogue_backward((hipStream_t)stream, e, sums ? (double*)ws : nullptr);
    return hip_check();
}

// the packed transposed W (the input gradient runs on the linear kernel), then
// the weight gradient's partial sums (sized as a 27-offset map's: the
// workgroups of the identity map's one offset take as many slots)
static size_t layout_linear_backward(void* ws, size_t bytes, int Cin, int Cout, void** wpack, float** partial) {
    Arena a(ws, bytes);
    a.take<Header>(1);
    *wpack = plan_linear_ws(a, Cout, Cin);
    *partial = (float*)plan_wgrad_ws(a, 27, Cin, Cout);
    return a.used;
}

size_t spv_linear_backward_workspace_bytes(int32_t Cin, int32_t Cout) {
    if (Cin <= 0 || Cout <= 0) return 0;
    void* wp;
    float* part;
    return layout_linear_backward(nullptr, 0, Cin, Cout, &wp, &part);
}

spv_status spv_linear_backward(void* stream, void* ws, size_t ws_bytes, const void* in, int64_t m, int32_t Cin,
                               const void* W, int32_t Cout, const void* da, void* din, float* dW, spv_dtype dt) {
    if (!ws_ok(ws) || m < 0 || m >= ((int64_t)1 << 31) || Cin <= 0 || Cout <= 0 || !W || !valid_dt(dt))
        return SPV_ERR_INVALID_ARG;
    if (m > 0 && (!in || !da || (!din && !dW))) return SPV_ERR_INVALID_ARG;
    if (!aligned16(in) || !aligned16(da) || !aligned16(din) || (din && (din == da || din == in)))
        return SPV_ERR_INVALID_ARG;
    if (dW && !wgrad_supported(Cin, Cout)) return SPV_ERR_UNSUPPORTED;
    void* wpack;
    float* partial;
    if (need(layout_linear_backward(nullptr, 0, Cin, Cout, &wpack, &partial), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_linear_backward(ws, ws_bytes, Cin, Cout, &wpack, &partial);
    const hipStream_t s = (hipStream_t)stream;
    if (din && m > 0) {
        // din = da @ W^T: the linear layer with Cout inputs, Cin outputs, W read transposed
        LinearArgs l{da, nullptr, m, Cout, Cin, (int)dt, W, Cout, nullptr, nullptr, 0, nullptr, 0, din};
        l.wt = 1;
        launch_linear(s, l, wpack, false);
    }
    if (dW) {
        // dW = in^T da: the weight gradient over the identity map (pair p = (p, p))
        WgradArgs w{in, m, Cin, da, m, Cout, nullptr, nullptr, m, 1, 0, (int)dt};
        w.slot_k3 = 27;
        launch_wgrad(s, w, partial, dW);
    }
    return hip_check();
}

size_t spv_devoxelize_backward_workspace_bytes(int64_t n, int64_t m) {
    if (n < 0 || m < 0) return 0;
    Arena a(nullptr, 0);
    plan_devox_backward_ws(a, n, m);
    return a.used;
}

spv_status spv_devoxelize_backward(void* stream, void* ws, size_t ws_bytes, const int32_t* corner_idx,
                                   const float* corner_w, const void* dout, int64_t n, int32_t C, float* dvfeat,
                                   int64_t m, spv_dtype dt) {
    if (!ws_ok(ws) || m < 0 || n < 0 || C <= 0 || !valid_dt(dt) || (m > 0 && !dvfeat)) return SPV_ERR_INVALID_ARG;
    if (n > 0 && (!corner_idx || !corner_w || !dout)) return SPV_ERR_INVALID_ARG;
    if (dvfeat && (const void*)dvfeat == dout) return SPV_ERR_INVALID_ARG;  // the gather reads dout while writing
    // entry numbers 8n and voxel positions fit int32
    if (n >= ((int64_t)1 << 28) || m >= ((int64_t)1 << 31) - 1) return SPV_ERR_INVALID_ARG;
    if (need(spv_devoxelize_backward_workspace_bytes(n, m), ws_bytes)) return SPV_ERR_CAPACITY;
    Arena a(ws, ws_bytes);
    const DvbWs w = plan_devox_backward_ws(a, n, m);
    launch_devoxelize_backward((hipStream_t)stream, w, corner_idx, corner_w, dout, n, C, dvfeat, m, (int)dt);
    return hip_check();
}

static spv_status linear_call(void* stream, void* ws, size_t ws_bytes, const void* in, const int64_t* m_dev,
                              int64_t m_cap, int32_t Cin, const void* W, int32_t Cin_full, int32_t Cout_full,
                              const void* packed, const float* scale, const float* shift, int32_t relu,
                              const void* res, int32_t res_after_act, void* out, int32_t Cout, spv_dtype dt) {
    if (!ws_ok(ws) || m_cap < 0 || m_cap >= ((int64_t)1 << 31) || Cin <= 0 || Cout <= 0 || !W || !valid_dt(dt) ||
        Cin > Cin_full || Cout > Cout_full)
        return SPV_ERR_INVALID_ARG;
    if (m_cap > 0 && (!in || !out)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(in) || !aligned16(out) || !aligned16(res) || (res && res == out) || in == out)
        return SPV_ERR_INVALID_ARG;
    void* wpack = nullptr;
    if (need(layout_linear(nullptr, 0, Cin, Cout, &wpack), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_linear(ws, ws_bytes, Cin, Cout, &wpack);
    if (m_cap == 0) return SPV_OK;
    LinearArgs a{in, m_dev, m_cap, Cin, Cout, (int)dt, W, Cout_full, scale, shift, relu, res, res_after_act ? 1 : 0,
                 out};
    launch_linear((hipStream_t)stream, a, packed ? const_cast<void*>(packed) : wpack, packed != nullptr);
    return hip_check();
}

spv_status spv_linear(void* stream, void* ws, size_t ws_bytes, const void* in, const int64_t* m_dev, int64_t m_cap,
                      int32_t Cin, const void* W, int32_t Cin_full, int32_t Cout_full, const float* scale,
                      const float* shift, int32_t relu, const void* res, int32_t res_after_act, void* out,
                      int32_t Cout, spv_dtype dt) {
    return linear_call(stream, ws, ws_bytes, in, m_dev, m_cap, Cin, W, Cin_full, Cout_full, nullptr, scale, shift,
                       relu, res, res_after_act, out, Cout, dt);
}

spv_status spv_linear_packed(void* stream, void* ws, size_t ws_bytes, const void* in, const int64_t* m_dev,
                             int64_t m_cap, int32_t Cin, const void* Wpacked, const float* scale, const float* shift,
                             int32_t relu, const void* res, int32_t res_after_act, void* out, int32_t Cout,
                             spv_dtype dt) {
    if (!Wpacked) return SPV_ERR_INVALID_ARG;
    // the vector-ALU path reads W itself: packed weights serve the matrix-core kernel only
    if (!linear_mfma_supported(Cin, Cout, dt)) return SPV_ERR_UNSUPPORTED;
    return linear_call(stream, ws, ws_bytes, in, m_dev, m_cap, Cin, Wpacked, Cin, Cout, Wpacked, scale, shift, relu,
                       res, res_after_act, out, Cout, dt);
}

// the fragment layout the neighbour-table, upsampling and linear kernels read
static bool packed_shape(int32_t K3, int32_t Cin, int32_t Cout, int* kch, int* nb) {
    const int k = (Cin + 31) / 32, n = (Cout + 15) / 16;
    if (K3 <= 0 || K3 > 27 || Cin <= 0 || Cout <= 0) return false;
    if (!(k == 1 || k == 2 || k == 3 || k == 4 || k == 6 || k == 8) || n > 16) return false;
    *kch = k;
    *nb = n;
    return true;
}

size_t spv_packed_weights_bytes(int32_t K3, int32_t Cin, int32_t Cout) {
    int kch, nb;
    if (!packed_shape(K3, Cin, Cout, &kch, &nb)) return 0;
    return (size_t)K3 * kch * nb * 64 * sizeof(uint4);
}

spv_status spv_pack_weights(void* stream, const void* W, int32_t K3, int32_t Cin_full, int32_t Cout_full, int32_t Cin,
                            int32_t Cout, spv_dtype dt, void* packed, size_t packed_bytes) {
    if (!W || !packed || Cin > Cin_full || Cout > Cout_full || !valid_dt(dt)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(packed)) return SPV_ERR_INVALID_ARG;
    int kch, nb;
    if (dt == SPV_F32 || !packed_shape(K3, Cin, Cout, &kch, &nb)) return SPV_ERR_UNSUPPORTED;
    if (packed_bytes < spv_packed_weights_bytes(K3, Cin, Cout)) return SPV_ERR_CAPACITY;
    PackJob q{(const uint16_t*)W, (uint4*)packed, K3, Cin, Cout, kch, nb, (int64_t)K3 * kch * nb * 64, Cout_full,
              (int64_t)Cin_full * Cout_full, 1};
    launch_pack_job((hipStream_t)stream, q);
    return hip_check();
}

spv_status spv_devoxelize(void* stream, void* ws, size_t ws_bytes, const int32_t* grid_coords, const int64_t* m_dev,
                          int64_t m_cap, int32_t stride_log2, const float* xyz, const int32_t* batch, int64_t n,
                          float voxel_size, spv_devox_mode mode, const void* vfeat, int32_t C, const void* pfeat,
                          int32_t Cp, const void* Wp, const float* scale_p, const float* shift_p, int32_t relu_p,
                          void* out, spv_dtype dt, int32_t* corner_idx, float* corner_w) {
    if (!ws_ok(ws) || n < 0 || n >= ((int64_t)1 << 31) || m_cap < 0 || m_cap >= ((int64_t)1 << 31) || C <= 0 ||
        !valid_dt(dt) || !valid_v(voxel_size) || stride_log2 < 0 || stride_log2 > 15)
        return SPV_ERR_INVALID_ARG;
    if (mode != SPV_DEVOX_CENTER && mode != SPV_DEVOX_CORNER && mode != SPV_DEVOX_NEAREST) return SPV_ERR_INVALID_ARG;
    if ((n > 0 && (!xyz || !out)) || (m_cap > 0 && (!grid_coords || !vfeat))) return SPV_ERR_INVALID_ARG;
    if (pfeat && (Cp <= 0 || !Wp)) return SPV_ERR_INVALID_ARG;
    if ((corner_idx == nullptr) != (corner_w == nullptr)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(vfeat) || !aligned16(out) || !aligned16(pfeat) || !aligned16(Wp)) return SPV_ERR_INVALID_ARG;
    const int cp = pfeat ? Cp : 0;
    DevoxLayout L;
    if (need(layout_devox(nullptr, 0, m_cap, n, C, cp, L), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_devox(ws, ws_bytes, m_cap, n, C, cp, L);
    hipStream_t s = (hipStream_t)stream;
    launch_clear(s, L.h, L.t, true);
    if (m_cap > 0) launch_table_build(s, L.h, L.t, grid_coords, m_dev, m_cap);
    DevoxArgs a;
    a.table = L.t;
    a.stride_log2 = stride_log2;
    a.xyz = xyz;
    a.batch = batch;
    a.n = n;
    a.voxel_size = voxel_size;
    a.mode = mode;
    a.vfeat = vfeat;
    a.C = C;
    a.pfeat = pfeat;
    a.Cp = cp;
    a.Wp = Wp;
    a.scale_p = scale_p;
    a.shift_p = shift_p;
    a.relu_p = relu_p;
    a.out = out;
    a.dt = dt;
    a.corner_idx = corner_idx;
    a.corner_w = corner_w;
    a.h = L.h;
    launch_devox(s, a, L.wpack, L.cidx, L.cw);
    return hip_check();
}

spv_status spv_devoxelize_nbr(void* stream, void* ws, size_t ws_bytes, const int32_t* grid_coords, const int64_t* m_dev,
                              int64_t m_cap, const int32_t* nbr, const int32_t* pt2vox, int32_t stride_log2,
                              const float* xyz, const int32_t* batch, int64_t n, float voxel_size, spv_devox_mode mode,
                              const void* vfeat, int32_t C, const void* pfeat, int32_t Cp, const void* Wp,
                              const float* scale_p, const float* shift_p, int32_t relu_p, void* out, spv_dtype dt) {
    if (!ws_ok(ws) || n < 0 || n >= ((int64_t)1 << 31) || m_cap < 0 || m_cap >= ((int64_t)1 << 31) || C <= 0 ||
        !valid_dt(dt) || !valid_v(voxel_size) || stride_log2 < 0 || stride_log2 > 15)
        return SPV_ERR_INVALID_ARG;
    if (mode != SPV_DEVOX_CENTER && mode != SPV_DEVOX_CORNER && mode != SPV_DEVOX_NEAREST) return SPV_ERR_INVALID_ARG;
    if ((n > 0 && (!xyz || !out || !pt2vox)) || (m_cap > 0 && (!grid_coords || !vfeat || !nbr)))
        return SPV_ERR_INVALID_ARG;
    if (pfeat && (Cp <= 0 || !Wp)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(vfeat) || !aligned16(out) || !aligned16(pfeat) || !aligned16(Wp)) return SPV_ERR_INVALID_ARG;
    const int cp = pfeat ? Cp : 0;
    // only the matrix-core kernel reads corners from the neighbour table
    if (!devox_mfma_supported(C, cp, dt)) return SPV_ERR_UNSUPPORTED;
    Arena probe(nullptr, 0);
    probe.take<Header>(1);
    take_table(probe, 4);
    void* wp_probe = plan_devox_ws(probe, C, cp);
    (void)wp_probe;
    if (need(probe.used, ws_bytes)) return SPV_ERR_CAPACITY;
    Arena ar(ws, ws_bytes);
    Header* h = ar.take<Header>(1);
    // an empty 4-slot table: the kernel's probe for a corner outside the point's
    // 3x3x3 neighbourhood (not reached when pt2vox is the grid's own) finds nothing
    Table t = take_table(ar, 4);
    void* wpack = plan_devox_ws(ar, C, cp);
    hipStream_t s = (hipStream_t)stream;
    launch_clear(s, h, t, true);
    DevoxArgs a;
    a.table = t;
    a.stride_log2 = stride_log2;
    a.xyz = xyz;
    a.batch = batch;
    a.n = n;
    a.voxel_size = voxel_size;
    a.mode = mode;
    a.vfeat = vfeat;
    a.C = C;
    a.pfeat = pfeat;
    a.Cp = cp;
    a.Wp = Wp;
    a.scale_p = scale_p;
    a.shift_p = shift_p;
    a.relu_p = relu_p;
    a.out = out;
    a.dt = dt;
    a.corner_idx = nullptr;
    a.corner_w = nullptr;
    a.h = h;
    a.pt2vox = pt2vox;
    a.grid_coords = grid_coords;
    a.nbr = nbr;
    a.nbr_rows = m_cap;
    a.nbr_m_dev = m_dev;
    launch_devox(s, a, wpack, nullptr, nullptr);
    return hip_check();
}

spv_status spv_block(void* stream, void* ws, size_t ws_bytes, const spv_block_params* p, const float* xyz,
                     const int32_t* batch, int64_t n, const void* feat, void* out, int64_t* m_host) {
    if (!ws_ok(ws) || !p || n < 0 || n >= ((int64_t)1 << 31) || p->C <= 0 || !valid_dt(p->dtype) ||
        !valid_v(p->voxel_size))
        return SPV_ERR_INVALID_ARG;
    if (p->n_convs < 1 || p->n_convs > 2 || !p->Wp) return SPV_ERR_INVALID_ARG;
    if (p->devox_mode != SPV_DEVOX_CENTER && p->devox_mode != SPV_DEVOX_CORNER && p->devox_mode != SPV_DEVOX_NEAREST)
        return SPV_ERR_INVALID_ARG;
    for (int l = 0; l < p->n_convs; ++l)
        if (!p->W[l] || !aligned16(p->W[l])) return SPV_ERR_INVALID_ARG;
    if (n > 0 && (!xyz || !feat || !out)) return SPV_ERR_INVALID_ARG;
    if (!aligned16(feat) || !aligned16(out) || !aligned16(p->Wp)) return SPV_ERR_INVALID_ARG;
    const int C = p->C, dt = p->dtype;
    BlockLayout L;
    if (need(layout_block(nullptr, 0, n, C, dt, L), ws_bytes)) return SPV_ERR_CAPACITY;
    layout_block(ws, ws_bytes, n, C, dt, L);
    hipStream_t s = (hipStream_t)stream;
    const int64_t nn = n > 0 ? n : 1;
    const bool prof = p->events && p->n_events >= 7;
    auto mark = [&](int i) {
        if (prof) hipEventRecord((hipEvent_t)p->events[i], s);
    };
    // devoxelization arguments (its MLP weight is packed by the prologue)
    DevoxArgs a;
    a.table = L.vox.table;
    a.stride_log2 = 0;
    a.xyz = xyz;
    a.batch = batch;
    a.n = n;
    a.voxel_size = p->voxel_size;
    a.mode = p->devox_mode;
    a.vfeat = nullptr;  // set once the convs have run
    a.C = C;
    a.pfeat = feat;
    a.Cp = C;
    a.Wp = p->Wp;
    a.scale_p = p->scale_p;
    a.shift_p = p->shift_p;
    a.relu_p = p->relu_p;
    a.out = out;
    a.dt = dt;
    a.corner_idx = nullptr;
    a.corner_w = nullptr;
    a.h = L.h;
    if (L.plan.use_union) {  // the map's neighbour table gives every point's corners
        a.pt2vox = L.pt2vox;
        a.grid_coords = L.coords;
        a.nbr = L.plan.nbr;
        a.nbr_rows = L.plan.m_cap;
        a.nbr_m_dev = L.m_dev;
    }
    mark(0);
    // voxel branch: Eq. 1-2 into the hashed grid; its first launch also clears
    // the voxel table and packs every weight of the block
    PackJob jobs[kMaxPackJobs];
    int njobs = 0;
    for (int l = 0; l < p->n_convs; ++l) jobs[njobs++] = conv_pack_job(27, p->W[l], L.wpack_conv[l], C, C, dt);
    jobs[njobs++] = devox_pack_job(a, L.wpack_mlp);
    // the neighbour-table map expects entries 14..26 of every row zeroed: the
    // voxelization's inserts do it
    if (L.plan.use_union) L.vox.nbr_upper = L.plan.nbr;
    launch_voxelize(s, L.vox, xyz, batch, n, p->voxel_size, feat, C, dt, L.coords, L.va, L.counts, L.pt2vox, L.m_dev,
                    jobs, njobs);
    mark(1);
    // one kernel map for both convs, probing the voxelization's table; the
    // neighbour-table conv needs only the table, the other kernels the pairs
    L.plan.m_out_dev = L.m_dev;
    if (L.plan.use_union) {
        launch_kernel_map_nbr(s, L.map, L.coords, L.m_dev, nn, L.plan.nbr);
        mark(2);
    } else {
        launch_kernel_map(s, L.map, false, L.coords, L.m_dev, nn, 3, 1, nullptr, nullptr, L.off, L.pairs, L.pair_cap);
        mark(2);
        launch_conv_plan(s, L.plan, L.off, L.pairs, 27, 0, L.pair_cap, nn, PackJob{});
    }
    mark(3);
    void* cur = L.va;
    void* nxt = L.vb;
    for (int l = 0; l < p->n_convs; ++l) {
        ConvPlan plan = L.plan;
        const bool res = p->residual && l == p->n_convs - 1;
        if (res) {
            // the last conv of a residual block adds the block's voxel input
            // (still in va) and writes a buffer that aliases neither
            plan.res = L.va;
            nxt = (cur == L.vb) ? L.vc : L.vb;
        }
        launch_conv_run(s, plan, cur, C, nn, L.pairs, L.pair_cap, 0, p->W[l], L.wpack_conv[l], p->scale[l],
                        p->shift[l], p->relu[l], nxt, C, dt);
        void* t = cur;
        cur = nxt;
        nxt = t;
        mark(4 + l);
    }
    if (p->n_convs == 1) mark(5);
    // devoxelize onto the points + point MLP + fusion by addition
    a.vfeat = cur;
    launch_devox(s, a, L.wpack_mlp, L.cidx, L.cw, true);
    mark(6);
    spv_status st = hip_check();
    if (st || !m_host) return st;
    Header h;
    st = sync_status(s, L.h, &h);
    *m_host = st ? 0 : (h.m > n ? n : h.m);
    return st;
}

}  // extern "C"
