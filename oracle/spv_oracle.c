/*
 * spv_oracle.c -- CPU oracle for the SPVConv hot path.  TEST INFRASTRUCTURE ONLY:
 * it is loaded by the tests, the smoke check and the bench's CPU-baseline leg,
 * never by the product path.  It shares no code with the HIP library.
 *
 * Everything here is the plain definition, evaluated directly:
 *   - the voxel set is the sorted list of distinct quantized keys (Eq. 1);
 *   - voxel features are the literal means of Eq. 2, summed in fp64 in point order;
 *   - kernel-map entries are found by binary search of each neighbour coordinate;
 *   - the convolution is the triple loop over (pair, c_in, c_out) in fp64;
 *   - trilinear devoxelization evaluates the 8 corner weights directly.
 * Parity status: every function here is pinned by the CPU test suite against an
 * independent formulation (dense 3D convolution on the zero-filled grid, literal
 * O(mn) Eq. 2, all-pairs neighbour search, dense trilinear sampling, closed forms).
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no fast-math: quantization and
 * corner weights must use IEEE single-precision division and products).
 */
#include "spv_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* storage dtypes                                                             */
/* ------------------------------------------------------------------------- */

static double dec_bf16(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

static double dec_f16(uint16_t h) {
    int s = (h >> 15) & 1, e = (h >> 10) & 31, mnt = h & 1023;
    double v;
    if (e == 0)
        v = ldexp((double)mnt, -24);
    else if (e == 31)
        v = mnt ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + mnt), e - 25);
    return s ? -v : v;
}

double spvo_decode(const void* buf, int64_t i, int32_t dtype) {
    if (dtype == SPVO_F32) return (double)((const float*)buf)[i];
    if (dtype == SPVO_BF16) return dec_bf16(((const uint16_t*)buf)[i]);
    return dec_f16(((const uint16_t*)buf)[i]);
}

/* Round x to p significant bits with minimum normal exponent emin, ties to even;
 * values beyond max_finite become infinities (IEEE round-to-nearest overflow). */
static double round_sig(double x, int p, int emin, double max_finite) {
    if (x == 0.0 || !isfinite(x)) return x;
    int e = ilogb(x);
    if (e < emin) e = emin;
    double q = ldexp(1.0, e - (p - 1));
    double r = nearbyint(x / q) * q;
    if (fabs(r) > max_finite) r = copysign(INFINITY, x);
    return r;
}

static uint16_t enc_bf16(double x) {
    if (isnan(x)) return (uint16_t)(signbit(x) ? 0xFFC0 : 0x7FC0);
    double r = round_sig(x, 8, -126, ldexp(255.0, 120)); /* (2 - 2^-7) * 2^127 */
    float f = (float)r;                                   /* exact */
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

static uint16_t enc_f16(double x) {
    uint16_t s = signbit(x) ? 0x8000 : 0;
    if (isnan(x)) return (uint16_t)(s | 0x7E00);
    double r = round_sig(x, 11, -14, 65504.0);
    if (isinf(r)) return (uint16_t)(s | 0x7C00);
    double a = fabs(r);
    if (a == 0.0) return s;
    int e = ilogb(a);
    if (e < -14) return (uint16_t)(s | (uint16_t)ldexp(a, 24)); /* subnormal */
    uint16_t mnt = (uint16_t)(ldexp(a, -e) * 1024.0 - 1024.0);
    return (uint16_t)(s | (uint16_t)((e + 15) << 10) | mnt);
}

void spvo_round_store(double x, void* buf, int64_t i, int32_t dtype) {
    if (dtype == SPVO_F32)
        ((float*)buf)[i] = (float)x; /* one round-to-nearest-even */
    else if (dtype == SPVO_BF16)
        ((uint16_t*)buf)[i] = enc_bf16(x);
    else
        ((uint16_t*)buf)[i] = enc_f16(x);
}

static int valid_dtype(int32_t dt) { return dt == SPVO_F32 || dt == SPVO_BF16 || dt == SPVO_F16; }

/* ------------------------------------------------------------------------- */
/* coordinates                                                                */
/* ------------------------------------------------------------------------- */

#define COORD_MIN (-32767)
#define COORD_MAX 32766
#define BATCH_MAX 65534

typedef struct {
    int32_t c[4]; /* b, x, y, z */
    int64_t idx;  /* original position */
} keyrec;

static int cmp_coord(const int32_t* a, const int32_t* b) {
    for (int d = 0; d < 4; ++d) {
        if (a[d] < b[d]) return -1;
        if (a[d] > b[d]) return 1;
    }
    return 0;
}

static int cmp_keyrec(const void* pa, const void* pb) {
    const keyrec* a = (const keyrec*)pa;
    const keyrec* b = (const keyrec*)pb;
    int r = cmp_coord(a->c, b->c);
    if (r) return r;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

/* Sorted lookup structure over a coordinate list (the ordered voxel set). */
typedef struct {
    keyrec* rec;
    int64_t n;
} coordset;

/* Returns SPVO_ERR_INVALID_ARG if the list holds a duplicate coordinate. */
static int coordset_build(coordset* s, const int32_t* coords, int64_t m) {
    s->n = m;
    s->rec = (keyrec*)malloc((size_t)(m > 0 ? m : 1) * sizeof(keyrec));
    if (!s->rec) return SPVO_ERR_CAPACITY;
    for (int64_t i = 0; i < m; ++i) {
        memcpy(s->rec[i].c, coords + 4 * i, 16);
        s->rec[i].idx = i;
    }
    qsort(s->rec, (size_t)m, sizeof(keyrec), cmp_keyrec);
    for (int64_t i = 1; i < m; ++i)
        if (cmp_coord(s->rec[i - 1].c, s->rec[i].c) == 0) return SPVO_ERR_INVALID_ARG;
    return SPVO_OK;
}

static int64_t coordset_find(const coordset* s, const int32_t* c) {
    int64_t lo = 0, hi = s->n;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        int r = cmp_coord(s->rec[mid].c, c);
        if (r == 0) return s->rec[mid].idx;
        if (r < 0)
            lo = mid + 1;
        else
            hi = mid;
    }
    return -1;
}

static void coordset_free(coordset* s) { free(s->rec); }

static int coords_in_range(const int32_t* coords, int64_t m) {
    for (int64_t i = 0; i < m; ++i) {
        const int32_t* c = coords + 4 * i;
        if (c[0] < 0 || c[0] > BATCH_MAX) return 0;
        for (int d = 1; d < 4; ++d)
            if (c[d] < COORD_MIN || c[d] > COORD_MAX) return 0;
    }
    return 1;
}

/* Eq. 1 for one axis: floor(x / v) with the division in IEEE single precision. */
static int quantize_axis(float x, float v, float* a_out, int32_t* q) {
    if (!isfinite(x)) return SPVO_ERR_NONFINITE;
    float a = x / v;
    if (!isfinite(a)) return SPVO_ERR_RANGE;
    double f = floor((double)a);
    if (f < (double)COORD_MIN || f > (double)COORD_MAX) return SPVO_ERR_RANGE;
    *q = (int32_t)f;
    if (a_out) *a_out = a;
    return SPVO_OK;
}

/* Validate all points: NONFINITE wins over RANGE; both scan every point. */
static int check_points(const float* xyz, const int32_t* batch, int64_t n, float v) {
    int nonfinite = 0, range = 0;
    for (int64_t k = 0; k < n; ++k) {
        for (int d = 0; d < 3; ++d) {
            int32_t q;
            int st = quantize_axis(xyz[3 * k + d], v, NULL, &q);
            if (st == SPVO_ERR_NONFINITE) nonfinite = 1;
            if (st == SPVO_ERR_RANGE) range = 1;
        }
        if (batch && (batch[k] < 0 || batch[k] > BATCH_MAX)) range = 1;
    }
    if (nonfinite) return SPVO_ERR_NONFINITE;
    if (range) return SPVO_ERR_RANGE;
    return SPVO_OK;
}

static int valid_voxel_size(float v) { return isfinite(v) && v > 0.0f; }

/* ------------------------------------------------------------------------- */
/* voxelize: Eq. 1 + Eq. 2                                                    */
/* ------------------------------------------------------------------------- */

int spvo_voxelize(const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                  const void* feat, int32_t C, int32_t dtype,
                  int32_t* coords, void* vfeat, int32_t* counts, int32_t* pt2vox,
                  int64_t* m_out) {
    if (n < 0 || n >= ((int64_t)1 << 31) || !m_out) return SPVO_ERR_INVALID_ARG;
    if (!valid_voxel_size(voxel_size)) return SPVO_ERR_INVALID_ARG;
    if (n > 0 && (!xyz || !coords || !counts || !pt2vox)) return SPVO_ERR_INVALID_ARG;
    if (feat && (C <= 0 || !vfeat || !valid_dtype(dtype))) return SPVO_ERR_INVALID_ARG;
    *m_out = 0;
    int st = check_points(xyz, batch, n, voxel_size);
    if (st) return st;

    /* Eq. 1: quantized key of every point */
    keyrec* rec = (keyrec*)malloc((size_t)(n > 0 ? n : 1) * sizeof(keyrec));
    if (!rec) return SPVO_ERR_CAPACITY;
    for (int64_t k = 0; k < n; ++k) {
        rec[k].c[0] = batch ? batch[k] : 0;
        for (int d = 0; d < 3; ++d) quantize_axis(xyz[3 * k + d], voxel_size, NULL, &rec[k].c[1 + d]);
        rec[k].idx = k;
    }
    /* the voxel set in ascending (b, x, y, z) order */
    qsort(rec, (size_t)n, sizeof(keyrec), cmp_keyrec);
    int64_t m = 0;
    for (int64_t r = 0; r < n; ++r) {
        if (r == 0 || cmp_coord(rec[r - 1].c, rec[r].c) != 0) {
            memcpy(coords + 4 * m, rec[r].c, 16);
            counts[m] = 0;
            ++m;
        }
        pt2vox[rec[r].idx] = (int32_t)(m - 1);
        counts[m - 1] += 1; /* N_m */
    }
    free(rec);

    /* Eq. 2: f_m = (1/N_m) sum_k 1[p_k in voxel m] f_k, summed in point order */
    if (feat) {
        double* acc = (double*)calloc((size_t)(m > 0 ? m : 1) * (size_t)C, sizeof(double));
        if (!acc) return SPVO_ERR_CAPACITY;
        for (int64_t k = 0; k < n; ++k) {
            double* a = acc + (int64_t)pt2vox[k] * C;
            for (int32_t c = 0; c < C; ++c) a[c] += spvo_decode(feat, k * C + c, dtype);
        }
        for (int64_t j = 0; j < m; ++j)
            for (int32_t c = 0; c < C; ++c)
                spvo_round_store(acc[j * C + c] / (double)counts[j], vfeat, j * C + c, dtype);
        free(acc);
    }
    *m_out = m;
    return SPVO_OK;
}

/* Eq. 2 onto a given voxel set: N_j and f_j over the points whose Eq. 1
 * coordinates equal coords[j]; points outside the set have pt2vox = -1, and a
 * voxel without points gets f_j = 0.  Features summed in point order. */
int spvo_voxelize_onto(const int32_t* coords, int64_t m, const float* xyz, const int32_t* batch, int64_t n,
                       float voxel_size, const void* feat, int32_t C, int32_t dtype,
                       void* vfeat, int32_t* counts, int32_t* pt2vox) {
    if (n < 0 || n >= ((int64_t)1 << 31) || m < 0 || m >= ((int64_t)1 << 31)) return SPVO_ERR_INVALID_ARG;
    if (!valid_voxel_size(voxel_size)) return SPVO_ERR_INVALID_ARG;
    if ((n > 0 && (!xyz || !pt2vox)) || (m > 0 && (!coords || !counts))) return SPVO_ERR_INVALID_ARG;
    if (feat && (C <= 0 || (m > 0 && !vfeat) || !valid_dtype(dtype))) return SPVO_ERR_INVALID_ARG;
    int st = check_points(xyz, batch, n, voxel_size);
    if (st) return st;
    if (!coords_in_range(coords, m)) return SPVO_ERR_RANGE;
    coordset set;
    st = coordset_build(&set, coords, m);
    if (st) {
        coordset_free(&set);
        return st;
    }
    for (int64_t j = 0; j < m; ++j) counts[j] = 0;
    for (int64_t k = 0; k < n; ++k) {
        int32_t c[4];
        c[0] = batch ? batch[k] : 0;
        for (int d = 0; d < 3; ++d) quantize_axis(xyz[3 * k + d], voxel_size, NULL, &c[1 + d]);
        const int64_t j = coordset_find(&set, c);
        pt2vox[k] = (int32_t)j;
        if (j >= 0) counts[j] += 1;
    }
    coordset_free(&set);
    if (feat && m > 0) {
        double* acc = (double*)calloc((size_t)m * (size_t)C, sizeof(double));
        if (!acc) return SPVO_ERR_CAPACITY;
        for (int64_t k = 0; k < n; ++k) {
            if (pt2vox[k] < 0) continue;
            double* a = acc + (int64_t)pt2vox[k] * C;
            for (int32_t c = 0; c < C; ++c) a[c] += spvo_decode(feat, k * C + c, dtype);
        }
        for (int64_t j = 0; j < m; ++j)
            for (int32_t c = 0; c < C; ++c)
                spvo_round_store(counts[j] ? acc[j * C + c] / (double)counts[j] : 0.0, vfeat, j * C + c, dtype);
        free(acc);
    }
    return SPVO_OK;
}

/* ------------------------------------------------------------------------- */
/* kernel map                                                                 */
/* ------------------------------------------------------------------------- */

/* floor(c / 2) for any sign */
static int32_t floor_half(int32_t c) { return (c >= 0) ? c / 2 : -((-c + 1) / 2); }

int spvo_kernel_map(const int32_t* in_coords, int64_t m_in, int32_t K, int32_t stride,
                    int32_t* out_coords, int64_t* m_out,
                    int32_t* off, int32_t* pairs, int64_t pair_cap, int64_t* total) {
    if (m_in < 0 || m_in >= ((int64_t)1 << 31) || !off || !total || !m_out || pair_cap < 0)
        return SPVO_ERR_INVALID_ARG;
    if (m_in > 0 && !in_coords) return SPVO_ERR_INVALID_ARG;
    if (!((K == 3 && (stride == 1 || stride == 2)) || (K == 2 && stride == 2))) return SPVO_ERR_UNSUPPORTED;
    if (stride == 2 && !out_coords) return SPVO_ERR_INVALID_ARG;
    if (!coords_in_range(in_coords, m_in)) return SPVO_ERR_RANGE;

    coordset fine;
    int st = coordset_build(&fine, in_coords, m_in);
    if (st) {
        coordset_free(&fine);
        return st;
    }
    const int K3 = K * K * K;
    int64_t mo = m_in;
    const int32_t* oc = in_coords;
    int32_t* coarse = NULL;
    if (stride == 2) {
        /* output set: the distinct floor(c/2), ascending */
        keyrec* rec = (keyrec*)malloc((size_t)(m_in > 0 ? m_in : 1) * sizeof(keyrec));
        for (int64_t i = 0; i < m_in; ++i) {
            rec[i].c[0] = in_coords[4 * i];
            for (int d = 1; d < 4; ++d) rec[i].c[d] = floor_half(in_coords[4 * i + d]);
            rec[i].idx = i;
        }
        qsort(rec, (size_t)m_in, sizeof(keyrec), cmp_keyrec);
        coarse = (int32_t*)malloc((size_t)(m_in > 0 ? m_in : 1) * 16);
        mo = 0;
        for (int64_t r = 0; r < m_in; ++r)
            if (r == 0 || cmp_coord(rec[r - 1].c, rec[r].c) != 0) memcpy(coarse + 4 * mo++, rec[r].c, 16);
        free(rec);
        oc = coarse;
    }

    /* pair (i, j, k) iff in_i = stride * out_j + delta_k; grouped by k, ascending j */
    int64_t cnt = 0;
    for (int k = 0; k < K3; ++k) {
        int32_t dlt[3];
        if (K == 3) {
            dlt[0] = k / 9 - 1;
            dlt[1] = (k / 3) % 3 - 1;
            dlt[2] = k % 3 - 1;
        } else {
            dlt[0] = (k >> 2) & 1;
            dlt[1] = (k >> 1) & 1;
            dlt[2] = k & 1;
        }
        off[k] = (int32_t)cnt;
        for (int64_t j = 0; j < mo; ++j) {
            int32_t q[4];
            q[0] = oc[4 * j];
            for (int d = 0; d < 3; ++d) q[1 + d] = stride * oc[4 * j + 1 + d] + dlt[d];
            int64_t i = coordset_find(&fine, q);
            if (i >= 0) {
                if (cnt < pair_cap && pairs) {
                    pairs[2 * cnt] = (int32_t)i;
                    pairs[2 * cnt + 1] = (int32_t)j;
                }
                ++cnt;
            }
        }
    }
    off[K3] = (int32_t)cnt;
    *total = cnt;
    *m_out = mo;
    if (stride == 2) memcpy(out_coords, coarse, (size_t)mo * 16);
    free(coarse);
    coordset_free(&fine);
    if (cnt > pair_cap) return SPVO_ERR_CAPACITY;
    return SPVO_OK;
}

/* ------------------------------------------------------------------------- */
/* sparse convolution on the map                                              */
/* ------------------------------------------------------------------------- */

/* res (NULL = none) is a residual input [m_out][Cout] of the storage type,
 * added after scale and shift and before the activation (the identity branch
 * of a residual block, Sec. 3.3 "Feature Aggregation"). */
int spvo_sparse_conv_res(const void* in, int64_t m_in, int32_t Cin,
                         const int32_t* off, const int32_t* pairs, int32_t K3, int32_t transposed,
                         const void* W, const float* scale, const float* shift, const void* res, int32_t relu,
                         void* out, int64_t m_out, int32_t Cout, int32_t dtype) {
    if (m_in < 0 || m_out < 0 || Cin <= 0 || Cout <= 0 || !off || !W || !valid_dtype(dtype))
        return SPVO_ERR_INVALID_ARG;
    if (!(K3 == 27 || K3 == 8)) return SPVO_ERR_UNSUPPORTED;
    if ((m_in > 0 && !in) || (m_out > 0 && !out)) return SPVO_ERR_INVALID_ARG;
    int64_t total = off[K3];
    if (total > 0 && !pairs) return SPVO_ERR_INVALID_ARG;
    for (int k = 0; k < K3; ++k)
        if (off[k] > off[k + 1] || off[0] != 0) return SPVO_ERR_INVALID_ARG;
    for (int64_t p = 0; p < total; ++p) {
        int64_t i = transposed ? pairs[2 * p + 1] : pairs[2 * p];
        int64_t j = transposed ? pairs[2 * p] : pairs[2 * p + 1];
        if (i < 0 || i >= m_in || j < 0 || j >= m_out) return SPVO_ERR_INVALID_ARG;
    }
    double* acc = (double*)calloc((size_t)(m_out > 0 ? m_out : 1) * (size_t)Cout, sizeof(double));
    if (!acc) return SPVO_ERR_CAPACITY;
    double* w = (double*)malloc((size_t)K3 * Cin * Cout * sizeof(double));
    for (int64_t t = 0; t < (int64_t)K3 * Cin * Cout; ++t) w[t] = spvo_decode(W, t, dtype);
    /* out[j] += in[i] @ W[k] for every pair (i, j) of offset k */
    for (int k = 0; k < K3; ++k) {
        for (int64_t p = off[k]; p < off[k + 1]; ++p) {
            int64_t i = transposed ? pairs[2 * p + 1] : pairs[2 * p];
            int64_t j = transposed ? pairs[2 * p] : pairs[2 * p + 1];
            double* a = acc + j * Cout;
            for (int32_t ci = 0; ci < Cin; ++ci) {
                double x = spvo_decode(in, i * Cin + ci, dtype);
                const double* wr = w + ((int64_t)k * Cin + ci) * Cout;
                for (int32_t co = 0; co < Cout; ++co) a[co] += x * wr[co];
            }
        }
    }
    for (int64_t j = 0; j < m_out; ++j)
        for (int32_t co = 0; co < Cout; ++co) {
            double y = acc[j * Cout + co];
            if (scale) y *= (double)scale[co];
            if (shift) y += (double)shift[co];
            if (res) y += spvo_decode(res, j * Cout + co, dtype);
            if (relu && y < 0.0) y = 0.0;
            spvo_round_store(y, out, j * Cout + co, dtype);
        }
    free(w);
    free(acc);
    return SPVO_OK;
}

int spvo_sparse_conv(const void* in, int64_t m_in, int32_t Cin,
                     const int32_t* off, const int32_t* pairs, int32_t K3, int32_t transposed,
                     const void* W, const float* scale, const float* shift, int32_t relu,
                     void* out, int64_t m_out, int32_t Cout, int32_t dtype) {
    return spvo_sparse_conv_res(in, m_in, Cin, off, pairs, K3, transposed, W, scale, shift, NULL, relu, out, m_out,
                                Cout, dtype);
}

/* ------------------------------------------------------------------------- */
/* backward passes                                                            */
/* ------------------------------------------------------------------------- */

/* weight gradient of a sparse conv: dW[k] = sum over the pairs (i, j) of offset
 * k of x[i]^T dy[j] (roles of the pair swapped with transposed = 1); fp64
 * accumulation in pair order, one rounding to float32 */
int spvo_sparse_conv_wgrad(const void* x, int64_t m_in, int32_t Cin, const void* dy, int64_t m_out, int32_t Cout,
                           const int32_t* off, const int32_t* pairs, int32_t K3, int32_t transposed, float* dW,
                           int32_t dtype) {
    if (m_in < 0 || m_out < 0 || Cin <= 0 || Cout <= 0 || !off || !dW || !valid_dtype(dtype))
        return SPVO_ERR_INVALID_ARG;
    if (!(K3 == 27 || K3 == 8)) return SPVO_ERR_UNSUPPORTED;
    for (int k = 0; k < K3; ++k)
        if (off[k] > off[k + 1] || off[0] != 0) return SPVO_ERR_INVALID_ARG;
    const int64_t total = off[K3];
    if (total > 0 && (!pairs || !x || !dy)) return SPVO_ERR_INVALID_ARG;
    double* acc = (double*)calloc((size_t)Cin * Cout, sizeof(double));
    double* xr = (double*)malloc((size_t)Cin * sizeof(double));
    double* gr = (double*)malloc((size_t)Cout * sizeof(double));
    int st = (acc && xr && gr) ? SPVO_OK : SPVO_ERR_CAPACITY;
    for (int k = 0; k < K3 && st == SPVO_OK; ++k) {
        for (int64_t t = 0; t < (int64_t)Cin * Cout; ++t) acc[t] = 0.0;
        for (int64_t p = off[k]; p < off[k + 1]; ++p) {
            const int64_t i = transposed ? pairs[2 * p + 1] : pairs[2 * p];
            const int64_t j = transposed ? pairs[2 * p] : pairs[2 * p + 1];
            if (i < 0 || i >= m_in || j < 0 || j >= m_out) {
                st = SPVO_ERR_INVALID_ARG;
                break;
            }
            /* the pair's two rows, decoded once */
            for (int32_t ci = 0; ci < Cin; ++ci) xr[ci] = spvo_decode(x, i * Cin + ci, dtype);
            for (int32_t co = 0; co < Cout; ++co) gr[co] = spvo_decode(dy, j * Cout + co, dtype);
            for (int32_t ci = 0; ci < Cin; ++ci)
                for (int32_t co = 0; co < Cout; ++co) acc[(int64_t)ci * Cout + co] += xr[ci] * gr[co];
        }
        for (int64_t t = 0; t < (int64_t)Cin * Cout; ++t) dW[(int64_t)k * Cin * Cout + t] = (float)acc[t];
    }
    free(acc);
    free(xr);
    free(gr);
    return st;
}

/* backward of the scatter-mean (Eq. 2): every point receives its voxel's
 * gradient divided by the voxel's point count N_m; one rounding */
int spvo_voxelize_backward(const void* dv, int64_t m, int32_t C, const int32_t* counts, const int32_t* pt2vox,
                           int64_t n, void* dfeat, int32_t dtype) {
    if (m < 0 || n < 0 || C <= 0 || !valid_dtype(dtype)) return SPVO_ERR_INVALID_ARG;
    if (n > 0 && (!pt2vox || !dfeat || !counts || !dv)) return SPVO_ERR_INVALID_ARG;
    for (int64_t k = 0; k < n; ++k) {
        const int64_t v = pt2vox[k];
        if (v < 0 || v >= m || counts[v] <= 0) return SPVO_ERR_INVALID_ARG;
        for (int32_t c = 0; c < C; ++c)
            spvo_round_store(spvo_decode(dv, v * C + c, dtype) / (double)counts[v], dfeat, k * C + c, dtype);
    }
    return SPVO_OK;
}

/* backward of the trilinear devoxelization w.r.t. the voxel features: point k
 * scatters dout[k] times the weight its corner c had -- the raw weight over the
 * sum of the present corners' raw weights -- to voxel idx[k][c]; fp64 sums,
 * one rounding to float32 */
int spvo_devoxelize_backward(const int32_t* cidx, const float* cw, const void* dout, int64_t n, int32_t C, float* dv,
                             int64_t m, int32_t dtype) {
    if (n < 0 || m < 0 || C <= 0 || !valid_dtype(dtype) || (m > 0 && !dv)) return SPVO_ERR_INVALID_ARG;
    if (n > 0 && (!cidx || !cw || !dout)) return SPVO_ERR_INVALID_ARG;
    double* acc = (double*)calloc((size_t)(m > 0 ? m : 1) * C, sizeof(double));
    if (!acc) return SPVO_ERR_CAPACITY;
    for (int64_t k = 0; k < n; ++k) {
        double den = 0.0;
        for (int c = 0; c < 8; ++c)
            if (cidx[8 * k + c] >= 0) den += (double)cw[8 * k + c];
        if (den <= 0.0) continue;
        for (int c = 0; c < 8; ++c) {
            const int64_t v = cidx[8 * k + c];
            if (v < 0) continue;
            if (v >= m) {
                free(acc);
                return SPVO_ERR_INVALID_ARG;
            }
            const double w = (double)cw[8 * k + c] / den;
            for (int32_t ch = 0; ch < C; ++ch) acc[v * C + ch] += w * spvo_decode(dout, k * C + ch, dtype);
        }
    }
    for (int64_t t = 0; t < m * C; ++t) dv[t] = (float)acc[t];
    free(acc);
    return SPVO_OK;
}

/* ------------------------------------------------------------------------- */
/* pointwise linear layer                                                     */
/* ------------------------------------------------------------------------- */

/* out[i] = act(scale * (in[i] @ W) + shift [+ res[i]]) [+ res[i]]: the point
 * branch's MLP (Sec. 3.3 "Point Transformation and Feature Fusion": linear, then
 * normalization and activation, then fusion by addition -- res after act), a 1x1
 * shortcut of a residual block (res before act), or a classifier (shift = bias). */
int spvo_linear(const void* in, int64_t m, int32_t Cin, const void* W, const float* scale, const float* shift,
                const void* res, int32_t res_after_act, int32_t relu, void* out, int32_t Cout, int32_t dtype) {
    if (m < 0 || Cin <= 0 || Cout <= 0 || !W || !valid_dtype(dtype)) return SPVO_ERR_INVALID_ARG;
    if (m > 0 && (!in || !out)) return SPVO_ERR_INVALID_ARG;
    double* w = (double*)malloc((size_t)Cin * Cout * sizeof(double));
    double* acc = (double*)malloc((size_t)Cout * sizeof(double));
    if (!w || !acc) {
        free(w);
        free(acc);
        return SPVO_ERR_CAPACITY;
    }
    for (int64_t t = 0; t < (int64_t)Cin * Cout; ++t) w[t] = spvo_decode(W, t, dtype);
    for (int64_t i = 0; i < m; ++i) {
        for (int32_t co = 0; co < Cout; ++co) acc[co] = 0.0;
        for (int32_t ci = 0; ci < Cin; ++ci) {
            const double x = spvo_decode(in, i * Cin + ci, dtype);
            for (int32_t co = 0; co < Cout; ++co) acc[co] += x * w[(int64_t)ci * Cout + co];
        }
        for (int32_t co = 0; co < Cout; ++co) {
            double y = acc[co];
            if (scale) y *= (double)scale[co];
            if (shift) y += (double)shift[co];
            const double r = res ? spvo_decode(res, i * Cout + co, dtype) : 0.0;
            if (!res_after_act) y += r;
            if (relu && y < 0.0) y = 0.0;
            if (res_after_act) y += r;
            spvo_round_store(y, out, i * Cout + co, dtype);
        }
    }
    free(w);
    free(acc);
    return SPVO_OK;
}

/* backward of the epilogue: the activation's input is formed in float32 the
 * way the kernels form it, so that both take the ReLU's decision on the same
 * value; everything after it is fp64 */
int spvo_epilogue_backward(const void* dy, const void* a, const float* scale, const float* shift, int32_t relu,
                           const void* res, int32_t res_after_act, int64_t m, int32_t C, void* da, void* dres,
                           float* dscale, float* dshift, int32_t dtype) {
    if (m < 0 || C <= 0 || !valid_dtype(dtype)) return SPVO_ERR_INVALID_ARG;
    if (m > 0 && (!dy || !a)) return SPVO_ERR_INVALID_ARG;
    double* ss = (double*)calloc((size_t)C, sizeof(double));
    double* sb = (double*)calloc((size_t)C, sizeof(double));
    if (!ss || !sb) {
        free(ss);
        free(sb);
        return SPVO_ERR_CAPACITY;
    }
    for (int64_t i = 0; i < m; ++i) {
        for (int32_t c = 0; c < C; ++c) {
            const int64_t t = i * C + c;
            const float av = (float)spvo_decode(a, t, dtype);
            const float s = scale ? scale[c] : 1.0f, b = shift ? shift[c] : 0.0f;
            float z = fmaf(av, s, b);
            if (res && !res_after_act) z = z + (float)spvo_decode(res, t, dtype);
            const double g = spvo_decode(dy, t, dtype);
            const double gz = (!relu || z > 0.0f) ? g : 0.0;
            if (da) spvo_round_store(gz * (double)s, da, t, dtype);
            if (dres) spvo_round_store(res_after_act ? g : gz, dres, t, dtype);
            ss[c] += gz * (double)av;
            sb[c] += gz;
        }
    }
    for (int32_t c = 0; c < C; ++c) {
        if (dscale) dscale[c] = (float)ss[c];
        if (dshift) dshift[c] = (float)sb[c];
    }
    free(ss);
    free(sb);
    return SPVO_OK;
}

int spvo_linear_backward(const void* in, int64_t m, int32_t Cin, const void* W, int32_t Cout, const void* da,
                         void* din, float* dW, int32_t dtype) {
    if (m < 0 || Cin <= 0 || Cout <= 0 || !W || !valid_dtype(dtype)) return SPVO_ERR_INVALID_ARG;
    if (m > 0 && (!in || !da)) return SPVO_ERR_INVALID_ARG;
    double* acc = (double*)calloc((size_t)Cin * Cout, sizeof(double));
    if (!acc) return SPVO_ERR_CAPACITY;
    for (int64_t i = 0; i < m; ++i) {
        for (int32_t ci = 0; ci < Cin; ++ci) {
            const double x = spvo_decode(in, i * Cin + ci, dtype);
            double s = 0.0;
            for (int32_t co = 0; co < Cout; ++co) {
                const double g = spvo_decode(da, i * Cout + co, dtype);
                s += g * spvo_decode(W, (int64_t)ci * Cout + co, dtype);
                acc[(int64_t)ci * Cout + co] += x * g;
            }
            if (din) spvo_round_store(s, din, i * Cin + ci, dtype);
        }
    }
    if (dW)
        for (int64_t t = 0; t < (int64_t)Cin * Cout; ++t) dW[t] = (float)acc[t];
    free(acc);
    return SPVO_OK;
}

/* ------------------------------------------------------------------------- */
/* devoxelize (trilinear over 8 neighbour voxels) + point MLP + add           */
/* ------------------------------------------------------------------------- */

int spvo_devoxelize(const int32_t* grid_coords, int64_t m, int32_t stride_log2,
                    const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                    int32_t mode, const void* vfeat, int32_t C,
                    const void* pfeat, int32_t Cp, const void* Wp,
                    const float* scale_p, const float* shift_p, int32_t relu_p,
                    void* out, int32_t dtype, int32_t* corner_idx, float* corner_w) {
    if (n < 0 || n >= ((int64_t)1 << 31) || m < 0 || C <= 0 || !valid_dtype(dtype))
        return SPVO_ERR_INVALID_ARG;
    if (!valid_voxel_size(voxel_size) || stride_log2 < 0 || stride_log2 > 15) return SPVO_ERR_INVALID_ARG;
    if (mode != SPVO_DEVOX_CENTER && mode != SPVO_DEVOX_CORNER && mode != SPVO_DEVOX_NEAREST)
        return SPVO_ERR_INVALID_ARG;
    if (n > 0 && (!xyz || !out)) return SPVO_ERR_INVALID_ARG;
    if (m > 0 && (!grid_coords || !vfeat)) return SPVO_ERR_INVALID_ARG;
    if (pfeat && (Cp <= 0 || !Wp)) return SPVO_ERR_INVALID_ARG;
    if (!coords_in_range(grid_coords, m)) return SPVO_ERR_RANGE;
    int st = check_points(xyz, batch, n, voxel_size);
    if (st) return st;
    coordset grid;
    st = coordset_build(&grid, grid_coords, m);
    if (st) {
        coordset_free(&grid);
        return st;
    }
    const float sfac = ldexpf(1.0f, -stride_log2);
    double* y = (double*)malloc((size_t)C * sizeof(double));
    double* num = (double*)malloc((size_t)C * sizeof(double));
    for (int64_t k = 0; k < n; ++k) {
        int32_t b = batch ? batch[k] : 0;
        float t[3];
        int32_t base[3];
        for (int d = 0; d < 3; ++d) {
            float a = 0.0f;
            int32_t q;
            quantize_axis(xyz[3 * k + d], voxel_size, &a, &q);
            float as = a * sfac; /* exact power-of-two scaling */
            /* CENTER: voxel q's feature sits at its centre, so shift by half a voxel */
            float u = (mode == SPVO_DEVOX_CENTER) ? as - 0.5f : as;
            float fb = floorf(u);
            base[d] = (int32_t)fb;
            /* NEAREST: the voxel containing the point takes all the weight (corner 0) */
            t[d] = (mode == SPVO_DEVOX_NEAREST) ? 0.0f : u - fb;
        }
        double den = 0.0;
        for (int32_t c = 0; c < C; ++c) num[c] = 0.0;
        for (int c8 = 0; c8 < 8; ++c8) {
            int cx = (c8 >> 2) & 1, cy = (c8 >> 1) & 1, cz = c8 & 1;
            float wx = cx ? t[0] : 1.0f - t[0];
            float wy = cy ? t[1] : 1.0f - t[1];
            float wz = cz ? t[2] : 1.0f - t[2];
            float w = wx * wy;
            w = w * wz;
            int32_t q[4] = {b, base[0] + cx, base[1] + cy, base[2] + cz};
            int64_t idx = coordset_find(&grid, q);
            if (corner_idx) corner_idx[8 * k + c8] = (int32_t)idx;
            if (corner_w) corner_w[8 * k + c8] = w;
            if (idx < 0) continue; /* absent corner: weight 0, renormalized below */
            den += (double)w;
            for (int32_t c = 0; c < C; ++c) num[c] += (double)w * spvo_decode(vfeat, idx * C + c, dtype);
        }
        for (int32_t c = 0; c < C; ++c) y[c] = (den > 0.0) ? num[c] / den : 0.0;
        if (pfeat) {
            for (int32_t c = 0; c < C; ++c) {
                double s = 0.0;
                for (int32_t ci = 0; ci < Cp; ++ci)
                    s += spvo_decode(pfeat, k * Cp + ci, dtype) * spvo_decode(Wp, (int64_t)ci * C + c, dtype);
                if (scale_p) s *= (double)scale_p[c];
                if (shift_p) s += (double)shift_p[c];
                if (relu_p && s < 0.0) s = 0.0;
                y[c] += s; /* fusion by addition */
            }
        }
        for (int32_t c = 0; c < C; ++c) spvo_round_store(y[c], out, k * C + c, dtype);
    }
    free(y);
    free(num);
    coordset_free(&grid);
    return SPVO_OK;
}

/* ------------------------------------------------------------------------- */
/* the SPVConv block                                                          */
/* ------------------------------------------------------------------------- */

int spvo_block(const spvo_block_params* p, const float* xyz, const int32_t* batch,
               int64_t n, const void* feat, void* out, int64_t* m_out) {
    if (!p || !m_out || n < 0 || p->C <= 0 || !valid_dtype(p->dtype)) return SPVO_ERR_INVALID_ARG;
    if (p->n_convs < 1 || p->n_convs > 2 || !p->Wp) return SPVO_ERR_INVALID_ARG;
    for (int l = 0; l < p->n_convs; ++l)
        if (!p->W[l]) return SPVO_ERR_INVALID_ARG;
    if (n > 0 && (!xyz || !feat || !out)) return SPVO_ERR_INVALID_ARG;
    const int32_t C = p->C;
    const size_t es = (p->dtype == SPVO_F32) ? 4 : 2;
    const size_t nn = (size_t)(n > 0 ? n : 1);
    int32_t* coords = (int32_t*)malloc(nn * 16);
    int32_t* counts = (int32_t*)malloc(nn * 4);
    int32_t* pt2vox = (int32_t*)malloc(nn * 4);
    void* va = malloc(nn * (size_t)C * es);
    void* vb = malloc(nn * (size_t)C * es);
    int32_t* off = (int32_t*)malloc(28 * 4);
    int32_t* pairs = (int32_t*)malloc(nn * 27 * 8);
    int64_t m = 0, mo = 0, total = 0;
    int st = spvo_voxelize(xyz, batch, n, p->voxel_size, feat, C, p->dtype, coords, va, counts, pt2vox, &m);
    if (!st) st = spvo_kernel_map(coords, m, 3, 1, NULL, &mo, off, pairs, (int64_t)nn * 27, &total);
    /* residual: the last conv adds the block's voxel input x before its activation */
    void* x = p->residual ? malloc(nn * (size_t)C * es) : NULL;
    if (x && !st) memcpy(x, va, (size_t)(m > 0 ? m : 1) * (size_t)C * es);
    for (int l = 0; l < p->n_convs && !st; ++l) {
        const void* res = (x && l == p->n_convs - 1) ? x : NULL;
        st = spvo_sparse_conv_res(va, m, C, off, pairs, 27, 0, p->W[l], p->scale[l], p->shift[l], res, p->relu[l],
                                  vb, m, C, p->dtype);
        void* t = va;
        va = vb;
        vb = t;
    }
    free(x);
    if (!st)
        st = spvo_devoxelize(coords, m, 0, xyz, batch, n, p->voxel_size, p->devox_mode, va, C, feat, C, p->Wp,
                             p->scale_p, p->shift_p, p->relu_p, out, p->dtype, NULL, NULL);
    *m_out = st ? 0 : m;
    free(coords);
    free(counts);
    free(pt2vox);
    free(va);
    free(vb);
    free(off);
    free(pairs);
    return st;
}
