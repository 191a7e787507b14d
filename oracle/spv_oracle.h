/*
 * spv_oracle.h -- plain, slow, single-threaded CPU oracle for the SPVConv hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the bench's
 * CPU-baseline leg may load this library.  It shares no code, header, table or
 * helper with the HIP library; the two agree only on the documented interface
 * (argument meaning, layouts and status numbers).
 *
 * What it computes (paper: "Searching Efficient 3D Architectures with Sparse
 * Point-Voxel Convolution", Sec. 3.3):
 *   spvo_voxelize    Eq. 1 (floor quantization) and Eq. 2 (mean of the point
 *                    features that fall into each non-empty voxel).
 *   spvo_kernel_map  the "kernel map" of Sec. 3.2: all active synapses between
 *                    input and output voxels, outputs restricted to input sites
 *                    (submanifold, K=3) or to the halved grid (K=2, stride 2).
 *   spvo_sparse_conv the convolution evaluated on that map (Sec. 3.2, 3.3
 *                    "Feature Aggregation").
 *   spvo_devoxelize  trilinear interpolation from the 8 neighbouring voxels
 *                    (Sec. 3.3 "Sparse Devoxelization"), plus the point-branch
 *                    MLP and the fusion by addition ("Point Transformation and
 *                    Feature Fusion").
 *   spvo_block       the SPVConv block of Fig. 2 composed from the above.
 *
 * All pointers are host pointers.  Feature storage dtype: 0 = float32,
 * 1 = bfloat16 bits, 2 = float16 bits.  Accumulation is fp64; each op rounds its
 * result once (round to nearest even) into the storage dtype.
 */
#ifndef SPV_ORACLE_H
#define SPV_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

/* status numbers (identical meaning to the HIP library's) */
#define SPVO_OK 0
#define SPVO_ERR_INVALID_ARG 1
#define SPVO_ERR_CAPACITY 2
#define SPVO_ERR_RANGE 3
#define SPVO_ERR_NONFINITE 4
#define SPVO_ERR_UNSUPPORTED 5

#define SPVO_F32 0
#define SPVO_BF16 1
#define SPVO_F16 2

#define SPVO_DEVOX_CENTER 0
#define SPVO_DEVOX_CORNER 1
#define SPVO_DEVOX_NEAREST 2 /* the point's own voxel only (the interpolation the paper sets trilinear against) */

/* Voxelize n points (Eq. 1, Eq. 2).  Outputs hold up to n voxels, in ascending
 * (batch, x, y, z) order.  feat may be NULL (C ignored): then only coordinates,
 * counts and pt2vox are produced.  coords is [m][4] = (b, x, y, z). */
int spvo_voxelize(const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                  const void* feat, int32_t C, int32_t dtype,
                  int32_t* coords, void* vfeat, int32_t* counts, int32_t* pt2vox,
                  int64_t* m_out);

/* Eq. 2 onto a given set of m distinct voxels coords[m][4] (output row j =
 * coords row j): counts[j] = N_j, vfeat[j] = mean of the features of those
 * points (0 when N_j = 0), pt2vox[k] = j or -1 when the point's voxel is not
 * in the set.  Duplicate coordinates: SPVO_ERR_INVALID_ARG. */
int spvo_voxelize_onto(const int32_t* coords, int64_t m, const float* xyz, const int32_t* batch, int64_t n,
                       float voxel_size, const void* feat, int32_t C, int32_t dtype,
                       void* vfeat, int32_t* counts, int32_t* pt2vox);

/* Kernel map.  K=3 stride=1: submanifold (outputs = inputs).  Stride 2 (K=2 or
 * K=3): outputs = unique floor(c/2), written to out_coords in ascending order;
 * (in, out) is a pair of offset k iff in = 2 out + delta_k (delta in {0,1}^3 for
 * K=2, {-1,0,1}^3 for K=3).  Pairs (in, out) grouped by offset k (CSR
 * off[K^3+1]), each group sorted by out. */
int spvo_kernel_map(const int32_t* in_coords, int64_t m_in, int32_t K, int32_t stride,
                    int32_t* out_coords, int64_t* m_out,
                    int32_t* off, int32_t* pairs, int64_t pair_cap, int64_t* total);

/* Sparse conv on a kernel map.  W is [K3][Cin][Cout] in the storage dtype;
 * scale/shift are float32 [Cout] or NULL (identity); relu 0/1.
 * transposed=1 uses each pair with its roles swapped (out, in). */
int spvo_sparse_conv(const void* in, int64_t m_in, int32_t Cin,
                     const int32_t* off, const int32_t* pairs, int32_t K3, int32_t transposed,
                     const void* W, const float* scale, const float* shift, int32_t relu,
                     void* out, int64_t m_out, int32_t Cout, int32_t dtype);
/* the same with a residual input res [m_out][Cout] (NULL = none), added after
 * scale and shift and before the activation */
int spvo_sparse_conv_res(const void* in, int64_t m_in, int32_t Cin,
                         const int32_t* off, const int32_t* pairs, int32_t K3, int32_t transposed,
                         const void* W, const float* scale, const float* shift, const void* res, int32_t relu,
                         void* out, int64_t m_out, int32_t Cout, int32_t dtype);

/* Backward passes.  Weight gradient of a sparse conv (float32 dW [K3][Cin][Cout]),
 * the scatter-mean's backward (dfeat[k] = dv[pt2vox[k]] / N), and the
 * devoxelization's backward w.r.t. the voxel features (float32 dv [m][C]) from the
 * corner indices / raw weights that spvo_devoxelize reports. */
int spvo_sparse_conv_wgrad(const void* x, int64_t m_in, int32_t Cin, const void* dy, int64_t m_out, int32_t Cout,
                           const int32_t* off, const int32_t* pairs, int32_t K3, int32_t transposed, float* dW,
                           int32_t dtype);
int spvo_voxelize_backward(const void* dv, int64_t m, int32_t C, const int32_t* counts, const int32_t* pt2vox,
                           int64_t n, void* dfeat, int32_t dtype);
int spvo_devoxelize_backward(const int32_t* cidx, const float* cw, const void* dout, int64_t n, int32_t C, float* dv,
                             int64_t m, int32_t dtype);

/* Pointwise linear layer: out[i] = act(scale * (in[i] @ W) + shift + res[i]) with
 * res_after_act = 0, act(scale * (in[i] @ W) + shift) + res[i] with 1.  W is
 * [Cin][Cout] (storage dtype); scale/shift f32 [Cout] or NULL; res [m][Cout] or NULL. */
int spvo_linear(const void* in, int64_t m, int32_t Cin, const void* W, const float* scale, const float* shift,
                const void* res, int32_t res_after_act, int32_t relu, void* out, int32_t Cout, int32_t dtype);

/* Backward of the epilogue the convolutions and linear layers apply to their
 * raw product a (Sec. 3.3's BN folded into scale / shift, then ReLU, with the
 * residual before or after it):
 *   z = fmaf(a, scale, shift) (+ res when res_after_act = 0), in float32;
 *   gz = dy where relu = 0 or z > 0, else 0;
 *   da = gz * scale (one rounding to dtype); dres = dy (res_after_act = 1) or gz;
 *   dscale[c] = sum_i gz * a, dshift[c] = sum_i gz (fp64 sums, one rounding).
 * scale / shift / res may be NULL (1, 0, 0); any output may be NULL. */
int spvo_epilogue_backward(const void* dy, const void* a, const float* scale, const float* shift, int32_t relu,
                           const void* res, int32_t res_after_act, int64_t m, int32_t C, void* da, void* dres,
                           float* dscale, float* dshift, int32_t dtype);

/* Gradients of the product out = in @ W: din = da @ W^T (one rounding to dtype),
 * dW = in^T @ da (float32); fp64 sums. */
int spvo_linear_backward(const void* in, int64_t m, int32_t Cin, const void* W, int32_t Cout, const void* da,
                         void* din, float* dW, int32_t dtype);

/* Devoxelize from a grid of voxel size voxel_size * 2^stride_log2 (coords in
 * that grid's units), optionally add the point MLP act(scale*(pfeat @ Wp)+shift).
 * corner_idx [n][8] / corner_w [n][8] (optional) receive the corner voxel index
 * (-1 if absent) and the raw trilinear weight of each corner. */
int spvo_devoxelize(const int32_t* grid_coords, int64_t m, int32_t stride_log2,
                    const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                    int32_t mode, const void* vfeat, int32_t C,
                    const void* pfeat, int32_t Cp, const void* Wp,
                    const float* scale_p, const float* shift_p, int32_t relu_p,
                    void* out, int32_t dtype, int32_t* corner_idx, float* corner_w);

/* SPVConv block: voxelize -> submanifold map -> n_convs x (conv + scale/shift
 * + ReLU) -> devoxelize + point MLP + add.  Channel count C throughout. */
typedef struct {
    int32_t C;
    int32_t dtype;
    float voxel_size;
    int32_t n_convs;            /* 1 or 2 */
    const void* W[2];           /* [27][C][C] */
    const float* scale[2];      /* [C] or NULL */
    const float* shift[2];      /* [C] or NULL */
    int32_t relu[2];
    const void* Wp;             /* [C][C] */
    const float* scale_p;       /* [C] or NULL */
    const float* shift_p;       /* [C] or NULL */
    int32_t relu_p;
    int32_t devox_mode;
    int32_t residual; /* nonzero: the last conv adds the block's voxel input before its activation */
} spvo_block_params;

int spvo_block(const spvo_block_params* p, const float* xyz, const int32_t* batch,
               int64_t n, const void* feat, void* out, int64_t* m_out);

/* storage conversion helpers exposed for the tests */
double spvo_decode(const void* buf, int64_t i, int32_t dtype);
void spvo_round_store(double x, void* buf, int64_t i, int32_t dtype);

#ifdef __cplusplus
}
#endif
#endif
