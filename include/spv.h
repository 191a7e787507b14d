/*
 * spv.h -- C ABI of libspv.so: the SPVConv hot path on one AMD Instinct MI355X
 * (gfx950), in hand-written HIP.
 *
 * The operations follow the paper "Searching Efficient 3D Architectures with
 * Sparse Point-Voxel Convolution" (Tang et al., ECCV 2020), Sec. 3.3 and Fig. 2:
 * a point cloud T = {(p_k, f_k)} is voxelized into a sparse tensor
 * S = ({(p_m, f_m)}, v) through a GPU hash table, convolved with sparse
 * convolutions built on kernel maps, and devoxelized back to the points by
 * trilinear interpolation, where it is fused by addition with a per-point MLP.
 *
 * Conventions (all entry points):
 *  - Tensor pointers are DEVICE pointers, row-major, allocated and owned by the
 *    caller.  The library never allocates device memory.  Scratch memory (hash
 *    tables, sort buffers, counters, the device status word) lives in a
 *    caller-provided workspace `ws` of `ws_bytes` bytes; the size each call needs
 *    comes from spv_workspace_bytes / spv_block_workspace_bytes.  The workspace
 *    must be 256-byte aligned and must not be shared by calls that overlap in time.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *    enqueues work on it and returns; nothing synchronizes unless an optional
 *    host read-back pointer (`*_host`) is non-NULL.
 *  - Sizes that only the device knows (the number of voxels m, the number of
 *    kernel-map pairs) are exchanged through device int64 counters (`*_dev`);
 *    host-side capacities (`*_cap`) bound every buffer.
 *  - Host-detectable errors return before any launch with outputs untouched.
 *    Device-detected errors (non-finite or out-of-range coordinates, exhausted
 *    capacity) are recorded in the workspace status word: spv_status_check
 *    (which synchronizes) or any call given a host read-back pointer returns them.
 *    Every call that can record such an error clears the status word when it
 *    starts, also when it has nothing to compute; spv_sparse_conv_nbr,
 *    spv_sparse_conv_up, spv_linear and spv_sparse_conv_wgrad record none and
 *    leave it as it is.  After a device
 *    error the contents of the outputs are unspecified (but every access stays
 *    inside the caller's buffers).
 *  - Feature storage dtype: SPV_F32, SPV_BF16 or SPV_F16; weights use the
 *    feature dtype; feature and weight pointers must be 16-byte aligned;
 *    BatchNorm-style scale/shift vectors are always float32.  bf16/f16 math
 *    accumulates in fp32 on matrix cores (MFMA).
 *  - Voxel coordinates are int32 (b, x, y, z) with x, y, z in [-32767, 32766]
 *    and batch b in [0, 65534]; they are packed into 64-bit hash keys.
 *    Voxel lists are in ascending (b, x, y, z) order (the canonical order).
 */
#ifndef SPV_H
#define SPV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum spv_status {
    SPV_OK = 0,
    SPV_ERR_INVALID_ARG = 1, /* null pointer, bad size, bad voxel size / dtype / K / stride */
    SPV_ERR_CAPACITY = 2,    /* workspace or output capacity too small */
    SPV_ERR_RANGE = 3,       /* a voxel coordinate or batch index outside the key range */
    SPV_ERR_NONFINITE = 4,   /* NaN or Inf in xyz */
    SPV_ERR_UNSUPPORTED = 5, /* shape / dtype combination not implemented */
    SPV_ERR_HIP = 6          /* HIP runtime error; see spv_last_hip_error() */
} spv_status;

typedef enum spv_dtype { SPV_F32 = 0, SPV_BF16 = 1, SPV_F16 = 2 } spv_dtype;

/* Where a voxel's feature sits for trilinear interpolation (Sec. 3.3, "Sparse
 * Devoxelization"): CENTER = at the voxel centre (q + 1/2) v, CORNER = at q v.
 * NEAREST is the nearest-voxel interpolation the paper weighs trilinear
 * against: a point takes the feature of the voxel that contains it (at the
 * grid's stride), or 0 if the grid lacks that voxel -- CORNER's corners with
 * all of the weight on corner 0. */
typedef enum spv_devox_mode {
    SPV_DEVOX_CENTER = 0,
    SPV_DEVOX_CORNER = 1,
    SPV_DEVOX_NEAREST = 2
} spv_devox_mode;

/* Workspace bytes sufficient for spv_voxelize, spv_kernel_map, spv_sparse_conv,
 * spv_devoxelize and spv_lookup on at most max_points points / voxels. */
size_t spv_workspace_bytes(int64_t max_points, int32_t max_C);

/*
 * spv_voxelize -- sparse voxelization (Sec. 3.3, Eq. 1 and Eq. 2).
 *   p_hat_k = floor(p_k / v) per axis (IEEE single-precision division, floor
 *   toward -inf); the non-empty voxels are found with a GPU hash table on the
 *   packed (b, x, y, z) keys; f_m = (1/N_m) sum of the features of the points in
 *   voxel m (fp32 accumulation, one rounding to dt).
 * In:  xyz [n][3] f32; batch [n] i32 or NULL (all 0); feat [n][C] (dt) or NULL.
 * Out: coords [cap][4] i32 (b,x,y,z) in ascending key order; vfeat [cap][C]
 *      (dt, unused when feat is NULL); counts [cap] i32 = N_m; pt2vox [n] i32;
 *      m_dev (device int64) = m.  Capacity cap = n suffices since m <= n.
 *      m_host (host, optional): when non-NULL the call synchronizes, stores m
 *      and returns any device-detected error.
 * Errors: SPV_ERR_INVALID_ARG (v <= 0 or non-finite, n < 0, null pointers,
 *      C <= 0 with feat), SPV_ERR_CAPACITY (ws too small), device-detected
 *      SPV_ERR_NONFINITE (xyz) and SPV_ERR_RANGE (coordinate / batch range).
 */
spv_status spv_voxelize(void* stream, void* ws, size_t ws_bytes,
                        const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                        const void* feat, int32_t C, spv_dtype dt,
                        int32_t* coords, void* vfeat, int32_t* counts, int32_t* pt2vox,
                        int64_t* m_dev, int64_t* m_host);

/*
 * spv_voxelize_onto -- the scatter-mean of Eq. 2 onto a given voxel set (the
 * re-voxelization of Sec. 3.3's later SPVConv modules, whose voxels at each
 * stride are already known): point k belongs to the voxel of coords whose
 * coordinates equal its Eq. 1 key at voxel_size;
 *   f_j = (1/N_j) sum of the features of the points of voxel j,
 * summed exactly for 16-bit features (fp64) and rounded once to dt; a voxel
 * of the set that no point falls into gets N_j = 0 and f_j = 0, and a point
 * whose voxel is not in the set gets pt2vox = -1 and adds to nothing.  No sort:
 * a hash table of the given set, one probe per point, a counting sort of the
 * points by voxel.  With coords = the output of spv_voxelize on the same
 * points and voxel size, the results equal spv_voxelize's.
 * In:  coords [m_cap][4] i32 (distinct; any order: output row j is coords
 *      row j); m_dev: device count (NULL = m_cap); xyz, batch, feat, C, dt as
 *      in spv_voxelize (feat may be NULL: counts and pt2vox only).
 * Out: vfeat [m_cap][C] (dt; rows < count written), counts [m_cap] i32 = N_j,
 *      pt2vox [n] i32.  Workspace: spv_workspace_bytes(max(n, m_cap), C).
 * Errors: as spv_voxelize; duplicate coordinates in the set are a
 *      device-detected SPV_ERR_INVALID_ARG.
 */
spv_status spv_voxelize_onto(void* stream, void* ws, size_t ws_bytes,
                             const int32_t* coords, const int64_t* m_dev, int64_t m_cap,
                             const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                             const void* feat, int32_t C, spv_dtype dt,
                             void* vfeat, int32_t* counts, int32_t* pt2vox);

/*
 * spv_kernel_map -- the kernel map of a sparse convolution (Sec. 3.2: all
 * active synapses between input and output voxels; Sec. 3.3 "Feature
 * Aggregation": built with the same GPU hash table as the voxelization).
 *   K=3, stride=1 (submanifold): outputs = the input voxels; pair (i, j, k) iff
 *     c_i = c_j + delta_k, delta_k in {-1,0,1}^3, k = 9(dx+1) + 3(dy+1) + (dz+1).
 *   K=2, stride=2 (downsampling): outputs = the distinct floor(c_i / 2), written
 *     to out_coords in ascending order; pair iff c_i = 2 c_j + delta_k with
 *     delta_k in {0,1}^3, k = 4 dx + 2 dy + dz.  The same pairs, used with
 *     transposed=1 in spv_sparse_conv, give the matching upsampling conv.
 *   K=3, stride=2 (downsampling with a 3x3x3 kernel, Sec. 3.2's strided sparse
 *     convolution): the same outputs as K=2; pair iff c_i = 2 c_j + delta_k with
 *     delta_k in {-1,0,1}^3, k = 9(dx+1) + 3(dy+1) + (dz+1).  An input is in at
 *     most 8 pairs (2 per odd coordinate), so pair_cap = 8 m_cap suffices.
 * In:  in_coords [m_cap][4] i32 (distinct); m_in_dev: device count (NULL = m_cap).
 * Out: out_coords [m_cap][4] (stride 2 only; may be NULL for stride 1);
 *      m_out_dev (device int64, may be NULL); off [K^3+1] i32 (CSR by offset,
 *      device); pairs [pair_cap][2] i32 as (in, out), grouped by k and sorted by
 *      out within a group.  total_host (optional): synchronizes and stores the
 *      number of pairs; SPV_ERR_CAPACITY if it exceeds pair_cap (K^3 * m_cap
 *      always suffices; for K=2 stride 2, m_cap does).
 */
spv_status spv_kernel_map(void* stream, void* ws, size_t ws_bytes,
                          const int32_t* in_coords, const int64_t* m_in_dev, int64_t m_cap,
                          int32_t K, int32_t stride,
                          int32_t* out_coords, int64_t* m_out_dev,
                          int32_t* off, int32_t* pairs, int64_t pair_cap, int64_t* total_host);

/*
 * spv_sparse_conv -- convolution on a kernel map (Sec. 3.2 / 3.3):
 *   out[j] = act(scale * sum_{(i, j, k)} in[i] @ W[k] + shift)
 * with act = ReLU when relu != 0.  transposed=1 uses every pair (i, j) with its
 * roles swapped, which turns a stride-2 map into the upsampling conv onto the
 * fine voxels.  Output rows with no pair get act(shift).
 * In:  in [in_rows][Cin] (dt); off [K3+1] / pairs [pair_cap][2] from spv_kernel_map
 *      (device; pairs past pair_cap and indices outside [0, in_rows) /
 *      [0, m_out) are ignored; within each offset the output rows must
 *      strictly increase -- a map with a pair out of order, or with two pairs
 *      for one (output, offset), sets SPV_ERR_INVALID_ARG in the workspace
 *      status, reported by spv_status_check); K3 = 27 or 8;
 *      W [K3][Cin][Cout] (dt);
 *      scale/shift [Cout] f32 or NULL.
 * Out: out [m_out_cap][Cout] (dt); rows < *m_out_dev are written (m_out_dev
 *      NULL = m_out_cap).
 * bf16/f16 with Cin % 8 == 0 and Cout % 16 == 0 run on MFMA; other shapes and
 * f32 run on a vector-ALU kernel with fp32 accumulation.
 */
spv_status spv_sparse_conv(void* stream, void* ws, size_t ws_bytes,
                           const void* in, int64_t in_rows, int32_t Cin,
                           const int32_t* off, const int32_t* pairs, int64_t pair_cap,
                           int32_t K3, int32_t transposed,
                           const void* W, const float* scale, const float* shift, int32_t relu,
                           void* out, const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout,
                           spv_dtype dt);

/*
 * spv_sparse_conv_sliced -- spv_sparse_conv with shared, channel-sliced weights
 * (Sec. 4.2 "Weight Sharing": a candidate layer of the super network with C_in
 * input and C_out output channels uses the first C_in input and the first C_out
 * output channels of the layer's full weight tensor, and its normalization the
 * first C_out entries of the full scale / shift).
 *   out[j] = act(scale[:Cout] * sum_{(i, j, k)} in[i] @ W[k][:Cin][:Cout] + shift[:Cout])
 * With res non-NULL the layer also adds a residual input before the activation:
 *   out[j] = act(scale * conv + shift + res[j])
 * (the second conv of a residual block adds its shortcut, Sec. 3.3; a conv
 * over concatenated inputs [a; b] is W_a a + W_b b: the conv of b takes the
 * conv of a, scaled and unshifted, as res).
 * In:  W [K3][Cin_full][Cout_full] (dt), the full tensor (not a copy of the
 *      slice; 16-byte aligned).  W may also point at input-channel row r0 of
 *      the full tensor (W_full + r0 * Cout_full; Cin_full still the full count,
 *      which sets the stride between offsets): the slice is then input channels
 *      r0 .. r0 + Cin - 1, and the caller guarantees r0 + Cin <= Cin_full;
 *      scale/shift: the full [Cout_full] f32 vectors or NULL (only the first
 *      Cout entries are read); res [m_out_cap][Cout] (dt, 16-byte aligned, not
 *      the output) or NULL; every other argument as in spv_sparse_conv (in
 *      [in_rows][Cin] and out [m_out_cap][Cout] are dense at the sliced widths).
 * Errors: as spv_sparse_conv, plus SPV_ERR_INVALID_ARG when Cin > Cin_full,
 *      Cout > Cout_full or res aliases out.  Cin_full = Cin, Cout_full = Cout
 *      and res = NULL is spv_sparse_conv.
 */
spv_status spv_sparse_conv_sliced(void* stream, void* ws, size_t ws_bytes,
                                  const void* in, int64_t in_rows, int32_t Cin,
                                  const int32_t* off, const int32_t* pairs, int64_t pair_cap,
                                  int32_t K3, int32_t transposed,
                                  const void* W, int32_t Cin_full, int32_t Cout_full,
                                  const float* scale, const float* shift, const void* res, int32_t relu,
                                  void* out, const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout,
                                  spv_dtype dt);

/*
 * A submanifold 3x3x3 map as a dense neighbour table, for a network that runs
 * several convolutions on one voxel set (Sec. 3.3's blocks, a U-Net stage):
 *
 * spv_kernel_map_nbr -- nbr[j][k] = i + 1 when voxel i sits at c_j + delta_k
 * (k = 9(dx+1) + 3(dy+1) + (dz+1)), 0 when no voxel does: the pairs of the
 * K=3 stride-1 spv_kernel_map, stored by output row.
 * In:  in_coords [m_cap][4] (distinct); m_in_dev: device count (NULL = m_cap).
 * Out: nbr [m_cap][27] int32 (rows < count written).  Device-detected errors
 *      (duplicate or out-of-range coordinates) go to the workspace status.
 *
 * spv_sparse_conv_nbr -- spv_sparse_conv_sliced on such a table: the
 * neighbour-table conv kernel without the per-call plan (no table build, only
 * the weight packing).  Only the shapes that kernel takes: bf16/f16 with Cin,
 * Cout in {32, 64, 96, 128, 256} (else SPV_ERR_UNSUPPORTED).
 * In:  nbr [m_out_cap][27] from spv_kernel_map_nbr on the output voxels (the
 *      inputs are the same voxels: in_rows = their count); every other
 *      argument as in spv_sparse_conv_sliced.
 */
spv_status spv_kernel_map_nbr(void* stream, void* ws, size_t ws_bytes,
                              const int32_t* in_coords, const int64_t* m_in_dev, int64_t m_cap, int32_t* nbr);
spv_status spv_sparse_conv_nbr(void* stream, void* ws, size_t ws_bytes,
                               const void* in, int64_t in_rows, int32_t Cin, const int32_t* nbr,
                               const void* W, int32_t Cin_full, int32_t Cout_full,
                               const float* scale, const float* shift, const void* res, int32_t relu,
                               void* out, const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout,
                               spv_dtype dt);

/*
 * spv_sparse_conv_nbr_noalloc -- spv_sparse_conv_nbr without a workspace, for
 * callers that cannot allocate device memory (code under graph capture, tight
 * serving loops, harnesses that forbid allocation).  It allocates nothing:
 * the packed weights go to a device-resident array of 3,538,944 bytes (the
 * packing of a 256 -> 256 layer) that the library holds on every device it
 * runs on until the process ends; its address is looked up once per device.
 * Arguments, outputs and the shapes taken are those of spv_sparse_conv_nbr;
 * packed weights larger than the array return SPV_ERR_CAPACITY, a current
 * device index of 64 or more SPV_ERR_UNSUPPORTED.  Every call on
 * one device uses the same array: calls that overlap in time on one device
 * (different streams without ordering between them) race and give undefined
 * results; calls in order on one stream are safe.
 */
spv_status spv_sparse_conv_nbr_noalloc(void* stream, const void* in, int64_t in_rows, int32_t Cin,
                                       const int32_t* nbr, const void* W, int32_t Cin_full, int32_t Cout_full,
                                       const float* scale, const float* shift, const void* res, int32_t relu,
                                       void* out, const int64_t* m_out_dev, int64_t m_out_cap, int32_t Cout,
                                       spv_dtype dt);

/*
 * The transposed k=2 s=2 conv (a decoder's upsampling) on the stride-2 map's
 * child table:
 *
 * spv_map_children -- children[j][k] = i + 1 for every pair (fine i, coarse j)
 * of offset k of a K=2 stride-2 map from spv_kernel_map, 0 where coarse voxel j
 * has no child at offset k.  Pairs past pair_cap or with rows outside
 * [0, fine_rows) / [0, coarse count) are ignored; a map with unsorted or
 * repeated pairs sets SPV_ERR_INVALID_ARG in the workspace status.
 * In:  off [9], pairs [pair_cap][2] (device); m_coarse_dev: device count of the
 *      coarse voxels (NULL = m_coarse_cap).
 * Out: children [m_coarse_cap][8] int32 (16-byte aligned).
 *
 * spv_sparse_conv_up -- for every coarse row j < count and offset k with
 * children[j][k] = i + 1 (i < out_rows):
 *   out[i] = act(scale * (in[j] @ W[k][:Cin][:Cout]) + shift + res[i])
 * which is spv_sparse_conv_sliced(transposed = 1) on that map whenever every
 * output row is some coarse voxel's child -- always the case for the fine
 * voxels a stride-2 spv_kernel_map was built on.  Output rows that are no
 * child are not written.  Each product row is stored once, straight from the
 * matrix-core accumulators (no gathers, no accumulation across pairs).
 * In:  in [m_in_cap][Cin] coarse rows (dt); children from spv_map_children;
 *      W [8][Cin_full][Cout_full] (dt) with the slicing of
 *      spv_sparse_conv_sliced; scale/shift f32 or NULL; res [out_rows][Cout]
 *      (dt) or NULL.  bf16/f16 with Cin, Cout in {32, 64, 96, 128, 256}, else
 *      SPV_ERR_UNSUPPORTED.
 * Out: out [out_rows][Cout] (dt).
 */
spv_status spv_map_children(void* stream, void* ws, size_t ws_bytes,
                            const int32_t* off, const int32_t* pairs, int64_t pair_cap, int64_t fine_rows,
                            const int64_t* m_coarse_dev, int64_t m_coarse_cap, int32_t* children);
spv_status spv_sparse_conv_up(void* stream, void* ws, size_t ws_bytes,
                              const void* in, const int64_t* m_in_dev, int64_t m_in_cap, int32_t Cin,
                              const int32_t* children, const void* W, int32_t Cin_full, int32_t Cout_full,
                              const float* scale, const float* shift, const void* res, int32_t relu,
                              void* out, int64_t out_rows, int32_t Cout, spv_dtype dt);

/*
 * spv_devoxelize_nbr -- spv_devoxelize (Sec. 3.3 "Sparse Devoxelization", with
 * the point MLP and the fusion add) on a grid that is the points' own
 * voxelization at voxel_size * 2^stride_log2: point k's voxel is pt2vox[k]
 * (from spv_voxelize or spv_voxelize_onto at that voxel size) and nbr is the
 * grid's neighbour table from spv_kernel_map_nbr.  Every corner of a point lies
 * within one voxel of its own, so the 8 corner indices are read from the
 * point's row of nbr: no hash table is built.  Results equal spv_devoxelize's
 * on the same grid.  A point with pt2vox outside [0, m_cap) has no corners
 * (its output is the MLP term alone).  Only the matrix-core kernel's shapes
 * (bf16/f16, C/16 in {1, 2, 4, 6, 8, 16}, Cp a multiple of 8 up to 128 or no
 * MLP), else SPV_ERR_UNSUPPORTED.  No corner outputs.
 * In:  grid_coords [m_cap][4], vfeat [m_cap][C], nbr [m_cap][27], pt2vox [n];
 *      the rest as in spv_devoxelize.
 */
spv_status spv_devoxelize_nbr(void* stream, void* ws, size_t ws_bytes,
                              const int32_t* grid_coords, const int64_t* m_dev, int64_t m_cap,
                              const int32_t* nbr, const int32_t* pt2vox, int32_t stride_log2,
                              const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                              spv_devox_mode mode, const void* vfeat, int32_t C,
                              const void* pfeat, int32_t Cp, const void* Wp,
                              const float* scale_p, const float* shift_p, int32_t relu_p,
                              void* out, spv_dtype dt);

/*
 * Pre-packed weights.  The neighbour-table conv, the upsampling conv and the
 * linear layer copy their weights into matrix-core fragments in every call; a
 * network whose weights stay fixed across forwards packs each once:
 *
 * spv_packed_weights_bytes -- bytes of the packed form of W[K3][Cin][Cout]
 * (K3 in 1..27), or 0 when no kernel reads that shape (ceil(Cin/32) must be 1,
 * 2, 3, 4, 6 or 8; ceil(Cout/16) at most 16).
 *
 * spv_pack_weights -- packs the slice W[:K3][:Cin][:Cout] of a 16-bit weight
 * tensor W[K3][Cin_full][Cout_full] (device) into `packed` (device, 16-byte
 * aligned, packed_bytes from spv_packed_weights_bytes).  A channel slice at an
 * input-channel offset is packed by passing W advanced by offset * Cout_full
 * elements.  Enqueued on `stream`, like the kernels that read it.
 * Errors: SPV_ERR_INVALID_ARG (null or misaligned pointers, a slice wider than
 * W), SPV_ERR_UNSUPPORTED (float32, or a shape of size 0 above),
 * SPV_ERR_CAPACITY (packed_bytes too small).
 *
 * spv_sparse_conv_nbr_packed, spv_sparse_conv_up_packed, spv_linear_packed --
 * spv_sparse_conv_nbr, spv_sparse_conv_up and spv_linear with weights packed by
 * spv_pack_weights for exactly (K3 = 27, 8 and 1 respectively, Cin, Cout) in
 * place of W, Cin_full and Cout_full; results are identical to the unpacked
 * calls'.  spv_linear_packed takes only the shapes of its matrix-core kernel
 * (bf16/f16, Cin a multiple of 8 with ceil(Cin/32) in {1, 2, 3, 4, 8}, Cout/16
 * rounded up in {1, 2, 4, 6, 8, 16}, Cout a multiple of 16 unless at most 32),
 * else SPV_ERR_UNSUPPORTED.  No weight packing is launched.
 */
size_t spv_packed_weights_bytes(int32_t K3, int32_t Cin, int32_t Cout);
spv_status spv_pack_weights(void* stream, const void* W, int32_t K3, int32_t Cin_full, int32_t Cout_full,
                            int32_t Cin, int32_t Cout, spv_dtype dt, void* packed, size_t packed_bytes);
spv_status spv_sparse_conv_nbr_packed(void* stream, void* ws, size_t ws_bytes,
                                      const void* in, int64_t in_rows, int32_t Cin, const int32_t* nbr,
                                      const void* Wpacked, const float* scale, const float* shift,
                                      const void* res, int32_t relu, void* out, const int64_t* m_out_dev,
                                      int64_t m_out_cap, int32_t Cout, spv_dtype dt);
spv_status spv_sparse_conv_up_packed(void* stream, void* ws, size_t ws_bytes,
                                     const void* in, const int64_t* m_in_dev, int64_t m_in_cap, int32_t Cin,
                                     const int32_t* children, const void* Wpacked,
                                     const float* scale, const float* shift, const void* res, int32_t relu,
                                     void* out, int64_t out_rows, int32_t Cout, spv_dtype dt);
spv_status spv_linear_packed(void* stream, void* ws, size_t ws_bytes,
                             const void* in, const int64_t* m_dev, int64_t m_cap, int32_t Cin,
                             const void* Wpacked, const float* scale, const float* shift, int32_t relu,
                             const void* res, int32_t res_after_act, void* out, int32_t Cout, spv_dtype dt);

/*
 * Backward passes (training, Sec. 4.2 trains the super network end to end).
 *
 * spv_sparse_conv_dgrad -- input gradient of spv_sparse_conv (without its
 * scale / shift / activation, whose backward is elementwise):
 *   dx[i] = sum over the pairs (i, j, k) of dy[j] @ W[k]^T
 * i.e. the conv over the same map with every pair's roles swapped and each W[k]
 * read transposed in place, on the same kernels.
 * In:  dy [dy_rows][Cout] (dt); off / pairs / pair_cap / K3 / transposed: the
 *      map and flag of the forward call; W [K3][Cin][Cout] (dt), the forward
 *      weights.
 * Out: dx [m_in_cap][Cin] (dt); rows < *m_in_dev (NULL = m_in_cap) are written.
 * Errors: as spv_sparse_conv.
 */
spv_status spv_sparse_conv_dgrad(void* stream, void* ws, size_t ws_bytes,
                                 const void* dy, int64_t dy_rows, int32_t Cout,
                                 const int32_t* off, const int32_t* pairs, int64_t pair_cap,
                                 int32_t K3, int32_t transposed, const void* W,
                                 void* dx, const int64_t* m_in_dev, int64_t m_in_cap, int32_t Cin,
                                 spv_dtype dt);

/*
 * spv_sparse_conv_dgrad_nbr -- spv_sparse_conv_dgrad for a submanifold 3x3x3
 * map given as its neighbour table (spv_kernel_map_nbr's [m][27], entry k of
 * row i = j + 1 for the voxel j at c_i + delta_k), with no per-call plan.  The
 * map of a set onto itself is symmetric: entry k of row i holds j exactly when
 * entry 26 - k of row j holds i, so
 *   dx[i] = sum over k of dy[nbr[i][k] - 1] @ W[26 - k]^T
 * is the neighbour-table conv with each W[26 - k] read transposed by the
 * weight packing.
 * In:  dy [m_cap][Cout] (dt); nbr [m_cap][27]; W [27][Cin][Cout] (dt), the
 *      forward weights; m_dev: device row count (NULL = m_cap).
 * Out: dx [m_cap][Cin] (dt); rows < *m_dev are written.
 * Errors: SPV_ERR_UNSUPPORTED for widths the neighbour-table kernel does not
 *      take (Cin, Cout in {32, 64, 96, 128, 256}, 16-bit), otherwise as
 *      spv_sparse_conv_nbr.
 */
spv_status spv_sparse_conv_dgrad_nbr(void* stream, void* ws, size_t ws_bytes,
                                     const void* dy, int32_t Cout, const int32_t* nbr, const void* W,
                                     void* dx, const int64_t* m_dev, int64_t m_cap, int32_t Cin,
                                     spv_dtype dt);

/*
 * spv_sparse_conv_wgrad -- weight gradient of spv_sparse_conv:
 *   dW[k] = sum over the pairs (i, j) of offset k of x[i]^T dy[j]
 * (roles of each pair swapped with transposed = 1); fp32 accumulation.  The
 * result is deterministic: fixed slices of every offset's pairs are summed
 * separately and the slices added in order.
 * In:  x [x_rows][Cin], dy [dy_rows][Cout] (dt, 16-byte aligned); the map of
 *      the forward call; pairs past pair_cap or with rows outside x / dy are
 *      ignored.
 * Out: dW [K3][Cin][Cout] float32.
 * bf16/f16 with Cin % 16 == 0, Cout % 16 == 0 and Cin + Cout <= 512 run on
 * MFMA; other shapes and f32 on a vector-ALU kernel.  Cin * Cout <= 65536.
 * The workspace holds the slices' partial sums:
 * spv_wgrad_workspace_bytes(K3, Cin, Cout) bytes (K3 * S * Cin * Cout * 4,
 * with S slices per offset: the largest power of two in [8, 64] for which
 * 27 * S * Cin * Cout * 4 <= 64 MiB, or 8).
 * Errors: SPV_ERR_INVALID_ARG, SPV_ERR_UNSUPPORTED (K3, Cin * Cout),
 *      SPV_ERR_CAPACITY (ws too small).
 */
size_t spv_wgrad_workspace_bytes(int32_t K3, int32_t Cin, int32_t Cout);
spv_status spv_sparse_conv_wgrad(void* stream, void* ws, size_t ws_bytes,
                                 const void* x, int64_t x_rows, int32_t Cin,
                                 const void* dy, int64_t dy_rows, int32_t Cout,
                                 const int32_t* off, const int32_t* pairs, int64_t pair_cap,
                                 int32_t K3, int32_t transposed, float* dW, spv_dtype dt);

/*
 * spv_voxelize_backward -- backward of the scatter-mean (Eq. 2):
 *   dfeat[k] = dvfeat[v] / N_v,  v = pt2vox[k]   (0 where v < 0 or v >= m)
 * fp64 quotient, one rounding to dt.  No workspace.
 * In:  dvfeat [m][C] (dt); counts [m] and pt2vox [n] from spv_voxelize.
 * Out: dfeat [n][C] (dt).
 */
spv_status spv_voxelize_backward(void* stream, const void* dvfeat, int64_t m, int32_t C,
                                 const int32_t* counts, const int32_t* pt2vox, int64_t n,
                                 void* dfeat, spv_dtype dt);

/*
 * spv_epilogue_backward -- backward of the epilogue the convolutions, the
 * linear layers and spv_block apply to their raw product a (Sec. 3.3: BN folded
 * into a per-channel scale and shift, ReLU, and the residual of a ResNet block
 * before the activation or the fusion by addition after it):
 *   forward  y = act(scale * a + shift + res)   (res_after_act = 0)
 *            y = act(scale * a + shift) + res   (res_after_act = 1)
 *   z = fmaf(a, scale, shift) (+ res when res_after_act = 0), in float32;
 *   gz = dy where relu = 0 or z > 0, else 0;
 *   da = gz * scale (one rounding to dt), dres = dy (res_after_act = 1) or gz;
 *   dscale[c] = sum_i gz * a, dshift[c] = sum_i gz (fp64 in a fixed order, one
 *   rounding: the same bits on every call).
 * a is the op's output with scale = shift = res = NULL and relu = 0 (the same
 * call without its epilogue).
 * In:  dy, a, res [m][C] (dt; res may be NULL); scale, shift [C] f32 or NULL
 *      (1, 0).
 * Out: da, dres [m][C] (dt), dscale, dshift [C] f32; any may be NULL.
 *      ws: spv_epilogue_backward_workspace_bytes(m, C) bytes, 256-byte aligned,
 *      needed only with dscale or dshift.
 * Errors: SPV_ERR_INVALID_ARG, SPV_ERR_CAPACITY.
 */
size_t spv_epilogue_backward_workspace_bytes(int64_t m, int32_t C);
spv_status spv_epilogue_backward(void* stream, void* ws, size_t ws_bytes,
                                 const void* dy, const void* a, const float* scale, const float* shift,
                                 int32_t relu, const void* res, int32_t res_after_act, int64_t m, int32_t C,
                                 void* da, void* dres, float* dscale, float* dshift, spv_dtype dt);

/*
 * spv_linear_backward -- gradients of the linear layer's product out = in @ W
 * (the point branch's MLP of Sec. 3.3, a 1x1 shortcut):
 *   din = da @ W^T  (fp32 accumulation, one rounding to dt)
 *   dW  = in^T @ da (float32; deterministic: fixed partial sums in a fixed order)
 * da is the gradient of the product (spv_epilogue_backward's da).
 * In:  in [m][Cin], W [Cin][Cout], da [m][Cout] (dt); in, da, din 16-byte aligned.
 * Out: din [m][Cin] (dt) and / or dW [Cin][Cout] f32 (either may be NULL).
 *      ws: spv_linear_backward_workspace_bytes(Cin, Cout) bytes, 256-byte aligned.
 * Errors: SPV_ERR_INVALID_ARG, SPV_ERR_CAPACITY, SPV_ERR_UNSUPPORTED (dW with
 *      Cin * Cout > 65536).
 */
size_t spv_linear_backward_workspace_bytes(int32_t Cin, int32_t Cout);
spv_status spv_linear_backward(void* stream, void* ws, size_t ws_bytes,
                               const void* in, int64_t m, int32_t Cin, const void* W, int32_t Cout,
                               const void* da, void* din, float* dW, spv_dtype dt);

/*
 * spv_devoxelize_backward -- backward of the trilinear devoxelization w.r.t.
 * the voxel features (Sec. 3.3 "Sparse Devoxelization"):
 *   dvfeat[v] = sum over the points k and corners c with corner_idx[k][c] = v
 *               of a_kc * dout[k],   a_kc = w_kc / (sum of k's present w)
 * (w = the raw trilinear weights; a corner is present when 0 <= index < m; a
 * point whose present weights sum to <= 0 adds nothing).  Deterministic: each
 * voxel sums its terms in ascending (k, c) order with fp32 fmas, so repeated
 * calls give the same bits; every row v < m is written (0 without terms).
 * In:  ws: spv_devoxelize_backward_workspace_bytes(n, m) bytes, 256-byte
 *      aligned; corner_idx [n][8] i32, corner_w [n][8] f32 as spv_devoxelize
 *      reports them; dout [n][C] (dt).
 * Out: dvfeat [m][C] float32.
 * Errors: SPV_ERR_INVALID_ARG (null pointers, negative sizes, n >= 2^28,
 *      m >= 2^31 - 1, dvfeat = dout), SPV_ERR_CAPACITY (ws too small); a corner index >= m is
 *      skipped and reported as SPV_ERR_RANGE through spv_status_check(ws).
 */
size_t spv_devoxelize_backward_workspace_bytes(int64_t n, int64_t m);
spv_status spv_devoxelize_backward(void* stream, void* ws, size_t ws_bytes,
                                   const int32_t* corner_idx, const float* corner_w,
                                   const void* dout, int64_t n, int32_t C, float* dvfeat, int64_t m,
                                   spv_dtype dt);

/*
 * spv_linear -- a pointwise linear layer on feature rows:
 *   res_after_act = 0:  out[i] = act(scale * (in[i] @ W) + shift + res[i])
 *   res_after_act = 1:  out[i] = act(scale * (in[i] @ W) + shift) + res[i]
 * The point branch's MLP with the fusion by addition (Sec. 3.3 "Point
 * Transformation and Feature Fusion": res = the devoxelized voxel features, added
 * after the activation); the 1x1 shortcut of a residual block; a classifier
 * (scale NULL, shift = bias, no activation).  fp32 accumulation, one rounding.
 * In:  in [m_cap][Cin] (dt, 16-byte aligned); m_dev: device row count (NULL =
 *      m_cap); W [Cin_full][Cout_full] (dt) of which the leading Cin x Cout block
 *      is used (channel slicing as in spv_sparse_conv_sliced; W may point at a
 *      later row of a wider tensor); scale/shift f32 [>= Cout] or NULL;
 *      res [m_cap][Cout] (dt, 16-byte aligned, not the output) or NULL.
 * Out: out [m_cap][Cout] (dt, 16-byte aligned, not the input); rows < *m_dev.
 * bf16/f16 with Cin % 8 == 0, ceil(Cin / 32) in {1, 2, 3, 4, 8} and Cout in
 * {16, 32, 64, 96, 128, 256} run on MFMA; other shapes and f32 on a vector-ALU
 * kernel.  The workspace from spv_workspace_bytes(., max(Cin, Cout)) suffices.
 * Errors: SPV_ERR_INVALID_ARG (sizes, Cin > Cin_full, Cout > Cout_full, null or
 *      misaligned pointers, aliasing), SPV_ERR_CAPACITY (ws too small).
 */
spv_status spv_linear(void* stream, void* ws, size_t ws_bytes,
                      const void* in, const int64_t* m_dev, int64_t m_cap, int32_t Cin,
                      const void* W, int32_t Cin_full, int32_t Cout_full,
                      const float* scale, const float* shift, int32_t relu,
                      const void* res, int32_t res_after_act,
                      void* out, int32_t Cout, spv_dtype dt);

/*
 * spv_devoxelize -- sparse devoxelization (Sec. 3.3 "Sparse Devoxelization":
 * trilinear interpolation from the 8 neighbouring voxels) fused with the
 * point-branch MLP and the fusion by addition ("Point Transformation and
 * Feature Fusion"):
 *   out_k = sum_c w_c V[idx_c] / sum_c w_c  +  act(scale_p * (pfeat_k @ Wp) + shift_p)
 * where the grid has voxel size v * 2^stride_log2 (coordinates in its units),
 * a = fl32(x / v) * 2^-stride_log2, u = a - 1/2 (CENTER) or a (CORNER),
 * base = floor(u), t = u - base, corner c = (cx, cy, cz) has index
 * 4 cx + 2 cy + cz and raw weight prod(c ? t : 1 - t) (fp32, x*y*z order);
 * absent corners get weight 0 and the rest are renormalized; a point with no
 * present corner gets 0 from the voxel branch.
 * In:  grid_coords [m_cap][4] (distinct), m_dev (NULL = m_cap); vfeat [*][C];
 *      pfeat [n][Cp] and Wp [Cp][C] (both NULL = no point branch).
 * Out: out [n][C] (dt); corner_idx [n][8] i32 and corner_w [n][8] f32 optional.
 */
spv_status spv_devoxelize(void* stream, void* ws, size_t ws_bytes,
                          const int32_t* grid_coords, const int64_t* m_dev, int64_t m_cap,
                          int32_t stride_log2,
                          const float* xyz, const int32_t* batch, int64_t n, float voxel_size,
                          spv_devox_mode mode,
                          const void* vfeat, int32_t C,
                          const void* pfeat, int32_t Cp, const void* Wp,
                          const float* scale_p, const float* shift_p, int32_t relu_p,
                          void* out, spv_dtype dt, int32_t* corner_idx, float* corner_w);

/* Parameters of the SPVConv block (Fig. 2): voxel branch = voxelize, n_convs
 * submanifold 3x3x3 convs C->C, each act(scale * conv + shift); point branch =
 * act(scale_p * (f @ Wp) + shift_p); fused by addition after devoxelization. */
typedef struct spv_block_params {
    int32_t C;
    spv_dtype dtype;
    float voxel_size;
    int32_t n_convs;        /* 1 or 2 */
    const void* W[2];       /* [27][C][C] (dt), device */
    const float* scale[2];  /* [C] f32 or NULL */
    const float* shift[2];  /* [C] f32 or NULL */
    int32_t relu[2];
    const void* Wp;         /* [C][C] (dt), device */
    const float* scale_p;   /* [C] f32 or NULL */
    const float* shift_p;   /* [C] f32 or NULL */
    int32_t relu_p;
    spv_devox_mode devox_mode;
    /* Residual block (Sec. 3.3: the voxel branch aggregates with residual
     * sparse-convolution blocks): nonzero makes the last conv add the block's
     * voxel input x (the voxelized point features) to its output after scale
     * and shift and before its ReLU: y = act(scale * conv(.) + shift + x). */
    int32_t residual;
    /* Optional profiling (NULL = off): n_events >= 7 hipEvent_t handles, created
     * by the caller, recorded on the stream at the phase boundaries:
     * [0] start, [1] voxelized, [2] kernel map built, [3] conv plan built and
     * weights packed, [4] conv 1 done, [5] conv 2 done (same point as [4] when
     * n_convs == 1), [6] devoxelized (end). */
    void* const* events;
    int32_t n_events;
} spv_block_params;

size_t spv_block_workspace_bytes(int64_t max_points, int32_t C);

/*
 * spv_block -- one SPVConv block (Sec. 3.3, Fig. 2): the hash table built by the
 * voxelization is reused by the kernel map and the devoxelization; the kernel
 * map is built once and shared by the convs.  out [n][C] (dt).  m_host optional
 * (synchronizes; returns device-detected errors).
 */
spv_status spv_block(void* stream, void* ws, size_t ws_bytes, const spv_block_params* p,
                     const float* xyz, const int32_t* batch, int64_t n, const void* feat,
                     void* out, int64_t* m_host);

/* Hash-table lookups (test hook for the voxel hash of Sec. 3.3): builds the
 * table of table_coords and writes idx[q] = index of qcoords[q] in it, or -1. */
spv_status spv_lookup(void* stream, void* ws, size_t ws_bytes,
                      const int32_t* table_coords, const int64_t* m_dev, int64_t m_cap,
                      const int32_t* qcoords, int64_t q, int32_t* idx);

/*
 * spv_voxel_lookup -- queries the hash table the last spv_voxelize call on ws
 * built (Sec. 3.3: one O(1) lookup per coordinate), without rebuilding it.
 * In:  ws / ws_bytes / n: the workspace and point count of that spv_voxelize
 *      call (the table's place in the workspace follows from n); qcoords
 *      [q][4] int32 (b, x, y, z), any values.
 * Out: idx [q] int32: the voxel's canonical index (its row in spv_voxelize's
 *      coords), -1 if the voxel is not in the table.
 * Errors: SPV_ERR_INVALID_ARG (null or misaligned ws, negative sizes),
 *      SPV_ERR_CAPACITY (ws_bytes below what n needs).  Reads ws only.
 */
spv_status spv_voxel_lookup(void* stream, const void* ws, size_t ws_bytes, int64_t n,
                            const int32_t* qcoords, int64_t q, int32_t* idx);

/*
 * spv_conv_kernel -- the kernel spv_sparse_conv (and its sliced / dgrad forms)
 * runs on for a shape and its sizes, as the call decides it on the host:
 * 0 = the neighbour-table MFMA kernel (3x3x3 maps), 1 = the tile MFMA kernel,
 * 2 = the vector-ALU kernel; -1 for arguments the calls reject.  The
 * neighbour-table kernel addresses the input rows and its table with 32-bit
 * offsets: in_rows * Cin * 2 and m_out_cap * 27 * 4 must stay below
 * 0xFFFFE000, else a larger shape falls back to the next kernel.  Host only.
 * spv_block_conv_kernel gives the same for the convs of spv_block(n, C, dt).
 */
int32_t spv_conv_kernel(int32_t K3, int32_t Cin, int32_t Cout, spv_dtype dt, int64_t in_rows, int64_t m_out_cap,
                        int64_t pair_cap, int32_t transposed);
int32_t spv_block_conv_kernel(int64_t n, int32_t C, spv_dtype dt);

/* Synchronizes the stream and returns the first device-detected error recorded
 * in the workspace status word (NONFINITE before RANGE before CAPACITY). */
spv_status spv_status_check(const void* ws, void* stream);

const char* spv_status_string(spv_status s);
int spv_last_hip_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPV_H */
