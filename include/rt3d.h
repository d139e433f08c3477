/*
 * rt3d.h -- C ABI of the MI355X (gfx950) library for forward 3-D convolution
 * under kernel-group-structured (KGS) sparsity, its vanilla special case, and
 * the dense baseline.  Paper: RT3D, arXiv 2007.09835.
 *
 * The operation (Section 3).  A 3-D CONV layer has a 5-D weight tensor
 * W[M][N][K_d][K_h][K_w] (M filters, N input channels; K_d is the temporal
 * kernel depth, called kt here).  The filters and channels are split into
 * kernel groups of g_M x g_N kernels, P = ceil(M/g_M) by Q = ceil(N/g_N)
 * groups (Section 4; the last group in each direction may be partial).  A
 * KGS mask keeps or prunes each kernel position of a group for all of the
 * group's kernels together (Fig. 1(b)); vanilla sparsity keeps or prunes a
 * group as a whole.  The pruned layer equals the dense layer with the pruned
 * weights set to zero, and since each group reshaped to a g_M x (g_N*K_s)
 * matrix merely loses columns, the kept part is a smaller dense matrix that
 * can be packed and multiplied on its own (Section 3, reshaping paragraph).
 *
 * Conventions used by every call:
 *   - Weights on the host are dense [M][N][kt][kh][kw] in the layer dtype.
 *   - Masks are uint8 [P][Q][kt*kh*kw]; 1 = keep, 0 = pruned, anything else
 *     is an error.  Kernel position pos = (it*kh + ih)*kw + iw.
 *   - Activations on the device are channels-last: x [n][t][h][w][c_in],
 *     y and residual [n][to][ho][wo][c_out] (torch.channels_last_3d).
 *   - The convolution is a cross-correlation with zero padding:
 *       y = act(sum_{c, kept pos} W[m][c][pos] * x[..shifted..] + bias[m]
 *               (+ residual))
 *     with act = ReLU when RT3D_RELU is set; to = (t + 2 pt - kt)/st + 1,
 *     likewise ho and wo.
 *   - Accumulation is float32 for every dtype; bias is float32; x, W, y and
 *     residual share the layer dtype; the output is rounded to nearest even.
 *   - Device calls are asynchronous on the caller's HIP stream (passed as
 *     void*, i.e. a hipStream_t; NULL is the default stream).  Faults inside
 *     a kernel surface at the next synchronisation of that stream.
 *   - Ownership: the caller owns every buffer.  The library never allocates
 *     caller-visible memory, never frees or retains a pointer past a call,
 *     and keeps no state except a thread-local error message, a per-device
 *     cache of runtime queries (compute-unit count, kernel occupancy) and the
 *     split-K scratch array of rt3d_kgs_conv3d_fwd_noalloc (one per device).
 *   - Tuning switch (benchmarks only; leave unset): the environment variable
 *     RT3D_TUNE="key=value,..." overrides planner choices.  Pack-time keys
 *     change the kernel layout written into a blob: slots=64|128 (voxel slots
 *     per workgroup), kgs_mfw=1|2|4 and dense_mfw=1|2|4 (16-filter MFMA rows
 *     per wave tile), small_mfw=1|2 and small_kernel=0 (the small-input-channel
 *     kernel), kgs_map=0|1|2 (16-bit KGS mapping: 0 = union of the tile's
 *     kept items, 1 = disjoint item pairs on the 2:4 sparse MFMA, 2 = pairs
 *     of adjacent channel blocks on the 2:4 sparse MFMA), pair_mfw=1|2|4
 *     (16-filter rows per pair-mapping tile), cc=N (at most N input channels
 *     per staged chunk, 16-bit), kgs_f32=0|1 (fp32 KGS: exact 4x4 blocks or
 *     the union of a 16-filter tile's items), kgs_order=0|1 (16-bit union
 *     with 4x4 groups: 4-filter blocks that keep similar items share a tile
 *     when that saves at least 5% of the K-steps by default; 1 = whenever it
 *     saves any, 0 = never).  Launch-time
 *     keys change the launch of a forward call: splits=N (input-channel
 *     splits) and wg_order=0|1 (workgroup order).  Results stay within the
 *     documented accuracy under every setting.
 *   - Errors: all arguments are validated before anything is launched; on
 *     error nothing is written to the outputs and rt3d_last_error_detail()
 *     describes the failure.
 */
#ifndef RT3D_H
#define RT3D_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RT3D_OK = 0,
    RT3D_ERR_INVALID_ARG = 1,      /* null pointer, non-positive size, bad mask byte */
    RT3D_ERR_UNSUPPORTED = 2,      /* valid but outside what the kernels implement */
    RT3D_ERR_BUFFER_TOO_SMALL = 3, /* a caller buffer is smaller than required */
    RT3D_ERR_BLOB_MISMATCH = 4,    /* packed blob/info does not belong to this desc */
    RT3D_ERR_HIP = 5               /* the HIP runtime reported an error */
} rt3d_status;

typedef enum { RT3D_F32 = 0, RT3D_BF16 = 1, RT3D_F16 = 2 } rt3d_dtype;

enum { RT3D_RELU = 1u, RT3D_RESIDUAL = 2u };

/* One convolution layer applied to one batch.  Supported: strides 1 or 2,
 * kernel extents 1..7, padding 0..kernel extent-1, group sizes g_m, g_n in
 * {4, 8, 16} (the paper uses g_N = 4 and g_M = 4 or 8, Section 3). */
typedef struct {
    int32_t n, c_in, c_out;   /* batch, N input channels, M filters */
    int32_t t, h, w;          /* input extent */
    int32_t kt, kh, kw;       /* kernel extent; kt is the temporal depth K_d */
    int32_t st, sh, sw;       /* stride */
    int32_t pt, ph, pw;       /* zero padding */
    int32_t g_m, g_n;         /* kernel-group size (KGS calls; ignored when dense) */
    int32_t dtype;            /* rt3d_dtype of x, W, y, residual */
    uint32_t flags;           /* RT3D_RELU | RT3D_RESIDUAL */
    int32_t qt, qh, qw;       /* fused max-pool window (= stride) applied after the
                                 activation, 0 or 1 = none; C3D pools 1x2x2 after conv1
                                 and 2x2x2 after conv2/3b/4b.  y then has the pooled
                                 extent floor(to/qt) x floor(ho/qh) x floor(wo/qw);
                                 the residual keeps the unpooled extent. */
    int32_t y_c_total, y_c_off; /* fused channel concatenation: y holds y_c_total
                                 channels per voxel and this layer writes channels
                                 [y_c_off, y_c_off + c_out) of it (the branches of an
                                 Inception block writing one output).  0, 0 = y has
                                 exactly c_out channels.  Otherwise y_c_off >= 0,
                                 y_c_off + c_out <= y_c_total, and both y_c_total and
                                 y_c_off are multiples of 4.  The residual always has
                                 c_out channels per voxel. */
    int32_t x_c_total, x_c_off; /* channel slice of the input: x holds x_c_total
                                 channels per voxel and the layer reads channels
                                 [x_c_off, x_c_off + c_in) (a layer consuming part of a
                                 wider tensor).  0, 0 = x has exactly c_in channels.
                                 Layers with c_in <= 4 (network inputs) need 0, 0. */
} rt3d_conv3d_desc;

/* Filled by the pack calls; plain data owned by the caller.  It describes
 * the blob and must be passed back unchanged to the forward call. */
typedef struct {
    uint64_t magic;            /* identifies a blob written by this library */
    uint64_t desc_hash;        /* hash of the weight-side desc fields */
    uint32_t version;
    uint32_t variant;          /* kernel mapping chosen at pack time */
    uint32_t tile_groups;      /* filter groups per wave tile (KGS) */
    uint32_t vanilla;          /* 1 if every mask row is all-0 or all-1 */
    uint64_t packed_bytes;     /* size of the blob */
    /* canonical sections of a KGS blob (byte offset and size within it):
     * [0] group_ptr u32[P*Q+1]  prefix sums of kept positions per group,
     *                           groups p-major, q-minor
     * [1] pos       u16[sum k]  ascending kept positions of each group
     * [2] val_ptr   u64[P*Q+1]  prefix sums of kept weights per group
     * [3] vals      dtype[...]  per group g (gm x gn kernels, k positions):
     *                           vals[val_ptr[g] + (i*gn + j)*k + r] =
     *                           W[p*g_m+i][q*g_n+j][pos_r]
     * A dense blob has no canonical sections (all zero). */
    uint64_t canon_off[4];
    uint64_t canon_bytes[4];
    uint64_t derived_off;      /* kernel-layout section */
    uint64_t derived_bytes;
    uint64_t kept_positions;   /* sum over groups of k */
    uint64_t kept_weights;     /* sum over groups of gm*gn*k: MACs per output voxel */
    uint64_t plan[16];         /* private to the library: the launch plan chosen at
                                  pack time; the forward call reads it, so the caller
                                  never has to read the device copy of the blob */
} rt3d_pack_info;

/* Static description of a status code (never NULL). */
const char *rt3d_status_string(rt3d_status status);

/* Message describing the last error raised on the calling thread ("" if
 * none).  Valid until the next library call on this thread. */
const char *rt3d_last_error_detail(void);

/* Output extent of a layer (after the fused pooling, if any).  Host only. */
rt3d_status rt3d_conv3d_out_shape(const rt3d_conv3d_desc *desc,
                                  int32_t *to, int32_t *ho, int32_t *wo);

/* Bytes of the KGS blob for this layer and mask (Section 3 compact format
 * plus the kernel layout).  Host only, deterministic.
 *
 * A blob (KGS or dense) is tied to every desc field except n and flags: the
 * kernel layout is planned for the layer's input extent, strides and
 * padding, so one blob serves any batch size and any epilogue flags, and a
 * forward call with other extents fails with RT3D_ERR_BLOB_MISMATCH.  The
 * layout's tile shapes are chosen for desc->n at pack time (the voxel brick
 * and the filter-tile width depend on how much parallelism the batch gives);
 * a blob packed for one batch size runs correctly at any other.  Device
 * pointers (x, y, residual, bias, blob, workspace) must be 16-byte aligned. */
rt3d_status rt3d_kgs_pack_size(const rt3d_conv3d_desc *desc, const uint8_t *mask,
                               uint64_t *bytes);

/* Pack dense host weights w_dense [M][N][kt][kh][kw] (layer dtype) and the
 * host mask into the host buffer blob (blob_bytes >= rt3d_kgs_pack_size).
 * Writes the canonical per-group sections (Section 3: each group keeps its
 * g_M x (g_N * k) matrix of surviving columns, positions ascending, groups
 * p-major) and the kernel layout, and fills *info.  Weights at pruned
 * positions are never read.  A mask whose rows are all-0 or all-1 is the
 * vanilla scheme (Section 3) and is recorded as such.  The caller copies the
 * blob to device memory before calling rt3d_kgs_conv3d_fwd.  Host only. */
rt3d_status rt3d_kgs_pack(const rt3d_conv3d_desc *desc, const void *w_dense,
                          const uint8_t *mask, void *blob, uint64_t blob_bytes,
                          rt3d_pack_info *info);

/* Inverse of the canonical sections: writes W * expand(mask) as dense host
 * weights [M][N][kt][kh][kw] (pruned positions are zero).  Host only. */
rt3d_status rt3d_kgs_unpack(const rt3d_conv3d_desc *desc, const rt3d_pack_info *info,
                            const void *blob, void *w_masked_dense);

/* Device workspace with which a forward call of this layer (at desc->n) runs
 * at full parallelism (0 if it needs none).  Layers whose output alone cannot
 * fill the GPU split their input channels across workgroups; the float32
 * partial sums go to this caller-owned device buffer (16-byte aligned) and a
 * second kernel adds them in a fixed order, so results stay bit-reproducible.
 * A forward call given less workspace (or none) uses fewer splits; it never
 * fails for lack of workspace. */
rt3d_status rt3d_conv3d_workspace_size(const rt3d_conv3d_desc *desc,
                                       const rt3d_pack_info *info, uint64_t *bytes);

/* KGS (and vanilla) sparse forward.  blob_dev: device copy of the blob that
 * rt3d_kgs_pack wrote with this desc (info from that call).  With n == 0
 * nothing is read or written and the device pointers may be NULL.  x, y, residual
 * are device pointers in the channels-last layout; bias is a device float32
 * [M] array or NULL (zero bias); residual must be non-NULL exactly when
 * RT3D_RESIDUAL is set.  y must not overlap x, residual or the blob.  Work
 * skipped: a (4-channel block, kernel position) item that no kernel group
 * of a wave's filter tile keeps is never read or multiplied (so a vanilla-
 * pruned group costs nothing when its tile-mates prune the same channels).
 * How a kept item is multiplied depends on the mapping chosen at pack time:
 * the exact fp32 kernel issues one 4x4 MFMA per kept (group, item); the
 * union mappings (16-bit, and fp32 for layers too small to be bound by
 * their MFMA work) multiply the tile's other groups at that item by zero
 * weights (the 16-bit union may place 4-filter blocks that keep similar
 * items in the same tile; outputs land in layer order either way); the
 * 16-bit pair mapping packs two items whose kept groups
 * are disjoint into one 2:4 sparse MFMA slot and streams kept weights only.
 * Asynchronous on `stream`.  Per-call limits (RT3D_ERR_UNSUPPORTED,
 * checked before any launch; the same for rt3d_conv3d_dense_fwd): fewer
 * than 2^24 output voxels and 2^24 workgroups, and for layers packed onto
 * the small-input-channel kernel (c_in <= 4) an input x of fewer than
 * 2^31 - 8 bytes. */
rt3d_status rt3d_kgs_conv3d_fwd(const rt3d_conv3d_desc *desc, const rt3d_pack_info *info,
                                const void *blob_dev, const void *x, const float *bias,
                                const void *residual, void *y,
                                void *workspace, uint64_t workspace_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the KGS
 * forward of rt3d_kgs_conv3d_fwd without a caller workspace.  Its split-K
 * partial sums go to the library's own device array of RT3D_NOALLOC_SCRATCH
 * bytes (32 MiB, held by every GPU the library runs on until the process
 * ends); the call allocates nothing.  The launch is the one
 * rt3d_kgs_conv3d_fwd makes with a workspace of at least
 * rt3d_conv3d_workspace_size bytes, so the results are identical.  A layer
 * whose split-K workspace at desc->n exceeds RT3D_NOALLOC_SCRATCH bytes is
 * rejected with RT3D_ERR_UNSUPPORTED before anything is launched (call
 * rt3d_kgs_conv3d_fwd with a workspace instead).  Every call on a GPU shares
 * that GPU's array: calls that overlap in time on one GPU (other streams,
 * other threads) race and must not be made; consecutive calls on one stream
 * are safe (each writes every partial sum it reads, so nothing needs to
 * start at zero).  Other arguments and errors as rt3d_kgs_conv3d_fwd. */
#define RT3D_NOALLOC_SCRATCH (32u << 20)
rt3d_status rt3d_kgs_conv3d_fwd_noalloc(const rt3d_conv3d_desc *desc, const rt3d_pack_info *info,
                                        const void *blob_dev, const void *x, const float *bias,
                                        const void *residual, void *y, void *stream);

/* Bytes of the dense blob.  Host only. */
rt3d_status rt3d_dense_pack_size(const rt3d_conv3d_desc *desc, uint64_t *bytes);

/* Reorganise dense host weights [M][N][kt][kh][kw] into the dense kernel's
 * layout (host blob) and fill *info.  Host only. */
rt3d_status rt3d_dense_pack(const rt3d_conv3d_desc *desc, const void *w_dense,
                            void *blob, uint64_t blob_bytes, rt3d_pack_info *info);

/* Dense forward (the baseline every speedup is measured against), same
 * argument conventions as rt3d_kgs_conv3d_fwd. */
rt3d_status rt3d_conv3d_dense_fwd(const rt3d_conv3d_desc *desc, const rt3d_pack_info *info,
                                  const void *blob_dev, const void *x, const float *bias,
                                  const void *residual, void *y,
                                  void *workspace, uint64_t workspace_bytes, void *stream);

/* 3-D max pooling between layers (C3D pools 1x2x2 after conv1 and 2x2x2
 * after conv2, conv3b, conv4b; the S3D-shaped stack pools 1x3x3 and 3x3x3
 * windows with padding): channels-last x [n][t][h][w][c] -> y
 * [n][to][ho][wo][c], to = (t + 2 pt - kt) / st + 1 (floor), likewise ho, wo.
 * Padded positions take no part in the max; padding is at most half the
 * window (so every window holds input voxels).  Asynchronous on `stream`. */
rt3d_status rt3d_maxpool3d_fwd(int32_t n, int32_t c, int32_t t, int32_t h, int32_t w,
                               int32_t kt, int32_t kh, int32_t kw,
                               int32_t st, int32_t sh, int32_t sw,
                               int32_t pt, int32_t ph, int32_t pw, int32_t dtype,
                               const void *x, void *y, void *stream);

/* ------------------------------------------------------------------------
 * Reweighted group-lasso penalty (Section 4)
 *
 * The pruning algorithms of Section 4 penalise the norm of kernel groups: the
 * regularization-based algorithm adds lambda * sum ||W^G||_g to the training
 * loss (eq. (1); per kernel position, eq. (2)), and the reweighted algorithm
 * (eq. (3)) multiplies each norm
 * by a penalty factor P that is reset after every iteration to
 * 1 / (||W^G||_g^2 + eps), so that large groups are penalised less and small
 * ones more; after a few iterations the groups whose norm has converged to
 * zero are pruned.  For KGS sparsity a norm covers the g_M x g_N weights of
 * one kernel group at one kernel position (Fig. 2 caption); for vanilla
 * sparsity it covers the whole group.  These norms are called units below:
 *   scope RT3D_SCOPE_KGS:     P * Q * K_s units, unit (p, q, pos) at index
 *                             (p*Q + q)*K_s + pos;
 *   scope RT3D_SCOPE_VANILLA: P * Q units, unit (p, q) at index p*Q + q.
 * norm = 1 or 2 selects the l1 or l2 norm of the unit's weights (the paper
 * allows either).
 * ------------------------------------------------------------------------ */

enum { RT3D_SCOPE_KGS = 0, RT3D_SCOPE_VANILLA = 1 };

typedef struct {
    int32_t c_out, c_in;      /* M filters, N input channels */
    int32_t kt, kh, kw;       /* kernel extent, 1..7 each; K_s = kt*kh*kw */
    int32_t g_m, g_n;         /* kernel-group size, 1..16 each (partial trailing groups) */
    int32_t dtype;            /* rt3d_dtype of the weights and of w_prox */
    int32_t norm;             /* 1 or 2 */
    int32_t scope;            /* RT3D_SCOPE_KGS or RT3D_SCOPE_VANILLA */
} rt3d_group_desc;

/* Number of units (norms) of a layer for this desc.  Host only. */
rt3d_status rt3d_group_units(const rt3d_group_desc *desc, int64_t *units);

/* Device workspace (bytes, caller-owned, 4-byte aligned) that
 * rt3d_group_reweight needs when it is asked for the penalty value reg: one
 * float per workgroup, added up in index order by a second kernel.  No
 * initial contents are needed.  Calls that share a workspace must not run
 * concurrently.  Host only. */
rt3d_status rt3d_group_workspace_size(const rt3d_group_desc *desc, uint64_t *bytes);

/* One pass over device weights w [M][N][kt][kh][kw] (desc->dtype) computing,
 * for every unit u with current penalty factor P_u (pen[u]; pen == NULL means
 * all ones) and norm n_u:
 *   norms[u]    = n_u                                     (float32 [units])
 *   pen_next[u] = 1 / (n_u^2 + eps)   (the reweighting update; float32 [units])
 *   *reg        = lambda * sum_u P_u * n_u   (the penalty term of eq. (3);
 *                                             one float32 in device memory)
 *   mask        = 1 where n_u > tau, else 0, for every kernel position the
 *                 unit covers: uint8 [P][Q][K_s], the layout rt3d_kgs_pack
 *                 takes (pruning what has converged to zero: tau = 0 prunes
 *                 exactly the zero units)
 *   grad       += lambda * P_u * d n_u / d w  (float32 [M][N][K_s], accumulated:
 *                 the penalty's share of the weight gradient; l2: w / n_u, and
 *                 0 for a zero unit; l1: sign(w), 0 at w = 0)
 *   w_prox      = the minimiser z of 1/2 |z - w|^2 + step * lambda * sum_u
 *                 P_u * n_u(z), in desc->dtype (rounded to nearest even):
 *                 l2: w * max(0, 1 - theta / n_u); l1: sign(w) * max(0, |w| -
 *                 theta) (the l1 norm of a unit is a sum over its weights);
 *                 theta = step * lambda * P_u.  A proximal step on the penalty.
 * Every output pointer may be NULL (not computed).  Norms and sums are
 * float32 with a fixed summation order, so repeated calls give identical
 * results.  pen_next may be the same array as pen, and w_prox the same array
 * as w (in-place updates); no other outputs may overlap each other or the
 * inputs.  eps must be > 0; lambda, step >= 0; all scalars finite.  A unit's
 * weights (g_m * g_n * K_s values) must fit the kernel's staging buffer:
 * g_m * g_n * K_s <= 12288, else RT3D_ERR_UNSUPPORTED.  reg needs workspace
 * of rt3d_group_workspace_size bytes (RT3D_ERR_BUFFER_TOO_SMALL otherwise).
 * Asynchronous on `stream`. */
rt3d_status rt3d_group_reweight(const rt3d_group_desc *desc, const void *w, const float *pen,
                                float lambda, float eps, float tau, float step,
                                float *norms, float *pen_next, float *reg, uint8_t *mask,
                                float *grad, void *w_prox,
                                void *workspace, uint64_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* RT3D_H */
