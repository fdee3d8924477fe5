/*
 * octree_nca.h -- C ABI of the MI355X (gfx950) OctreeNCA inference library.
 *
 * OctreeNCA (arXiv 2508.06993) segments an image (2D) or a volume / video
 * (3D, 2D+t) by running a Neural Cellular Automaton over an octree pyramid:
 *   - the input is average-pooled into L levels (Sec. 3.2, "Repeated hidden
 *     channel upscaling"; supplement S7, table of octree level resolutions);
 *   - the coarsest level starts from the image in the first n_in channels
 *     and zeros in the hidden ones (Sec. 3.1);
 *   - every level runs its own NCA for a number of steps, then its state is
 *     upsampled by nearest neighbour to the next finer level, whose image is
 *     written back into the input channels (Sec. 3.2; supplement S6,
 *     Listings 2 and 3);
 *   - one NCA step (Sec. 3.1; supplement S3, Listing 1) is, for every cell,
 *     a depthwise 3x3 (2D) or 3x3x3 (3D) convolution of each channel with
 *     zero padding plus a bias, concatenated after the cell's own state
 *     (2C features), a linear layer to H hidden units with bias, ReLU, a
 *     linear layer to the hidden channels without bias, multiplied by the
 *     cell's stochastic fire bit and added to the state; input channels are
 *     never changed; the step is computed out of place (supplement S3).
 *
 * Conventions shared by every entry point
 *   - Level 0 is the finest (original resolution), level L-1 the coarsest.
 *   - Extents are (d, h, w); a 2D model uses d = 1.  Cells are stored
 *     row-major over (z, y, x) with the channels innermost ("channels
 *     last"): element (z, y, x, c) of a buffer with c_n channels sits at
 *     ((z*h + y)*w + x)*c_n + c.  State buffers have C channels, images
 *     n_in channels, both in the model's storage type (fp32 or fp16).
 *   - The canonical cell index idx = (z*h + y)*w + x at a level drives the
 *     fire mask, so results do not depend on tiling or launch shape.
 *   - Fire mask (the paper draws it with PyTorch's generator; this library
 *     uses a counter-based generator so any implementation can reproduce
 *     it): Philox4x64-10 (Salmon et al., SC 2011) with counter
 *     (idx >> 3, step, level, b) and key (seed, 0), one call per block of 8
 *     cells; cell idx takes output word (idx >> 1) & 3, its upper 32 bits if
 *     idx is odd and its lower 32 bits if even, and fires iff that draw < T,
 *     where T = min(2^32, floor(fire_rate * 2^32)), fire_rate in [0, 1].
 *     b is the image's index in a batch (octree_nca_infer_batch); every other
 *     entry point uses b = 0.
 *   - Weights are fp32, per level, in device memory, in the layout of
 *     octnca_level_weights.
 *   - All pointers to arrays are DEVICE pointers unless marked "host".
 *     Every buffer is owned by the caller; the library allocates and frees
 *     nothing and keeps no state between calls.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*, NULL =
 *     the default stream) and is asynchronous: no call synchronises the
 *     host.  A device fault surfaces at the caller's next synchronisation.
 *   - Every call checks its arguments before it enqueues anything; on an
 *     invalid argument it returns a negative status, enqueues nothing and
 *     writes nothing.  A failed launch returns OCTNCA_EHIP.
 *   - Calls on different streams are independent.  Buffers written by one
 *     call must not be read or written by another call running at the same
 *     time.
 */
#ifndef OCTREE_NCA_H
#define OCTREE_NCA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OCTNCA_ABI_VERSION 5

typedef enum {
    OCTNCA_OK = 0,
    OCTNCA_EINVAL = -1,       /* null pointer, bad count, fire rate outside [0,1], aliasing */
    OCTNCA_EUNSUPPORTED = -2, /* model (ndim, C, H, n_in, dtype) not compiled in */
    OCTNCA_ESHAPE = -3,       /* extent <= 0, too large, or not divisible by a factor */
    OCTNCA_EHIP = -4,         /* the HIP runtime reported an error */
    OCTNCA_ESPACE = -5        /* workspace too small */
} octnca_status;

typedef enum { OCTNCA_F32 = 0, OCTNCA_F16 = 1 } octnca_dtype;

/* MLP arithmetic of the step kernel (octnca_model.mlp).  The step's
 * definition (Sec. 3.1) fixes no precision; these are the operand types the
 * kernels offer, all accumulating in fp32. */
typedef enum {
    OCTNCA_MLP_AUTO = 0,   /* OCTNCA_MLP_F16S for fp32 states, OCTNCA_MLP_F16 for fp16 states */
    OCTNCA_MLP_F32 = 1,    /* matrix cores, fp32 operands */
    OCTNCA_MLP_BF16X3 = 2, /* matrix cores, operands split into bf16 hi + lo, three products */
    OCTNCA_MLP_F16 = 3,    /* matrix cores, fp16 operands (fp16 states only) */
    OCTNCA_MLP_F16S = 4,   /* matrix cores, activations scaled by 2^-8 and rounded to fp16,
                              weights split into fp16 hi + lo (fp32 states only) */
    OCTNCA_MLP_VALU = 5    /* no matrix cores: one thread per cell, fp32 FMAs */
} octnca_mlp;

/* Work layout of the 2D matrix-core step (octnca_model.layout2d); results do
 * not depend on it.  3D steps ignore it. */
typedef enum {
    OCTNCA_LAYOUT_AUTO = 0,  /* strips of 32 cells streamed over runs of 128 rows, shorter runs
                                (down to 2 rows) on levels with fewer than 1024 such runs; two
                                steps per launch (strips of 30) on levels with >= 2048 of those */
    OCTNCA_LAYOUT_ROWS = 1,  /* as AUTO, with two steps per launch wherever that kernel applies */
    OCTNCA_LAYOUT_TILES = 2  /* 16 x 32 cell tiles, one step per launch */
} octnca_layout;

/* Architecture of one NCA (all levels share it; supplement S3 fixes C and H
 * at compile time) and the step kernel that runs it.  Supported: ndim in
 * {2, 3}, (channels, hidden) in {(16, 64), (12, 48), (20, 100)} (the paper's
 * model and the two other sizes of its ablation, supplement S10), n_in in
 * {1, 3}, state_dtype in {OCTNCA_F32, OCTNCA_F16}.
 * Step kernel: a zero-initialised tail (mlp, layout2d, steps_per_launch all
 * 0) is the library's default.  C = 16, H = 64 takes every option; the
 * other sizes take OCTNCA_MLP_AUTO (the default arithmetic on the matrix
 * cores) or OCTNCA_MLP_VALU only.  With OCTNCA_MLP_AUTO, fp32 states of
 * C = 12, H = 48 run on the kernels of C = 16, H = 64 (in 2D the row kernels:
 * layout2d and steps_per_launch apply as for that size, and
 * OCTNCA_LAYOUT_TILES selects 8 x 32 tiles of a generic kernel); their fp16
 * steps and all steps of C = 20, H = 100 run on that generic kernel.  Combinations that no kernel
 * implements (OCTNCA_MLP_F16 with fp32 states, OCTNCA_MLP_F16S with
 * fp16 states) give OCTNCA_EUNSUPPORTED; values outside the enums give
 * OCTNCA_EINVAL.  The training entry points choose their own arithmetic
 * (split-bf16 MLP operands in the forward, fp32 in the backward) and ignore
 * these three fields. */
typedef struct {
    int32_t ndim;        /* 2: 3x3 taps, d must be 1; 3: 3x3x3 taps */
    int32_t channels;    /* C: state channels per cell */
    int32_t hidden;      /* H: hidden units of the per-cell MLP */
    int32_t n_in;        /* input (image) channels, the first n_in of C */
    int32_t state_dtype; /* storage type of states and images (octnca_dtype) */
    int32_t mlp;         /* octnca_mlp */
    int32_t layout2d;    /* octnca_layout */
    int32_t steps_per_launch; /* 0: two steps per launch on 2D fp32 levels in the row layout
                                 with the OCTNCA_MLP_F16S arithmetic (the state between the
                                 two steps stays on chip; same result bit for bit), one
                                 elsewhere; 1: always one */
} octnca_model;

typedef struct {
    int64_t d, h, w;     /* cells along z (depth / time), y, x */
} octnca_extent;

/* One level's weights, fp32, device memory.  Sizes follow the parameter
 * counts the paper prints (supplement S10 and S11 tables): conv weights and
 * bias, first linear layer with bias, second linear layer without bias. */
typedef struct {
    const float *conv_w; /* [C][3^ndim]: taps row-major over (dz, dy, dx) in {-1,0,1};
                            applied as a cross-correlation (tap (0,0,0) is the cell) */
    const float *conv_b; /* [C] */
    const float *w1;     /* [H][2C]: column k < C multiplies state channel k,
                            column C + k multiplies perception channel k */
    const float *b1;     /* [H] */
    const float *w2;     /* [C][H]: row c gives the update of channel c; rows c < n_in
                            must be allocated but their values are ignored (read,
                            then replaced by 0: input channels are not updated) */
} octnca_level_weights;

/* Image pyramid by node averaging (Sec. 3.2; supplement S7 table).
 *   image          [d][h][w][n_in] finest image (level 0), storage type.
 *   finest         extent of level 0.
 *   levels         L >= 1.
 *   factors        host, [(L-1)*3]: (fz, fy, fx) of the transition from level l to
 *                  l+1 at factors[3l .. 3l+2]; each in 1 .. 8; ndim 2 needs fz = 1.
 *   level_images   host array of L-1 device pointers; level_images[l-1] receives
 *                  level l, [d_l][h_l][w_l][n_in] with d_l = d_{l-1} / fz etc.
 * I_l[z,y,x,c] = mean of I_{l-1} over the fz*fy*fx block at (fz*z, fy*y, fx*x),
 * summed in fp32 and rounded once to the storage type.
 * Errors: EINVAL (null pointer, L < 1), ESHAPE (indivisible extent, bad factor),
 * EUNSUPPORTED, EHIP. */
int octree_nca_build_pyramid(const octnca_model *model, const void *image,
                             octnca_extent finest, int32_t levels, const int32_t *factors,
                             void *const *level_images, void *stream);

/* Upsample one level's state to the next finer level and inject its image
 * (Sec. 3.2; supplement S6, Listings 2 and 3):
 *   fine_state[z,y,x,c] = coarse_state[z/fz, y/fy, x/fx, c]   for c >= n_in,
 *   fine_state[z,y,x,c] = fine_image[z,y,x,c]                  for c <  n_in.
 *   coarse_state  [coarse][C];  factor  host, (fz, fy, fx);
 *   fine_image    [coarse*factor][n_in];  fine_state  [coarse*factor][C], written.
 * fine_state must not overlap coarse_state or fine_image (EINVAL).
 * Errors: EINVAL, ESHAPE, EUNSUPPORTED, EHIP. */
int octree_nca_upsample(const octnca_model *model, const void *coarse_state,
                        octnca_extent coarse, const int32_t *factor, const void *fine_image,
                        void *fine_state, void *stream);

/* Run `steps` NCA steps t = 0 .. steps-1 of one level (Sec. 3.1; supplement
 * S3, Listing 1), out of place, alternating between two buffers: launch k
 * reads bufs[k % 2] and writes bufs[(k+1) % 2].  A launch runs one step, or
 * two (t, t+1) where model->steps_per_launch allows it and the level runs the
 * 2D fp32 row layout; the state after step t then stays on chip and the
 * result is the same bit for bit.  The number of two-step launches is kept
 * even, so the final state is in buf1 exactly when `steps` is odd, whatever
 * kernels run and on whatever device.
 *   buf0     [extent][C], the level's state on entry.
 *   buf1     [extent][C], scratch of the same size; must not overlap buf0.
 *   weights  host pointer to one octnca_level_weights (device arrays).
 *   level    the level index, used only by the fire mask (0 = finest).
 *   steps    >= 0; 0 leaves buf0 as it is.
 *   fire_rate in [0, 1]; seed: fire-mask key.
 *   result_in_buf1  host, may be NULL: set to steps % 2 (1 when the final
 *            state is in buf1, 0 when it is in buf0).
 * Errors: EINVAL, ESHAPE, EUNSUPPORTED, EHIP. */
int octree_nca_run_level(const octnca_model *model, void *buf0, void *buf1,
                         octnca_extent extent, const octnca_level_weights *weights,
                         int32_t level, int32_t steps, float fire_rate, uint64_t seed,
                         int32_t *result_in_buf1, void *stream);

/* Two-class readout on the finest level (Sec. 3.2 predicts the segmentation
 * in the last hidden channels): seg[p] = 1 if state[p, C-1] > state[p, C-2],
 * else 0 (ties and NaNs give 0).
 *   state [extent][C];  seg [extent] uint8, written.
 * Errors: EINVAL, ESHAPE, EUNSUPPORTED, EHIP. */
int octree_nca_readout(const octnca_model *model, const void *state, octnca_extent extent,
                       uint8_t *seg, void *stream);

/* K-class readout on the finest level, for models whose last K hidden
 * channels score K classes (the paper's surgery data has several classes,
 * Sec. 4): seg[p] = the index k in [0, K) of the largest of
 * state[p, C-K+k], found by scanning k upwards and moving only on a strictly
 * greater value, so ties go to the lower class and a NaN never replaces an
 * earlier channel.  K = 2 gives the same result as octree_nca_readout.
 *   state [extent][C];  classes K in [2, C - n_in];  seg [extent] uint8, written.
 * Errors: EINVAL (null pointer, K out of range), ESHAPE, EUNSUPPORTED, EHIP. */
int octree_nca_readout_classes(const octnca_model *model, const void *state,
                               octnca_extent extent, int32_t classes, uint8_t *seg,
                               void *stream);

/* Bytes of device workspace octree_nca_infer needs for this model, finest
 * extent and pyramid: the images of levels 1..L-1, plus one finest-size state
 * buffer when final_state is given (two when it is NULL), each 256-byte
 * aligned.  Returns 0 on invalid arguments. */
size_t octree_nca_workspace_bytes(const octnca_model *model, octnca_extent finest,
                                  int32_t levels, const int32_t *factors,
                                  int32_t with_final_state);

/* Whole OctreeNCA inference (Sec. 3.2; supplement S6, Listing 3): pyramid,
 * coarsest seed (image in channels < n_in, zeros elsewhere), then for
 * l = L-1 .. 0: upsample + inject (l < L-1) and steps[l] NCA steps with
 * weights[l]; finally the readout.
 *   image        [finest][n_in], storage type.
 *   factors      host, [(L-1)*3] as in octree_nca_build_pyramid.
 *   weights      host, [L]; index 0 = finest level.
 *   steps        host, [L]; steps[l] >= 0.
 *   workspace    device, >= octree_nca_workspace_bytes(..., final_state != NULL).
 *   final_state  [finest][C] written with the final state, or NULL.
 *   seg          [finest] uint8 written with the readout, or NULL.
 *   level_events host, NULL or [2*L] hipEvent_t handles (void*): event 2l is
 *                recorded on `stream` before level l's first step and 2l+1
 *                after its last step (timing hook; events are not created here).
 * The final state lands directly in final_state (no copy): the buffer order is
 * chosen from the parity of the step counts.
 * Errors: EINVAL, ESHAPE, EUNSUPPORTED, ESPACE, EHIP. */
int octree_nca_infer(const octnca_model *model, const void *image, octnca_extent finest,
                     int32_t levels, const int32_t *factors,
                     const octnca_level_weights *weights, const int32_t *steps,
                     float fire_rate, uint64_t seed, void *workspace, size_t workspace_bytes,
                     void *final_state, uint8_t *seg, void *const *level_events, void *stream);

/* Step-kernel launches that octree_nca_infer enqueues for each level with the
 * model's step kernel (a measurement aid: the launches of a level add up to
 * its steps, one or two steps per launch).  The count depends only on the
 * arguments, not on the device.
 *   launches  host, [L], written: launches[l] for level l (index 0 = finest).
 * Host only: enqueues nothing.  Errors: EINVAL (null pointer, a negative
 * step count), ESHAPE, EUNSUPPORTED. */
int octree_nca_infer_launches(const octnca_model *model, octnca_extent finest, int32_t levels,
                              const int32_t *factors, const int32_t *steps, int32_t *launches);

/* Size of the static device array octree_nca_infer_static uses as its
 * workspace (64 MiB per device). */
#define OCTNCA_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

/* octree_nca_infer for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same inference, with the workspace taken from a static device array of
 * OCTNCA_STATIC_SCRATCH_BYTES that the library holds on each device it runs
 * on until the process ends.  The call allocates nothing (no hipMalloc, no
 * hipFree, no allocating library routine); the first call on a device looks
 * the array's address up once.  The caller passes inputs and outputs as for
 * octree_nca_infer; final_state is required.
 *   Arguments: as octree_nca_infer, without workspace and level_events.
 *   final_state  [finest][C], written; must not be NULL.
 * Workspace needed: octree_nca_workspace_bytes(..., with_final_state = 1)
 * (pyramid images of levels 1..L-1 plus one finest-size state buffer); a
 * larger need returns OCTNCA_ESPACE before anything is enqueued.
 * Every call on one device uses that device's one array, which keeps what the
 * last call left there (nothing in it needs to start at zero): calls that may
 * run at the same time on one device (other streams, other host threads) race
 * and must be serialised by the caller.
 * Errors: EINVAL (as octree_nca_infer; final_state NULL), ESHAPE, EUNSUPPORTED,
 * ESPACE (the workspace would exceed the static array), EHIP. */
int octree_nca_infer_static(const octnca_model *model, const void *image, octnca_extent finest,
                            int32_t levels, const int32_t *factors,
                            const octnca_level_weights *weights, const int32_t *steps,
                            float fire_rate, uint64_t seed, void *final_state, uint8_t *seg,
                            void *stream);

/* Inference of a batch of images of the same extent (the paper's kernel
 * works on one image and notes that a batch is an extra dimension to iterate
 * over, supplement S3): image b runs exactly as octree_nca_infer, with the
 * fire-mask counter word 3 set to b, so the images draw independent masks and
 * image 0 reproduces octree_nca_infer.  The images run one after another on
 * `stream` and share one workspace.
 *   images       [batch][finest][n_in], storage type;  batch >= 1.
 *   workspace    device, >= octree_nca_workspace_bytes(..., final_states != NULL).
 *   final_states [batch][finest][C] written, or NULL.
 *   segs         [batch][finest] uint8 written with the two-class readout, or NULL.
 * Outputs must not overlap the images or the workspace (EINVAL).  All images'
 * arguments are checked before anything is enqueued.  A batch whose states
 * would exceed 2^48 bytes is rejected (EINVAL).
 * Errors: EINVAL, ESHAPE, EUNSUPPORTED, ESPACE, EHIP. */
int octree_nca_infer_batch(const octnca_model *model, const void *images, int32_t batch,
                           octnca_extent finest, int32_t levels, const int32_t *factors,
                           const octnca_level_weights *weights, const int32_t *steps,
                           float fire_rate, uint64_t seed, void *workspace,
                           size_t workspace_bytes, void *final_states, uint8_t *segs,
                           void *stream);

/* Number of steps of the first (coarsest) level under the schedule rule of
 * the paper's ablation (supplement S10): alpha0 * max(H, W, D) of that level,
 * rounded down (the paper does not state the rounding; its alpha0 values are
 * 1.0, 1.5 and 2.0).  With alpha0 = 1 this is the max(H, W) / 2^L steps that
 * Sec. 3.2 names as enough to carry information across the coarsest level.
 *   alpha0    >= 0 and finite;  coarsest  extent of level L-1 (d = 1 for 2D).
 * Returns the step count, or -1 for invalid arguments or a count above
 * INT32_MAX.  Host only: enqueues nothing. */
int32_t octree_nca_first_level_steps(float alpha0, octnca_extent coarsest);

/* Export the fire mask of one step of one level (test hook for the
 * generator described above): mask[idx] = 1 if cell idx fires, else 0.
 *   mask [extent] uint8, written.
 * Errors: EINVAL, ESHAPE, EHIP. */
int octree_nca_fire_mask(uint64_t seed, int32_t level, int32_t step, octnca_extent extent,
                         float fire_rate, uint8_t *mask, void *stream);

/* ---------------------------------------------------------------------------
 * Training gradients (fp32 states only).  The paper trains OctreeNCA end to
 * end by backpropagation through every step of every level (Sec. 3.2,
 * efficient training; supplement S7).  These calls give the gradient of a
 * scalar loss with respect to each level's weights, recomputing a step's
 * activations from its input state (only states are kept).  Other storage
 * types return OCTNCA_EUNSUPPORTED.
 * ------------------------------------------------------------------------- */

/* One level's weight gradients, fp32, device memory, the layouts of
 * octnca_level_weights. */
typedef struct {
    float *conv_w; /* [C][3^ndim] */
    float *conv_b; /* [C] */
    float *w1;     /* [H][2C] */
    float *b1;     /* [H] */
    float *w2;     /* [C][H]; rows c < n_in receive 0 */
} octnca_level_grads;

/* Bytes of workspace octree_nca_step_backward needs for `extent` (0 if the
 * model or extent is invalid). */
size_t octree_nca_step_backward_workspace_bytes(const octnca_model *model, octnca_extent extent);

/* Backward of one NCA step (Sec. 3.1 step; supplement S3 Listing 1):
 *   state      [extent][C] fp32, the state the step read (level `level`, step `step`);
 *   grad_out   [extent][C] fp32, dL/dS' of the step's output;
 *   grad_in    [extent][C] fp32, receives dL/dS of its input; may be grad_out itself
 *              (in place), must not overlap state or workspace otherwise;
 *   grads      the step's weight gradients are ADDED to these (zero them first);
 *   fire_rate, seed, level, step  as for octree_nca_run_level (same fire mask).
 * dL/dS = G' + [W1^T ga]_state + transposed depthwise conv of [W1^T ga]_perception,
 * with ga = (W2^T m G'_hidden) * [W1 f + b1 > 0]; ReLU' is 0 at 0.
 * Errors: EINVAL (null, aliasing, level/step < 0, fire rate), ESPACE, ESHAPE,
 * EUNSUPPORTED (fp16), EHIP. */
int octree_nca_step_backward(const octnca_model *model, const void *state, const void *grad_out,
                             octnca_extent extent, const octnca_level_weights *weights,
                             int32_t level, int32_t step, float fire_rate, uint64_t seed,
                             void *grad_in, const octnca_level_grads *grads, void *workspace,
                             size_t workspace_bytes, void *stream);

/* Adjoint of octree_nca_upsample (Sec. 3.2): grad_coarse[q][c] = sum of
 * grad_fine over q's fz*fy*fx children for c >= n_in, 0 for c < n_in (the input
 * channels are overwritten by the image).  grad_fine [coarse * factor][C],
 * grad_coarse [coarse][C], fp32, not overlapping.  Errors: EINVAL, ESHAPE,
 * EUNSUPPORTED, EHIP. */
int octree_nca_upsample_backward(const octnca_model *model, const void *grad_fine,
                                 octnca_extent coarse, const int32_t *factor, void *grad_coarse,
                                 void *stream);

/* Bytes of workspace octree_nca_readout_mse needs (0 for an invalid extent). */
size_t octree_nca_readout_mse_workspace_bytes(octnca_extent extent);

/* Synthetic training loss on the readout channels (the last two, Sec. 3.2):
 *   L = 1/2 sum over cells and k in {0, 1} of (state[p][C-2+k] - target[p][k])^2.
 *   target [extent][2] fp32; grad [extent][C] fp32 receives dL/dS (zero in the
 *   other channels); *loss (device double) receives L, summed in fp64.
 * Errors: EINVAL, ESPACE, ESHAPE, EUNSUPPORTED, EHIP. */
int octree_nca_readout_mse(const octnca_model *model, const void *state, const float *target,
                           octnca_extent extent, void *grad, double *loss, void *workspace,
                           size_t workspace_bytes, void *stream);

/* Bytes of workspace octree_nca_train_step needs: pyramid images, every state
 * of every level, two finest-size gradients and the backward's workspace
 * (0 if an argument is invalid). */
size_t octree_nca_train_workspace_bytes(const octnca_model *model, octnca_extent finest,
                                        int32_t levels, const int32_t *factors,
                                        const int32_t *steps);

/* One fused training step: the inference of octree_nca_infer (same arguments,
 * split-bf16 MLP operands, products to about 2^-16) keeping every state,
 * the readout MSE against `target`,
 * and the backward through all steps and levels (finest first, the upsample's
 * adjoint between levels).
 *   grads   host array of `levels` gradient sets (index = level), OVERWRITTEN;
 *   loss    device double, receives L;
 *   final_state  [finest][C] fp32 or NULL: receives the forward's final state.
 * Errors: EINVAL, ESPACE, ESHAPE, EUNSUPPORTED (fp16), EHIP. */
int octree_nca_train_step(const octnca_model *model, const void *image, octnca_extent finest,
                          int32_t levels, const int32_t *factors,
                          const octnca_level_weights *weights, const int32_t *steps,
                          float fire_rate, uint64_t seed, const float *target, void *workspace,
                          size_t workspace_bytes, const octnca_level_grads *grads, double *loss,
                          void *final_state, void *stream);

/* Static text for a status code; never NULL. */
const char *octree_nca_strerror(int status);

/* OCTNCA_ABI_VERSION of the built library. */
int octree_nca_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* OCTREE_NCA_H */
