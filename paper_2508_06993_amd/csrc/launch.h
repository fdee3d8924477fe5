// Internal launch interface between the C ABI layer (api.hip) and the kernel
// files.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"

namespace octnca {

struct Extent3 {
    int64_t d, h, w;
    int64_t cells() const { return d * h * w; }
};

enum class Dtype : int { F32 = 0, F16 = 1 };

// Pyramid: dst = mean of src over (fz, fy, fx) blocks; dst_ext = src_ext / f.
hipError_t launch_pool(Dtype dt, const void *src, Extent3 dst_ext, void *dst, int fz, int fy,
                       int fx, int n_in, hipStream_t stream);

// Upsample + inject.  coarse == nullptr seeds the hidden channels with zeros
// (coarsest level initialisation, factors then must be 1).
hipError_t launch_upsample(Dtype dt, const void *coarse, Extent3 fine_ext, int fz, int fy, int fx,
                           const void *img, void *fine, int n_in, int channels,
                           hipStream_t stream);
hipError_t launch_readout(Dtype dt, const void *state, int64_t cells, int channels, uint8_t *seg,
                          hipStream_t stream);
hipError_t launch_readout_classes(Dtype dt, const void *state, int64_t cells, int channels,
                                  int classes, uint8_t *seg, hipStream_t stream);

hipError_t launch_fire_mask(uint64_t seed, uint32_t level, uint32_t step, int64_t cells,
                            uint64_t threshold, uint8_t *mask, hipStream_t stream);

// MLP operand precision of the MFMA step kernel.  Default: scaled fp16
// activations with split fp16 weights (F16S) for fp32 states, fp16 for fp16 states.
enum class MfmaMlp : int { Default = 0, F32 = 1, Bf16x3 = 2, F16 = 3, F16S = 4 };
// Work layout of the 2D MFMA step.  Auto: row streaming on large levels,
// 16 x 32 tiles on small ones; Rows / Tiles force one (3D steps ignore it).
enum class Layout2d : int { Auto = 0, Rows = 1, Tiles = 2 };
// Step kernel chosen by the caller (the model description of the C ABI):
// vector kernel or matrix cores, MLP operands, 2D work layout, and whether
// two steps may run in one launch.  The default-constructed value is the
// library's default.
struct KernelChoice {
    bool valu = false;    // one thread per cell on the vector ALUs
    bool pairs = true;    // two steps per launch where the two-step kernel applies
    MfmaMlp mlp = MfmaMlp::Default;
    Layout2d layout = Layout2d::Auto;
};

// One NCA step src -> dst over a level of extent `ext`.
struct StepArgs {
    Dtype dtype;
    int ndim;
    int n_in;
    Extent3 ext;
    LevelWeightsDev w;
    uint32_t level;
    uint32_t step;
    uint32_t batch = 0;   // image index in a batch (fire-mask counter word 3)
    int channels = kC;    // C and H of the model (the matrix-core kernels need 16 / 64)
    int hidden = kH;
    uint64_t seed;
    uint64_t threshold;
    // Device [cells] uint8 or null: a two-step launch, or a single step of the
    // fp16 3D kernel (see step_single_fuses_readout), also writes the
    // two-class readout of the state it stores.
    uint8_t *seg = nullptr;
    KernelChoice kc;      // step kernel of the matrix-core / vector paths
};
hipError_t launch_step(const StepArgs &a, const void *src, void *dst, hipStream_t stream);
// Whether launch_step would fuse a level's first step with the upsample from
// the next coarser level (see launch_step_mfma_up), and that fused launch.
bool step_fuses_upsample(const StepArgs &a);
hipError_t launch_step_up(const StepArgs &a, const void *coarse, int coarse_h, int coarse_w,
                          int fz, int fy, int fx, const void *img, void *dst,
                          hipStream_t stream);
hipError_t launch_step_valu(const StepArgs &a, const void *src, void *dst, hipStream_t stream);
// Matrix-core step for the model sizes other than C = 16, H = 64 (the
// ablation's 12 / 48 and 20 / 100): whether it serves `a`, and the launch.
bool step_gen_serves(const StepArgs &a);
hipError_t launch_step_gen(const StepArgs &a, const void *src, void *dst, hipStream_t stream);
// Whether launch_step_pair runs steps a.step and a.step + 1 in one launch, and
// that launch (the state after step a.step is not written to memory).
bool step_pairs(const StepArgs &a);
// Whether the single-step launch that launch_step makes for `a` writes StepArgs::seg.
bool step_single_fuses_readout(const StepArgs &a);
hipError_t launch_step_pair(const StepArgs &a, const void *src, void *dst, hipStream_t stream);
// The first two steps of a level, the first fused with the upsample (when
// step_pairs and step_fuses_upsample both hold).
hipError_t launch_step_pair_up(const StepArgs &a, const void *coarse, int coarse_w, int fz,
                               int fy, int fx, const void *img, void *dst, hipStream_t stream);

// Training (fp32 states): backward of one step (state `src` before the step,
// gout = dL/dS'), writing gin = dL/dS (may alias gout) and adding the weight
// gradients to g; ws holds step_backward_workspace_floats floats.
size_t step_backward_workspace_floats(int ndim, int channels, int hidden, Extent3 extent);
hipError_t launch_step_backward(const StepArgs &a, const float *src, const float *gout,
                                float *gin, LevelGradsDev g, float *ws, hipStream_t stream);
// Backward of all `steps` steps of a level (a.step unused): states holds the
// level's states before steps 0 .. steps-1 (state t at states + t * cells * C),
// gout = dL/dS after the last step; gin receives dL/dS of the level's first
// state (must not alias gout or states) and g receives the level's weight
// gradients (written, not added: the buffers need no clearing).  ws holds
// level_backward_workspace_floats floats.  steps = 0 enqueues nothing (neither
// gin nor g is written).
size_t level_backward_workspace_floats(int ndim, int channels, int hidden, Extent3 extent);
hipError_t launch_level_backward(const StepArgs &a, int32_t steps, const float *states,
                                 const float *gout, float *gin, LevelGradsDev g, float *ws,
                                 hipStream_t stream);
// Adjoint of the upsample + inject from `coarse` (extent of the coarse level).
hipError_t launch_upsample_adjoint(const float *gfine, Extent3 coarse, int fz, int fy, int fx,
                                   int n_in, int channels, float *gcoarse, hipStream_t stream);
// Readout-channel MSE: grad = dL/dS, *loss = L (device); ws holds
// mse_workspace_doubles doubles.
size_t mse_workspace_doubles(int64_t cells);
hipError_t launch_readout_mse(const float *state, const float *target, int64_t cells, int channels,
                              float *grad, double *loss, double *ws, hipStream_t stream);
hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t stream);
// The specialised matrix-core steps: every step of C = 16, H = 64 models and
// the 2D fp32 steps of C = 12, H = 48 models in the row layout (default
// operand policy); step_mfma_serves says whether launch_step_mfma runs `a`.
bool step_mfma_serves(const StepArgs &a, Layout2d layout);
hipError_t launch_step_mfma(const StepArgs &a, MfmaMlp mlp, Layout2d layout, const void *src,
                            void *dst, hipStream_t stream);
// The first step of a level fused with the upsample + inject from the next
// coarser level (2D row-streaming kernel and fp16 3D kernel, default operand
// policy only):
// step_mfma_fuses_upsample says whether launch_step_mfma would run that kernel
// for `a`; launch_step_mfma_up then reads the coarse state (width coarse_w,
// factors fy, fx) and the level's image instead of a state of the level.
bool step_mfma_fuses_upsample(const StepArgs &a, MfmaMlp mlp, Layout2d layout);
// Two steps, a.step and a.step + 1, in one launch (2D fp32 row layout, default
// operand policy): step_mfma_pairs says whether that kernel exists for `a`;
// launch_step2_mfma reads src and writes the state after both steps to dst.
bool step_mfma_pairs(const StepArgs &a, MfmaMlp mlp, Layout2d layout);
// Whether a single-step launch of launch_step_mfma for `a` writes StepArgs::seg.
bool step_mfma_single_readout(const StepArgs &a, MfmaMlp mlp);
hipError_t launch_step2_mfma(const StepArgs &a, MfmaMlp mlp, Layout2d layout, const void *src,
                             void *dst, hipStream_t stream);
// The same two steps with step a.step fused with the upsample + inject from
// the coarse state (width coarse_w, factors fy, fx) and the level's image.
hipError_t launch_step2_mfma_up(const StepArgs &a, MfmaMlp mlp, Layout2d layout,
                                const void *coarse, int coarse_w, int fy, int fx, const void *img,
                                void *dst, hipStream_t stream);
hipError_t launch_step_mfma_up(const StepArgs &a, Layout2d layout, const void *coarse,
                               int coarse_h, int coarse_w, int fz, int fy, int fx,
                               const void *img, void *dst, hipStream_t stream);

}  // namespace octnca
