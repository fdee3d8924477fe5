// C ABI of the OctreeNCA inference library (include/octree_nca.h): argument
// checks, buffer planning and the launch sequence of the octree inference
// (Sec. 3.2; supplement S6, Listing 3).  Every entry point validates all of its
// arguments before it enqueues any work, allocates nothing and never
// synchronises the host.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <cmath>
#include <algorithm>
#include <mutex>
#include <utility>
#include "launch.h"
#include "octree_nca.h"

using namespace octnca;

namespace {

constexpr int64_t kMaxDim = int64_t(1) << 30;      // per axis (kernels index with int)
constexpr int64_t kMaxCells = int64_t(1) << 36;    // per level
constexpr int kMaxLevels = 16;
constexpr size_t kAlign = 256;

size_t align_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

int check_model(const octnca_model *m) {
    if (m == nullptr) return OCTNCA_EINVAL;
    if (m->ndim != 2 && m->ndim != 3) return OCTNCA_EUNSUPPORTED;
    // C / H: the paper's 16 / 64 and the 12 / 48 and 20 / 100 of its ablation
    // (supplement S10); every size runs on the matrix cores (the specialised
    // kernels for 16 / 64 and fp32 12 / 48, a generic kernel otherwise) and on
    // the vector kernel
    const bool size_ok = (m->channels == 16 && m->hidden == 64) ||
                         (m->channels == 12 && m->hidden == 48) ||
                         (m->channels == 20 && m->hidden == 100);
    if (!size_ok) return OCTNCA_EUNSUPPORTED;
    if (m->n_in != 1 && m->n_in != 3) return OCTNCA_EUNSUPPORTED;
    if (m->state_dtype != OCTNCA_F32 && m->state_dtype != OCTNCA_F16) return OCTNCA_EUNSUPPORTED;
    // step kernel choice
    if (m->mlp < OCTNCA_MLP_AUTO || m->mlp > OCTNCA_MLP_VALU) return OCTNCA_EINVAL;
    if (m->layout2d < OCTNCA_LAYOUT_AUTO || m->layout2d > OCTNCA_LAYOUT_TILES) return OCTNCA_EINVAL;
    if (m->steps_per_launch != 0 && m->steps_per_launch != 1) return OCTNCA_EINVAL;
    if (!(m->channels == 16 && m->hidden == 64) && m->mlp != OCTNCA_MLP_AUTO &&
        m->mlp != OCTNCA_MLP_VALU)
        return OCTNCA_EUNSUPPORTED;   // only the vector kernel serves the other sizes
    if (m->mlp == OCTNCA_MLP_F16 && m->state_dtype != OCTNCA_F16) return OCTNCA_EUNSUPPORTED;
    if (m->mlp == OCTNCA_MLP_F16S && m->state_dtype != OCTNCA_F32) return OCTNCA_EUNSUPPORTED;
    return OCTNCA_OK;
}

// The caller's step-kernel choice (fields checked by check_model).
KernelChoice kernel_choice(const octnca_model *m) {
    KernelChoice k;
    k.valu = m->mlp == OCTNCA_MLP_VALU;
    k.pairs = m->steps_per_launch == 0;
    switch (m->mlp) {
        case OCTNCA_MLP_F32: k.mlp = MfmaMlp::F32; break;
        case OCTNCA_MLP_BF16X3: k.mlp = MfmaMlp::Bf16x3; break;
        case OCTNCA_MLP_F16: k.mlp = MfmaMlp::F16; break;
        case OCTNCA_MLP_F16S: k.mlp = MfmaMlp::F16S; break;
        default: k.mlp = MfmaMlp::Default; break;
    }
    k.layout = m->layout2d == OCTNCA_LAYOUT_ROWS    ? Layout2d::Rows
               : m->layout2d == OCTNCA_LAYOUT_TILES ? Layout2d::Tiles
                                                    : Layout2d::Auto;
    return k;
}

int check_extent(const octnca_model *m, const octnca_extent &e) {
    if (e.d <= 0 || e.h <= 0 || e.w <= 0) return OCTNCA_ESHAPE;
    if (e.d > kMaxDim || e.h > kMaxDim || e.w > kMaxDim) return OCTNCA_ESHAPE;
    if (m->ndim == 2 && e.d != 1) return OCTNCA_ESHAPE;
    // d * h <= 2^60 cannot overflow; the cell count is bounded by division
    // (d * h * w itself could reach 2^90)
    if (e.d * e.h > kMaxCells || e.w > kMaxCells / (e.d * e.h)) return OCTNCA_ESHAPE;
    return OCTNCA_OK;
}

int check_factor(const octnca_model *m, const int32_t *f) {
    for (int a = 0; a < 3; ++a)
        if (f[a] < 1 || f[a] > 8) return OCTNCA_ESHAPE;
    if (m->ndim == 2 && f[0] != 1) return OCTNCA_ESHAPE;
    return OCTNCA_OK;
}

// fire_rate in [0, 1] (NaN rejected); threshold = min(2^32, floor(rate * 2^32)).
bool fire_threshold(float rate, uint64_t *out) {
    if (!(rate >= 0.0f && rate <= 1.0f)) return false;
    const double t = floor((double)rate * 4294967296.0);
    *out = t >= 4294967296.0 ? (uint64_t(1) << 32) : (uint64_t)t;
    return true;
}

size_t elem_bytes(const octnca_model *m) { return m->state_dtype == OCTNCA_F16 ? 2 : 4; }

Extent3 ext3(const octnca_extent &e) { return Extent3{e.d, e.h, e.w}; }

bool overlap(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
    return pa < pb + nb && pb < pa + na;
}

int hip_status(hipError_t e) { return e == hipSuccess ? OCTNCA_OK : OCTNCA_EHIP; }

// Level extents, finest first; ESHAPE when a factor does not divide.
int level_extents(const octnca_model *m, octnca_extent finest, int32_t levels,
                  const int32_t *factors, octnca_extent *out) {
    if (levels < 1 || levels > kMaxLevels) return OCTNCA_EINVAL;
    if (levels > 1 && factors == nullptr) return OCTNCA_EINVAL;
    int st = check_extent(m, finest);
    if (st) return st;
    out[0] = finest;
    for (int l = 1; l < levels; ++l) {
        const int32_t *f = factors + 3 * (l - 1);
        if ((st = check_factor(m, f))) return st;
        const octnca_extent &p = out[l - 1];
        if (p.d % f[0] || p.h % f[1] || p.w % f[2]) return OCTNCA_ESHAPE;
        out[l] = octnca_extent{p.d / f[0], p.h / f[1], p.w / f[2]};
    }
    return OCTNCA_OK;
}

bool weights_ok(const octnca_level_weights *w) {
    return w != nullptr && w->conv_w && w->conv_b && w->w1 && w->b1 && w->w2;
}

LevelWeightsDev to_dev(const octnca_level_weights *w) {
    return LevelWeightsDev{w->conv_w, w->conv_b, w->w1, w->b1, w->w2};
}

Dtype dtype_of(const octnca_model *m) { return m->state_dtype == OCTNCA_F16 ? Dtype::F16 : Dtype::F32; }

StepArgs step_args(const octnca_model *m, const octnca_extent &e, const octnca_level_weights *w,
                   int32_t level, uint64_t seed, uint64_t threshold, uint32_t batch) {
    StepArgs a;
    a.batch = batch;
    a.dtype = dtype_of(m);
    a.ndim = m->ndim;
    a.n_in = m->n_in;
    a.ext = ext3(e);
    a.w = to_dev(w);
    a.level = (uint32_t)level;
    a.step = 0;
    a.seed = seed;
    a.threshold = threshold;
    a.channels = m->channels;
    a.hidden = m->hidden;
    a.kc = kernel_choice(m);
    return a;
}

// Launches that run steps t0 .. t1-1 of a level: one per step, or one per two
// steps where the two-step kernel applies (a trailing odd step runs alone).
int32_t level_launches(const StepArgs &a, int32_t t0, int32_t t1) {
    if (t1 <= t0) return 0;
    return step_pairs(a) ? (t1 - t0 + 1) / 2 : t1 - t0;
}

// Steps run by a level's first launch when it is fused with the upsample: two
// where the two-step kernel applies and the level has two steps, else one; 0
// when the first step is not fused.
int32_t fused_up_steps(const StepArgs &a, bool fused, int32_t steps) {
    if (!fused) return 0;
    return steps >= 2 && step_pairs(a) ? 2 : 1;
}

// Enqueue steps t0 .. t1-1 of a level; launch k reads bufs[k % 2] and writes
// bufs[(k + 1) % 2], so the result is in bufs[level_launches(..) % 2].
// seg_last: the last launch also writes the readout of its result there (null:
// no readout); the caller passes it only where that launch's kernel can.
// max_pairs caps the two-step launches (the remaining steps run one per
// launch); it is unlimited by default.
int run_steps(const octnca_model *m, void *b0, void *b1, const octnca_extent &e,
              const octnca_level_weights *w, int32_t level, int32_t t0, int32_t t1,
              uint64_t seed, uint64_t threshold, hipStream_t stream, uint32_t batch = 0,
              uint8_t *seg_last = nullptr, int32_t max_pairs = INT32_MAX) {
    StepArgs a = step_args(m, e, w, level, seed, threshold, batch);
    void *bufs[2] = {b0, b1};
    const bool pairs = step_pairs(a);
    int k = 0;
    int32_t pairs_left = max_pairs;
    for (int32_t t = t0; t < t1; k ^= 1) {
        a.step = (uint32_t)t;
        hipError_t err;
        if (pairs && pairs_left > 0 && t + 1 < t1) {
            --pairs_left;
            a.seg = t + 2 == t1 ? seg_last : nullptr;
            err = launch_step_pair(a, bufs[k], bufs[k ^ 1], stream);
            a.seg = nullptr;
            t += 2;
        } else {
            a.seg = t + 1 == t1 ? seg_last : nullptr;
            err = launch_step(a, bufs[k], bufs[k ^ 1], stream);
            a.seg = nullptr;
            t += 1;
        }
        if (err != hipSuccess) return OCTNCA_EHIP;
    }
    return OCTNCA_OK;
}

struct Plan {
    octnca_extent ext[kMaxLevels];
    size_t image_off[kMaxLevels];   // workspace offsets of level images 1..L-1
    size_t state_off[2];            // workspace offsets of the state buffers it holds
    size_t bytes;
};

int make_plan(const octnca_model *m, octnca_extent finest, int32_t levels, const int32_t *factors,
              bool with_final_state, Plan *p) {
    int st = check_model(m);
    if (st) return st;
    if ((st = level_extents(m, finest, levels, factors, p->ext))) return st;
    const size_t eb = elem_bytes(m);
    size_t off = 0;
    p->image_off[0] = 0;
    for (int l = 1; l < levels; ++l) {
        p->image_off[l] = off;
        off += align_up((size_t)(p->ext[l].d * p->ext[l].h * p->ext[l].w) * m->n_in * eb);
    }
    const size_t state_bytes = align_up((size_t)(finest.d * finest.h * finest.w) * m->channels * eb);
    p->state_off[0] = off;
    off += state_bytes;
    p->state_off[1] = off;
    if (!with_final_state) off += state_bytes;
    p->bytes = off;
    return OCTNCA_OK;
}

}  // namespace

extern "C" {

int octree_nca_abi_version(void) { return OCTNCA_ABI_VERSION; }

const char *octree_nca_strerror(int status) {
    switch (status) {
        case OCTNCA_OK: return "ok";
        case OCTNCA_EINVAL: return "invalid argument";
        case OCTNCA_EUNSUPPORTED: return "model configuration not compiled into this library";
        case OCTNCA_ESHAPE: return "invalid extent or pooling factor";
        case OCTNCA_EHIP: return "HIP runtime error";
        case OCTNCA_ESPACE: return "workspace too small";
        default: return "unknown status";
    }
}

int octree_nca_build_pyramid(const octnca_model *model, const void *image, octnca_extent finest,
                             int32_t levels, const int32_t *factors, void *const *level_images,
                             void *stream) {
    int st = check_model(model);
    if (st) return st;
    octnca_extent ext[kMaxLevels];
    if ((st = level_extents(model, finest, levels, factors, ext))) return st;
    if (image == nullptr || (levels > 1 && level_images == nullptr)) return OCTNCA_EINVAL;
    for (int l = 1; l < levels; ++l)
        if (level_images[l - 1] == nullptr) return OCTNCA_EINVAL;
    const hipStream_t s = (hipStream_t)stream;
    const void *prev = image;
    for (int l = 1; l < levels; ++l) {
        const int32_t *f = factors + 3 * (l - 1);
        const hipError_t e = launch_pool(dtype_of(model), prev, ext3(ext[l]), level_images[l - 1],
                                         f[0], f[1], f[2], model->n_in, s);
        if (e != hipSuccess) return OCTNCA_EHIP;
        prev = level_images[l - 1];
    }
    return OCTNCA_OK;
}

int octree_nca_upsample(const octnca_model *model, const void *coarse_state, octnca_extent coarse,
                        const int32_t *factor, const void *fine_image, void *fine_state,
                        void *stream) {
    int st = check_model(model);
    if (st) return st;
    if (factor == nullptr || coarse_state == nullptr || fine_image == nullptr ||
        fine_state == nullptr)
        return OCTNCA_EINVAL;
    if ((st = check_extent(model, coarse)) || (st = check_factor(model, factor))) return st;
    const octnca_extent fine{coarse.d * factor[0], coarse.h * factor[1], coarse.w * factor[2]};
    if ((st = check_extent(model, fine))) return st;
    const size_t eb = elem_bytes(model);
    const size_t fine_bytes = (size_t)(fine.d * fine.h * fine.w) * model->channels * eb;
    if (overlap(fine_state, fine_bytes, coarse_state,
                (size_t)(coarse.d * coarse.h * coarse.w) * model->channels * eb) ||
        overlap(fine_state, fine_bytes, fine_image,
                (size_t)(fine.d * fine.h * fine.w) * model->n_in * eb))
        return OCTNCA_EINVAL;
    return hip_status(launch_upsample(dtype_of(model), coarse_state, ext3(fine), factor[0],
                                      factor[1], factor[2], fine_image, fine_state, model->n_in,
                                      model->channels, (hipStream_t)stream));
}

int octree_nca_run_level(const octnca_model *model, void *buf0, void *buf1, octnca_extent extent,
                         const octnca_level_weights *weights, int32_t level, int32_t steps,
                         float fire_rate, uint64_t seed, int32_t *result_in_buf1, void *stream) {
    int st = check_model(model);
    if (st) return st;
    if ((st = check_extent(model, extent))) return st;
    uint64_t threshold;
    if (buf0 == nullptr || buf1 == nullptr || !weights_ok(weights) || level < 0 || steps < 0 ||
        !fire_threshold(fire_rate, &threshold))
        return OCTNCA_EINVAL;
    const size_t bytes =
        (size_t)(extent.d * extent.h * extent.w) * model->channels * elem_bytes(model);
    if (overlap(buf0, bytes, buf1, bytes)) return OCTNCA_EINVAL;
    // An even number of two-step launches (the rest one step each) keeps the
    // number of launches of the same parity as `steps`: the result is in buf1
    // exactly when steps is odd, whichever kernels run.
    st = run_steps(model, buf0, buf1, extent, weights, level, 0, steps, seed, threshold,
                   (hipStream_t)stream, 0, nullptr, steps / 4 * 2);
    if (st) return st;
    if (result_in_buf1) *result_in_buf1 = steps & 1;
    return OCTNCA_OK;
}

int octree_nca_readout(const octnca_model *model, const void *state, octnca_extent extent,
                       uint8_t *seg, void *stream) {
    int st = check_model(model);
    if (st) return st;
    if ((st = check_extent(model, extent))) return st;
    if (state == nullptr || seg == nullptr) return OCTNCA_EINVAL;
    return hip_status(launch_readout(dtype_of(model), state, extent.d * extent.h * extent.w,
                                     model->channels, seg, (hipStream_t)stream));
}

int octree_nca_readout_classes(const octnca_model *model, const void *state, octnca_extent extent,
                               int32_t classes, uint8_t *seg, void *stream) {
    int st = check_model(model);
    if (st) return st;
    if ((st = check_extent(model, extent))) return st;
    if (state == nullptr || seg == nullptr || classes < 2 || classes > model->channels - model->n_in)
        return OCTNCA_EINVAL;
    return hip_status(launch_readout_classes(dtype_of(model), state,
                                             extent.d * extent.h * extent.w, model->channels,
                                             classes, seg, (hipStream_t)stream));
}

int32_t octree_nca_first_level_steps(float alpha0, octnca_extent coarsest) {
    if (!(alpha0 >= 0.f) || !std::isfinite(alpha0)) return -1;
    if (coarsest.d <= 0 || coarsest.h <= 0 || coarsest.w <= 0) return -1;
    const int64_t m = std::max(coarsest.d, std::max(coarsest.h, coarsest.w));
    const double steps = std::floor((double)alpha0 * (double)m);
    if (steps > (double)INT32_MAX) return -1;
    return (int32_t)steps;
}

int octree_nca_fire_mask(uint64_t seed, int32_t level, int32_t step, octnca_extent extent,
                         float fire_rate, uint8_t *mask, void *stream) {
    uint64_t threshold;
    if (mask == nullptr || level < 0 || step < 0 || !fire_threshold(fire_rate, &threshold))
        return OCTNCA_EINVAL;
    if (extent.d <= 0 || extent.h <= 0 || extent.w <= 0 || extent.d > kMaxDim ||
        extent.h > kMaxDim || extent.w > kMaxDim || extent.d * extent.h > kMaxCells ||
        extent.d * extent.h * extent.w > kMaxCells)
        return OCTNCA_ESHAPE;
    return hip_status(launch_fire_mask(seed, (uint32_t)level, (uint32_t)step,
                                       extent.d * extent.h * extent.w, threshold, mask,
                                       (hipStream_t)stream));
}

size_t octree_nca_workspace_bytes(const octnca_model *model, octnca_extent finest, int32_t levels,
                                  const int32_t *factors, int32_t with_final_state) {
    Plan p;
    if (make_plan(model, finest, levels, factors, with_final_state != 0, &p)) return 0;
    return p.bytes;
}

int octree_nca_infer_launches(const octnca_model *model, octnca_extent finest, int32_t levels,
                              const int32_t *factors, const int32_t *steps, int32_t *launches) {
    Plan p;
    const int st = make_plan(model, finest, levels, factors, true, &p);
    if (st) return st;
    if (steps == nullptr || launches == nullptr) return OCTNCA_EINVAL;
    for (int l = 0; l < levels; ++l)
        if (steps[l] < 0) return OCTNCA_EINVAL;
    const octnca_level_weights none{};
    for (int l = 0; l < levels; ++l) {
        const StepArgs a = step_args(model, p.ext[l], &none, l, 0, 0, 0);
        const bool fused = l + 1 < levels && steps[l] >= 1 && step_fuses_upsample(a);
        launches[l] = (fused ? 1 : 0) + level_launches(a, fused_up_steps(a, fused, steps[l]),
                                                       steps[l]);
    }
    return OCTNCA_OK;
}

}  // extern "C"

namespace {

int infer_impl(const octnca_model *model, const void *image, octnca_extent finest,
               int32_t levels, const int32_t *factors, const octnca_level_weights *weights,
               const int32_t *steps, float fire_rate, uint64_t seed, void *workspace,
               size_t workspace_bytes, void *final_state, uint8_t *seg,
               void *const *level_events, void *stream, uint32_t batch, bool check_only) {
    Plan p;
    int st = make_plan(model, finest, levels, factors, final_state != nullptr, &p);
    if (st) return st;
    uint64_t threshold;
    if (image == nullptr || weights == nullptr || steps == nullptr || workspace == nullptr ||
        !fire_threshold(fire_rate, &threshold))
        return OCTNCA_EINVAL;
    for (int l = 0; l < levels; ++l)
        if (!weights_ok(&weights[l]) || steps[l] < 0) return OCTNCA_EINVAL;
    if (workspace_bytes < p.bytes) return OCTNCA_ESPACE;
    const size_t eb = elem_bytes(model);
    const size_t state_bytes = (size_t)(finest.d * finest.h * finest.w) * model->channels * eb;
    char *ws = (char *)workspace;
    if (final_state != nullptr &&
        (overlap(final_state, state_bytes, workspace, p.bytes) ||
         overlap(final_state, state_bytes, image,
                 (size_t)(finest.d * finest.h * finest.w) * model->n_in * eb)))
        return OCTNCA_EINVAL;
    if (overlap(workspace, p.bytes, image,
                (size_t)(finest.d * finest.h * finest.w) * model->n_in * eb))
        return OCTNCA_EINVAL;
    if (check_only) return OCTNCA_OK;

    // bufs[0] ends up holding the final state: the coarsest seed goes to the
    // buffer that makes the parity of (upsamples + steps) land there.
    void *bufs[2];
    bufs[0] = final_state != nullptr ? final_state : (void *)(ws + p.state_off[1]);
    bufs[1] = (void *)(ws + p.state_off[0]);
    const void *img[kMaxLevels];
    img[0] = image;
    for (int l = 1; l < levels; ++l) img[l] = ws + p.image_off[l];

    const hipStream_t s = (hipStream_t)stream;
    const Dtype dt = dtype_of(model);
    // Levels whose first step reads the next coarser state directly (upsample
    // + inject fused into the step): that transition flips no buffer.
    // Buffer flips: one per unfused upsample and one per step launch.
    bool fused[kMaxLevels] = {};
    int64_t flips = 0;
    for (int l = 0; l < levels; ++l) {
        const StepArgs a = step_args(model, p.ext[l], &weights[l], l, seed, threshold, batch);
        if (l + 1 < levels && steps[l] >= 1) fused[l] = step_fuses_upsample(a);
        const int32_t t0 = fused_up_steps(a, fused[l], steps[l]);
        flips += (l + 1 < levels ? 1 : 0) + level_launches(a, t0, steps[l]);
    }
    for (int l = 1; l < levels; ++l) {
        const int32_t *f = factors + 3 * (l - 1);
        if (launch_pool(dt, img[l - 1], ext3(p.ext[l]), (void *)img[l], f[0], f[1], f[2],
                        model->n_in, s) != hipSuccess)
            return OCTNCA_EHIP;
    }
    int cur = (int)(flips & 1);
    if (launch_upsample(dt, nullptr, ext3(p.ext[levels - 1]), 1, 1, 1, img[levels - 1], bufs[cur],
                        model->n_in, model->channels, s) != hipSuccess)
        return OCTNCA_EHIP;
    bool seg_fused = false;
    for (int l = levels - 1; l >= 0; --l) {
        const int32_t *f = factors + 3 * l;
        if (l < levels - 1 && !fused[l]) {
            if (launch_upsample(dt, bufs[cur], ext3(p.ext[l]), f[0], f[1], f[2], img[l],
                                bufs[cur ^ 1], model->n_in, model->channels, s) != hipSuccess)
                return OCTNCA_EHIP;
            cur ^= 1;
        }
        if (level_events && level_events[2 * l] &&
            hipEventRecord((hipEvent_t)level_events[2 * l], s) != hipSuccess)
            return OCTNCA_EHIP;
        // The finest level's last launch writes the readout too when it is a
        // two-step launch; otherwise the readout kernel runs at the end.
        uint8_t *seg_last = nullptr;
        if (l == 0 && seg != nullptr) {
            const StepArgs a = step_args(model, p.ext[0], &weights[0], 0, seed, threshold, batch);
            const int32_t first = fused_up_steps(a, fused[0], steps[0]);
            const int32_t rest = steps[0] - first;
            bool ok;
            if (step_pairs(a))   // the last launch runs two steps
                ok = rest % 2 == 0 && (rest > 0 || first == 2);
            else                 // the last launch is a single step after the first
                ok = rest >= 1 && step_single_fuses_readout(a);
            if (ok) seg_last = seg;
            seg_fused = ok;
        }
        int32_t t0 = 0;
        if (fused[l]) {
            // step 0 (or steps 0 and 1) from the coarse state bufs[cur] (level
            // l + 1) and image l
            StepArgs a = step_args(model, p.ext[l], &weights[l], l, seed, threshold, batch);
            t0 = fused_up_steps(a, true, steps[l]);
            if (t0 == steps[l]) a.seg = seg_last;   // this launch is the level's last
            const hipError_t err =
                t0 == 2 ? launch_step_pair_up(a, bufs[cur], (int)p.ext[l + 1].w, f[0], f[1], f[2],
                                              img[l], bufs[cur ^ 1], s)
                        : launch_step_up(a, bufs[cur], (int)p.ext[l + 1].h, (int)p.ext[l + 1].w,
                                         f[0], f[1], f[2], img[l], bufs[cur ^ 1], s);
            if (err != hipSuccess) return OCTNCA_EHIP;
            cur ^= 1;
        }
        st = run_steps(model, bufs[cur], bufs[cur ^ 1], p.ext[l], &weights[l], l, t0, steps[l],
                       seed, threshold, s, batch, seg_last);
        if (st) return st;
        cur ^= level_launches(step_args(model, p.ext[l], &weights[l], l, seed, threshold, batch),
                              t0, steps[l]) & 1;
        if (level_events && level_events[2 * l + 1] &&
            hipEventRecord((hipEvent_t)level_events[2 * l + 1], s) != hipSuccess)
            return OCTNCA_EHIP;
    }
    // cur == 0 here by construction of the seed buffer
    if (seg != nullptr && !seg_fused &&
        launch_readout(dt, bufs[cur], finest.d * finest.h * finest.w, model->channels, seg, s) !=
            hipSuccess)
        return OCTNCA_EHIP;
    return OCTNCA_OK;
}

}  // namespace

extern "C" {

int octree_nca_infer(const octnca_model *model, const void *image, octnca_extent finest,
                     int32_t levels, const int32_t *factors, const octnca_level_weights *weights,
                     const int32_t *steps, float fire_rate, uint64_t seed, void *workspace,
                     size_t workspace_bytes, void *final_state, uint8_t *seg,
                     void *const *level_events, void *stream) {
    return infer_impl(model, image, finest, levels, factors, weights, steps, fire_rate, seed,
                      workspace, workspace_bytes, final_state, seg, level_events, stream, 0,
                      false);
}

// ---------------------------------------------------------------------------
// Inference without allocation: the workspace is a static device array.
// ---------------------------------------------------------------------------

}  // extern "C"

namespace {

// Static scratch of octree_nca_infer_static: the pyramid images and the second
// state buffer of one inference.  Each device the library runs on holds its
// own copy until the process ends.  In host code `scratch` only names the
// symbol; its device address comes from hipGetSymbolAddress, per device.
__device__ __align__(256) unsigned char scratch[OCTNCA_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

// Device address of the current device's scratch, looked up once per device
// (with that device current) and kept; nullptr if the lookup failed.
void *scratch_ptr() {
    static std::mutex mu;
    static void *ptrs[kMaxDevices] = {};
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    if (ptrs[dev] == nullptr) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return nullptr;
        ptrs[dev] = p;
    }
    return ptrs[dev];
}

}  // namespace

extern "C" {

int octree_nca_infer_static(const octnca_model *model, const void *image, octnca_extent finest,
                            int32_t levels, const int32_t *factors,
                            const octnca_level_weights *weights, const int32_t *steps,
                            float fire_rate, uint64_t seed, void *final_state, uint8_t *seg,
                            void *stream) {
    Plan p;
    int st = make_plan(model, finest, levels, factors, true, &p);
    if (st) return st;
    if (final_state == nullptr) return OCTNCA_EINVAL;
    if (p.bytes > (size_t)OCTNCA_STATIC_SCRATCH_BYTES) return OCTNCA_ESPACE;
    void *ws = scratch_ptr();
    if (ws == nullptr) return OCTNCA_EHIP;
    // Nothing in the workspace needs to start at zero: every pyramid image is
    // written by the pooling and the state buffer by the seed or a step before
    // it is read.
    return infer_impl(model, image, finest, levels, factors, weights, steps, fire_rate, seed, ws,
                      (size_t)OCTNCA_STATIC_SCRATCH_BYTES, final_state, seg, nullptr, stream, 0,
                      false);
}

int octree_nca_infer_batch(const octnca_model *model, const void *images, int32_t batch,
                           octnca_extent finest, int32_t levels, const int32_t *factors,
                           const octnca_level_weights *weights, const int32_t *steps,
                           float fire_rate, uint64_t seed, void *workspace,
                           size_t workspace_bytes, void *final_states, uint8_t *segs,
                           void *stream) {
    int st = check_model(model);
    if (st) return st;
    if (images == nullptr || batch < 1) return OCTNCA_EINVAL;
    if ((st = check_extent(model, finest))) return st;
    const size_t cells = (size_t)(finest.d * finest.h * finest.w);
    const size_t eb = elem_bytes(model);
    const size_t image_bytes = cells * model->n_in * eb;
    const size_t state_bytes = cells * model->channels * eb;
    // the byte counts below (state_bytes * batch at most) stay far from 2^64
    if ((uint64_t)batch > (uint64_t(1) << 48) / state_bytes) return OCTNCA_EINVAL;
    // the batch's outputs must not overlap its inputs or the workspace
    if (final_states != nullptr &&
        (overlap(final_states, state_bytes * batch, images, image_bytes * batch) ||
         (workspace != nullptr &&
          overlap(final_states, state_bytes * batch, workspace, workspace_bytes))))
        return OCTNCA_EINVAL;
    if (segs != nullptr &&
        (overlap(segs, cells * batch, images, image_bytes * batch) ||
         (final_states != nullptr && overlap(segs, cells * batch, final_states,
                                             state_bytes * batch)) ||
         (workspace != nullptr && overlap(segs, cells * batch, workspace, workspace_bytes))))
        return OCTNCA_EINVAL;
    if (workspace != nullptr && overlap(workspace, workspace_bytes, images, image_bytes * batch))
        return OCTNCA_EINVAL;
    auto image_of = [&](int32_t b) { return (const char *)images + image_bytes * b; };
    auto state_of = [&](int32_t b) {
        return final_states ? (void *)((char *)final_states + state_bytes * b) : nullptr;
    };
    auto seg_of = [&](int32_t b) { return segs ? segs + cells * b : nullptr; };
    // every image's arguments are checked before anything is enqueued
    for (int32_t b = 0; b < batch; ++b) {
        st = infer_impl(model, image_of(b), finest, levels, factors, weights, steps, fire_rate,
                        seed, workspace, workspace_bytes, state_of(b), seg_of(b), nullptr, stream,
                        (uint32_t)b, true);
        if (st) return st;
    }
    for (int32_t b = 0; b < batch; ++b) {
        st = infer_impl(model, image_of(b), finest, levels, factors, weights, steps, fire_rate,
                        seed, workspace, workspace_bytes, state_of(b), seg_of(b), nullptr, stream,
                        (uint32_t)b, false);
        if (st) return st;
    }
    return OCTNCA_OK;
}

// ---------------------------------------------------------------------------
// Training (fp32 states): backward of a step, of the upsample, a readout MSE
// and the whole training step (Sec. 3.2 efficient training; supplement S7).
// ---------------------------------------------------------------------------

size_t octree_nca_step_backward_workspace_bytes(const octnca_model *model, octnca_extent extent) {
    if (check_model(model) || check_extent(model, extent)) return 0;
    return step_backward_workspace_floats(model->ndim, model->channels, model->hidden,
                                          ext3(extent)) *
           sizeof(float);
}

int octree_nca_step_backward(const octnca_model *model, const void *state, const void *grad_out,
                             octnca_extent extent, const octnca_level_weights *weights,
                             int32_t level, int32_t step, float fire_rate, uint64_t seed,
                             void *grad_in, const octnca_level_grads *grads, void *workspace,
                             size_t workspace_bytes, void *stream) {
    int st = check_model(model);
    if (st) return st;
    if (model->state_dtype != OCTNCA_F32) return OCTNCA_EUNSUPPORTED;
    if ((st = check_extent(model, extent))) return st;
    uint64_t threshold;
    if (state == nullptr || grad_out == nullptr || grad_in == nullptr || workspace == nullptr ||
        !weights_ok(weights) || grads == nullptr || !grads->conv_w || !grads->conv_b ||
        !grads->w1 || !grads->b1 || !grads->w2 || level < 0 || step < 0 ||
        !fire_threshold(fire_rate, &threshold))
        return OCTNCA_EINVAL;
    const size_t need = octree_nca_step_backward_workspace_bytes(model, extent);
    if (workspace_bytes < need) return OCTNCA_ESPACE;
    const size_t bytes = (size_t)(extent.d * extent.h * extent.w) * model->channels * sizeof(float);
    if (overlap(grad_in, bytes, state, bytes) || overlap(workspace, need, state, bytes) ||
        overlap(workspace, need, grad_in, bytes) || overlap(workspace, need, grad_out, bytes))
        return OCTNCA_EINVAL;
    if (grad_in != grad_out && overlap(grad_in, bytes, grad_out, bytes)) return OCTNCA_EINVAL;
    StepArgs a = step_args(model, extent, weights, level, seed, threshold, 0);
    a.step = (uint32_t)step;
    const LevelGradsDev g{grads->conv_w, grads->conv_b, grads->w1, grads->b1, grads->w2};
    return hip_status(launch_step_backward(a, (const float *)state, (const float *)grad_out,
                                           (float *)grad_in, g, (float *)workspace,
                                           (hipStream_t)stream));
}

int octree_nca_upsample_backward(const octnca_model *model, const void *grad_fine,
                                 octnca_extent coarse, const int32_t *factor, void *grad_coarse,
                                 void *stream) {
    int st = check_model(model);
    if (st) return st;
    if (model->state_dtype != OCTNCA_F32) return OCTNCA_EUNSUPPORTED;
    if (grad_fine == nullptr || grad_coarse == nullptr || factor == nullptr) return OCTNCA_EINVAL;
    if ((st = check_extent(model, coarse)) || (st = check_factor(model, factor))) return st;
    const octnca_extent fine{coarse.d * factor[0], coarse.h * factor[1], coarse.w * factor[2]};
    if ((st = check_extent(model, fine))) return st;
    if (overlap(grad_coarse, (size_t)(coarse.d * coarse.h * coarse.w) * model->channels * 4,
                grad_fine, (size_t)(fine.d * fine.h * fine.w) * model->channels * 4))
        return OCTNCA_EINVAL;
    return hip_status(launch_upsample_adjoint((const float *)grad_fine, ext3(coarse), factor[0],
                                              factor[1], factor[2], model->n_in, model->channels,
                                              (float *)grad_coarse, (hipStream_t)stream));
}

size_t octree_nca_readout_mse_workspace_bytes(octnca_extent extent) {
    if (extent.d <= 0 || extent.h <= 0 || extent.w <= 0) return 0;
    return mse_workspace_doubles(extent.d * extent.h * extent.w) * sizeof(double);
}

int octree_nca_readout_mse(const octnca_model *model, const void *state, const float *target,
                           octnca_extent extent, void *grad, double *loss, void *workspace,
                           size_t workspace_bytes, void *stream) {
    int st = check_model(model);
    if (st) return st;
    if (model->state_dtype != OCTNCA_F32) return OCTNCA_EUNSUPPORTED;
    if ((st = check_extent(model, extent))) return st;
    if (state == nullptr || target == nullptr || grad == nullptr || loss == nullptr ||
        workspace == nullptr)
        return OCTNCA_EINVAL;
    const int64_t cells = extent.d * extent.h * extent.w;
    if (workspace_bytes < octree_nca_readout_mse_workspace_bytes(extent)) return OCTNCA_ESPACE;
    const size_t bytes = (size_t)cells * model->channels * sizeof(float);
    if (overlap(grad, bytes, state, bytes) || overlap(grad, bytes, target, (size_t)cells * 8) ||
        overlap(workspace, workspace_bytes, grad, bytes))
        return OCTNCA_EINVAL;
    return hip_status(launch_readout_mse((const float *)state, target, cells, model->channels,
                                         (float *)grad, loss, (double *)workspace,
                                         (hipStream_t)stream));
}

}  // extern "C"

namespace {

// Workspace of a training step: pyramid images 1..L-1, the states of every
// level (before each step and after the last), two finest-size gradient
// buffers, the level-backward workspace (finest size) and the loss partials.
struct TrainPlan {
    octnca_extent ext[kMaxLevels];
    size_t image_off[kMaxLevels];
    size_t tape_off[kMaxLevels];    // state t of level l at tape_off[l] + t * state bytes of l
    size_t grad_off[2], bwd_off, mse_off, bytes;
};

int make_train_plan(const octnca_model *m, octnca_extent finest, int32_t levels,
                    const int32_t *factors, const int32_t *steps, TrainPlan *p) {
    int st = check_model(m);
    if (st) return st;
    if (m->state_dtype != OCTNCA_F32) return OCTNCA_EUNSUPPORTED;
    if ((st = level_extents(m, finest, levels, factors, p->ext))) return st;
    if (steps == nullptr) return OCTNCA_EINVAL;
    for (int l = 0; l < levels; ++l)
        if (steps[l] < 0) return OCTNCA_EINVAL;
    size_t off = 0;
    p->image_off[0] = 0;
    for (int l = 1; l < levels; ++l) {
        p->image_off[l] = off;
        off += align_up((size_t)(p->ext[l].d * p->ext[l].h * p->ext[l].w) * m->n_in * 4);
    }
    for (int l = 0; l < levels; ++l) {
        p->tape_off[l] = off;
        const size_t sb = (size_t)(p->ext[l].d * p->ext[l].h * p->ext[l].w) * m->channels * 4;
        off += align_up(sb * ((size_t)steps[l] + 1));
    }
    const int64_t cells = finest.d * finest.h * finest.w;
    const size_t gb = align_up((size_t)cells * m->channels * 4);
    p->grad_off[0] = off;
    off += gb;
    p->grad_off[1] = off;
    off += gb;
    p->bwd_off = off;
    // the finest level needs the most (every level's extent is at most the finest's)
    off += align_up(level_backward_workspace_floats(m->ndim, m->channels, m->hidden, ext3(finest)) *
                    4);
    p->mse_off = off;
    off += align_up(mse_workspace_doubles(cells) * sizeof(double));
    p->bytes = off;
    return OCTNCA_OK;
}

// Forward step of a training pass: split-bf16 MLP operands on the
// matrix-core kernel for C = 16, H = 64 (each product to about 2^-16, three
// bf16 products instead of one fp32 one: a fifth of the matrix-core time),
// fp32 FMAs on the vector kernel otherwise.
hipError_t train_forward_step(const StepArgs &a, const void *src, void *dst, hipStream_t s) {
    if (a.channels == kC && a.hidden == kH)
        return launch_step_mfma(a, MfmaMlp::Bf16x3, Layout2d::Auto, src, dst, s);
    return launch_step_valu(a, src, dst, s);
}

}  // namespace

extern "C" {

size_t octree_nca_train_workspace_bytes(const octnca_model *model, octnca_extent finest,
                                        int32_t levels, const int32_t *factors,
                                        const int32_t *steps) {
    TrainPlan p;
    return make_train_plan(model, finest, levels, factors, steps, &p) ? 0 : p.bytes;
}

int octree_nca_train_step(const octnca_model *model, const void *image, octnca_extent finest,
                          int32_t levels, const int32_t *factors,
                          const octnca_level_weights *weights, const int32_t *steps,
                          float fire_rate, uint64_t seed, const float *target, void *workspace,
                          size_t workspace_bytes, const octnca_level_grads *grads, double *loss,
                          void *final_state, void *stream) {
    TrainPlan p;
    int st = make_train_plan(model, finest, levels, factors, steps, &p);
    if (st) return st;
    uint64_t threshold;
    if (image == nullptr || weights == nullptr || target == nullptr || workspace == nullptr ||
        grads == nullptr || loss == nullptr || !fire_threshold(fire_rate, &threshold))
        return OCTNCA_EINVAL;
    for (int l = 0; l < levels; ++l)
        if (!weights_ok(&weights[l]) || !grads[l].conv_w || !grads[l].conv_b || !grads[l].w1 ||
            !grads[l].b1 || !grads[l].w2)
            return OCTNCA_EINVAL;
    if (workspace_bytes < p.bytes) return OCTNCA_ESPACE;
    const int64_t cells = finest.d * finest.h * finest.w;
    const size_t state_bytes = (size_t)cells * model->channels * 4;
    if (overlap(workspace, p.bytes, image, (size_t)cells * model->n_in * 4) ||
        overlap(workspace, p.bytes, target, (size_t)cells * 8) ||
        (final_state && overlap(workspace, p.bytes, final_state, state_bytes)))
        return OCTNCA_EINVAL;

    const hipStream_t s = (hipStream_t)stream;
    char *ws = (char *)workspace;
    auto img = [&](int l) { return l == 0 ? image : (const void *)(ws + p.image_off[l]); };
    auto cells_of = [&](int l) { return p.ext[l].d * p.ext[l].h * p.ext[l].w; };
    auto tape = [&](int l, int t) {
        return (float *)(ws + p.tape_off[l]) + (size_t)t * cells_of(l) * model->channels;
    };
    auto ok = [](hipError_t e) { return e == hipSuccess; };

    // forward, keeping every state
    for (int l = 1; l < levels; ++l) {
        const int32_t *f = factors + 3 * (l - 1);
        if (!ok(launch_pool(Dtype::F32, img(l - 1), ext3(p.ext[l]), ws + p.image_off[l], f[0],
                            f[1], f[2], model->n_in, s)))
            return OCTNCA_EHIP;
    }
    for (int l = levels - 1; l >= 0; --l) {
        const hipError_t e =
            l == levels - 1
                ? launch_upsample(Dtype::F32, nullptr, ext3(p.ext[l]), 1, 1, 1, img(l), tape(l, 0),
                                  model->n_in, model->channels, s)
                : launch_upsample(Dtype::F32, tape(l + 1, steps[l + 1]), ext3(p.ext[l]),
                                  factors[3 * l], factors[3 * l + 1], factors[3 * l + 2], img(l),
                                  tape(l, 0), model->n_in, model->channels, s);
        if (!ok(e)) return OCTNCA_EHIP;
        StepArgs a = step_args(model, p.ext[l], &weights[l], l, seed, threshold, 0);
        for (int t = 0; t < steps[l]; ++t) {
            a.step = (uint32_t)t;
            if (!ok(train_forward_step(a, tape(l, t), tape(l, t + 1), s))) return OCTNCA_EHIP;
        }
    }
    const float *final_fine = tape(0, steps[0]);
    float *g = (float *)(ws + p.grad_off[0]);
    float *g_other = (float *)(ws + p.grad_off[1]);
    if (!ok(launch_readout_mse(final_fine, target, cells, model->channels, g, loss,
                               (double *)(ws + p.mse_off), s)))
        return OCTNCA_EHIP;
    if (final_state &&
        !ok(hipMemcpyAsync(final_state, final_fine, state_bytes, hipMemcpyDeviceToDevice, s)))
        return OCTNCA_EHIP;

    // backward, finest level first; a level's backward writes its weight
    // gradients, so only levels without steps are cleared here
    const int taps = model->ndim == 3 ? 27 : 9;
    for (int l = 0; l < levels; ++l) {
        if (steps[l] > 0) continue;
        const int64_t c = model->channels, h = model->hidden;
        const octnca_level_grads &gr = grads[l];
        if (!ok(launch_fill_zero(gr.conv_w, c * taps, s)) || !ok(launch_fill_zero(gr.conv_b, c, s)) ||
            !ok(launch_fill_zero(gr.w1, h * 2 * c, s)) || !ok(launch_fill_zero(gr.b1, h, s)) ||
            !ok(launch_fill_zero(gr.w2, c * h, s)))
            return OCTNCA_EHIP;
    }
    for (int l = 0; l < levels; ++l) {
        StepArgs a = step_args(model, p.ext[l], &weights[l], l, seed, threshold, 0);
        const LevelGradsDev gd{grads[l].conv_w, grads[l].conv_b, grads[l].w1, grads[l].b1,
                               grads[l].w2};
        // all steps of the level, last first (dL/dS of its first state lands
        // in the other gradient buffer)
        if (steps[l] > 0) {
            if (!ok(launch_level_backward(a, steps[l], tape(l, 0), g, g_other, gd,
                                          (float *)(ws + p.bwd_off), s)))
                return OCTNCA_EHIP;
            std::swap(g, g_other);
        }
        if (l + 1 < levels) {
            if (!ok(launch_upsample_adjoint(g, ext3(p.ext[l + 1]), factors[3 * l],
                                            factors[3 * l + 1], factors[3 * l + 2], model->n_in,
                                            model->channels, g_other, s)))
                return OCTNCA_EHIP;
            std::swap(g, g_other);
        }
    }
    return OCTNCA_OK;
}

}  // extern "C"

namespace octnca {
// The step kernel comes with the arguments (StepArgs::kc, filled from the
// caller's octnca_model); nothing here reads the environment.
hipError_t launch_step(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (a.kc.valu) return launch_step_valu(a, src, dst, stream);
    // the specialised matrix-core kernels serve C = 16, H = 64 and the 2D
    // fp32 row layout of C = 12, H = 48; the other steps of the ablation's
    // sizes run on the generic matrix-core kernel
    if (!step_mfma_serves(a, a.kc.layout)) return launch_step_gen(a, src, dst, stream);
    return launch_step_mfma(a, a.kc.mlp, a.kc.layout, src, dst, stream);
}

bool step_single_fuses_readout(const StepArgs &a) {
    return !a.kc.valu && step_mfma_single_readout(a, a.kc.mlp);
}

bool step_pairs(const StepArgs &a) {
    return !a.kc.valu && a.kc.pairs && step_mfma_pairs(a, a.kc.mlp, a.kc.layout);
}

hipError_t launch_step_pair(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (!step_pairs(a)) return hipErrorInvalidValue;
    return launch_step2_mfma(a, a.kc.mlp, a.kc.layout, src, dst, stream);
}

hipError_t launch_step_pair_up(const StepArgs &a, const void *coarse, int coarse_w, int fz,
                               int fy, int fx, const void *img, void *dst, hipStream_t stream) {
    if (fz != 1 || !step_pairs(a) || !step_fuses_upsample(a)) return hipErrorInvalidValue;
    return launch_step2_mfma_up(a, a.kc.mlp, a.kc.layout, coarse, coarse_w, fy, fx, img, dst,
                                stream);
}

bool step_fuses_upsample(const StepArgs &a) {
    return !a.kc.valu && step_mfma_fuses_upsample(a, a.kc.mlp, a.kc.layout);
}

hipError_t launch_step_up(const StepArgs &a, const void *coarse, int coarse_h, int coarse_w,
                          int fz, int fy, int fx, const void *img, void *dst,
                          hipStream_t stream) {
    if (!step_fuses_upsample(a)) return hipErrorInvalidValue;
    return launch_step_mfma_up(a, a.kc.layout, coarse, coarse_h, coarse_w, fz, fy, fx, img, dst,
                               stream);
}
}  // namespace octnca
