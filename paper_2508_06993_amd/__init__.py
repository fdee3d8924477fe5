"""Python binding of liboctree_nca.so, the MI355X (gfx950) OctreeNCA inference
library (arXiv 2508.06993).

Argument marshalling only: every function here checks and converts its
arguments, then calls the C entry point of the same name (include/octree_nca.h).
All arithmetic runs in the library's HIP kernels.  PyTorch supplies device
memory and the current stream.  There is no CPU fallback: if the library is
missing, every call raises ``OctreeNCAError``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

from .build import LIB_PATH

__all__ = [
    "OctreeNCAError", "Model", "lib", "library_path", "level_weights_struct",
    "octree_nca_build_pyramid", "octree_nca_upsample", "octree_nca_run_level",
    "octree_nca_readout", "octree_nca_readout_classes", "octree_nca_workspace_bytes",
    "octree_nca_infer", "octree_nca_infer_batch", "octree_nca_infer_launches",
    "octree_nca_infer_static", "OCTNCA_STATIC_SCRATCH_BYTES",
    "octree_nca_first_level_steps",
    "octree_nca_fire_mask", "octree_nca_strerror", "octree_nca_abi_version",
    "octree_nca_step_backward_workspace_bytes", "octree_nca_step_backward",
    "octree_nca_upsample_backward", "octree_nca_readout_mse_workspace_bytes",
    "octree_nca_readout_mse", "octree_nca_train_workspace_bytes", "octree_nca_train_step",
    "level_grads_struct", "EXPORTED_SYMBOLS", "OCTNCA_OK", "OCTNCA_EINVAL",
    "OCTNCA_EUNSUPPORTED", "OCTNCA_ESHAPE",
    "OCTNCA_EHIP", "OCTNCA_ESPACE", "OCTNCA_F32", "OCTNCA_F16", "KERNEL_NAMES", "kernel_fields",
]

OCTNCA_OK, OCTNCA_EINVAL, OCTNCA_EUNSUPPORTED, OCTNCA_ESHAPE, OCTNCA_EHIP, OCTNCA_ESPACE = \
    0, -1, -2, -3, -4, -5
OCTNCA_F32, OCTNCA_F16 = 0, 1
(OCTNCA_MLP_AUTO, OCTNCA_MLP_F32, OCTNCA_MLP_BF16X3, OCTNCA_MLP_F16, OCTNCA_MLP_F16S,
 OCTNCA_MLP_VALU) = range(6)
OCTNCA_LAYOUT_AUTO, OCTNCA_LAYOUT_ROWS, OCTNCA_LAYOUT_TILES = range(3)
OCTNCA_STATIC_SCRATCH_BYTES = 64 << 20   # octree_nca_infer_static's device array

# Step-kernel names accepted by Model(kernel=...): a comma-separated list of
# these, each setting one field of the C model description (octnca_model).
KERNEL_NAMES = {
    "mfma": {},                                   # the library's default
    "mfma_f32": {"mlp": OCTNCA_MLP_F32},
    "mfma_bf16x3": {"mlp": OCTNCA_MLP_BF16X3},
    "mfma_f16": {"mlp": OCTNCA_MLP_F16},
    "mfma_f16s": {"mlp": OCTNCA_MLP_F16S},
    "valu": {"mlp": OCTNCA_MLP_VALU},
    "mfma_rows": {"layout2d": OCTNCA_LAYOUT_ROWS},
    "mfma_tiles": {"layout2d": OCTNCA_LAYOUT_TILES},
    "mfma_1step": {"steps_per_launch": 1},
}


def kernel_fields(kernel: str) -> dict:
    """octnca_model step-kernel fields (mlp, layout2d, steps_per_launch) of a
    name such as "mfma_rows,mfma_1step"."""
    out = {"mlp": OCTNCA_MLP_AUTO, "layout2d": OCTNCA_LAYOUT_AUTO, "steps_per_launch": 0}
    for name in kernel.split(","):
        if name not in KERNEL_NAMES:
            raise ValueError(f"unknown step kernel {name!r}; known: {sorted(KERNEL_NAMES)}")
        out.update(KERNEL_NAMES[name])
    return out

EXPORTED_SYMBOLS = (
    "octree_nca_build_pyramid", "octree_nca_upsample", "octree_nca_run_level",
    "octree_nca_readout", "octree_nca_readout_classes", "octree_nca_workspace_bytes",
    "octree_nca_infer", "octree_nca_infer_batch", "octree_nca_infer_launches",
    "octree_nca_infer_static",
    "octree_nca_first_level_steps",
    "octree_nca_fire_mask", "octree_nca_strerror", "octree_nca_abi_version",
    "octree_nca_step_backward_workspace_bytes", "octree_nca_step_backward",
    "octree_nca_upsample_backward", "octree_nca_readout_mse_workspace_bytes",
    "octree_nca_readout_mse", "octree_nca_train_workspace_bytes", "octree_nca_train_step",
)


class OctreeNCAError(RuntimeError):
    def __init__(self, msg, status=None):
        super().__init__(msg)
        self.status = status


class _Model(ctypes.Structure):
    _fields_ = [("ndim", ctypes.c_int32), ("channels", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("n_in", ctypes.c_int32),
                ("state_dtype", ctypes.c_int32), ("mlp", ctypes.c_int32),
                ("layout2d", ctypes.c_int32), ("steps_per_launch", ctypes.c_int32)]


class _Extent(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int64), ("h", ctypes.c_int64), ("w", ctypes.c_int64)]


class _LevelWeights(ctypes.Structure):
    _fields_ = [("conv_w", ctypes.c_void_p), ("conv_b", ctypes.c_void_p),
                ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p)]


class _LevelGrads(ctypes.Structure):
    _fields_ = [("conv_w", ctypes.c_void_p), ("conv_b", ctypes.c_void_p),
                ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p)]


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_SIGS = {
    "octree_nca_build_pyramid": (_I32, [ctypes.POINTER(_Model), _P, _Extent, _I32,
                                        ctypes.POINTER(_I32), ctypes.POINTER(_P), _P]),
    "octree_nca_upsample": (_I32, [ctypes.POINTER(_Model), _P, _Extent, ctypes.POINTER(_I32),
                                   _P, _P, _P]),
    "octree_nca_run_level": (_I32, [ctypes.POINTER(_Model), _P, _P, _Extent,
                                    ctypes.POINTER(_LevelWeights), _I32, _I32, ctypes.c_float,
                                    ctypes.c_uint64, ctypes.POINTER(_I32), _P]),
    "octree_nca_readout": (_I32, [ctypes.POINTER(_Model), _P, _Extent, _P, _P]),
    "octree_nca_readout_classes": (_I32, [ctypes.POINTER(_Model), _P, _Extent, _I32, _P, _P]),
    "octree_nca_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(_Model), _Extent, _I32,
                                                     ctypes.POINTER(_I32), _I32]),
    "octree_nca_infer_launches": (_I32, [ctypes.POINTER(_Model), _Extent, _I32,
                                         ctypes.POINTER(_I32), ctypes.POINTER(_I32),
                                         ctypes.POINTER(_I32)]),
    "octree_nca_infer": (_I32, [ctypes.POINTER(_Model), _P, _Extent, _I32, ctypes.POINTER(_I32),
                                ctypes.POINTER(_LevelWeights), ctypes.POINTER(_I32),
                                ctypes.c_float, ctypes.c_uint64, _P, ctypes.c_size_t, _P, _P,
                                ctypes.POINTER(_P), _P]),
    "octree_nca_infer_static": (_I32, [ctypes.POINTER(_Model), _P, _Extent, _I32,
                                       ctypes.POINTER(_I32), ctypes.POINTER(_LevelWeights),
                                       ctypes.POINTER(_I32), ctypes.c_float, ctypes.c_uint64, _P,
                                       _P, _P]),
    "octree_nca_infer_batch": (_I32, [ctypes.POINTER(_Model), _P, _I32, _Extent, _I32,
                                      ctypes.POINTER(_I32), ctypes.POINTER(_LevelWeights),
                                      ctypes.POINTER(_I32), ctypes.c_float, ctypes.c_uint64, _P,
                                      ctypes.c_size_t, _P, _P, _P]),
    "octree_nca_fire_mask": (_I32, [ctypes.c_uint64, _I32, _I32, _Extent, ctypes.c_float, _P,
                                    _P]),
    "octree_nca_first_level_steps": (_I32, [ctypes.c_float, _Extent]),
    "octree_nca_step_backward_workspace_bytes": (ctypes.c_size_t,
                                                 [ctypes.POINTER(_Model), _Extent]),
    "octree_nca_step_backward": (_I32, [ctypes.POINTER(_Model), _P, _P, _Extent,
                                        ctypes.POINTER(_LevelWeights), _I32, _I32,
                                        ctypes.c_float, ctypes.c_uint64, _P,
                                        ctypes.POINTER(_LevelGrads), _P, ctypes.c_size_t, _P]),
    "octree_nca_upsample_backward": (_I32, [ctypes.POINTER(_Model), _P, _Extent,
                                            ctypes.POINTER(_I32), _P, _P]),
    "octree_nca_readout_mse_workspace_bytes": (ctypes.c_size_t, [_Extent]),
    "octree_nca_readout_mse": (_I32, [ctypes.POINTER(_Model), _P, _P, _Extent, _P, _P, _P,
                                      ctypes.c_size_t, _P]),
    "octree_nca_train_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(_Model), _Extent, _I32,
                                                           ctypes.POINTER(_I32),
                                                           ctypes.POINTER(_I32)]),
    "octree_nca_train_step": (_I32, [ctypes.POINTER(_Model), _P, _Extent, _I32,
                                     ctypes.POINTER(_I32), ctypes.POINTER(_LevelWeights),
                                     ctypes.POINTER(_I32), ctypes.c_float, ctypes.c_uint64, _P,
                                     _P, ctypes.c_size_t, ctypes.POINTER(_LevelGrads), _P, _P,
                                     _P]),
    "octree_nca_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "octree_nca_abi_version": (ctypes.c_int, []),
}

_lib = None


def library_path() -> str:
    return os.environ.get("OCTREE_NCA_LIB", LIB_PATH)


def lib():
    """The loaded library (loaded on first use).  Raises if it is not built."""
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise OctreeNCAError(
                f"HIP library {path} is not built; run `python -m paper_2508_06993_amd.build` "
                "(there is no CPU fallback)")
        handle = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Model:
    ndim: int
    n_in: int
    dtype: str = "f32"          # storage of states and images: "f32" or "f16"
    channels: int = 16
    hidden: int = 64
    kernel: str = "mfma"        # step kernel: names of KERNEL_NAMES, comma-separated

    @property
    def torch_dtype(self):
        return torch.float16 if self.dtype == "f16" else torch.float32

    def struct(self) -> _Model:
        k = kernel_fields(self.kernel)
        return _Model(self.ndim, self.channels, self.hidden, self.n_in,
                      OCTNCA_F16 if self.dtype == "f16" else OCTNCA_F32, k["mlp"],
                      k["layout2d"], k["steps_per_launch"])


def _extent(ext: Sequence[int]) -> _Extent:
    d, h, w = (int(v) for v in ext)
    return _Extent(d, h, w)


def _ptr(t: Optional[torch.Tensor], dtype=None, name="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor")
    if t.device.type != "cuda":
        raise OctreeNCAError(f"{name}: must be a device (cuda) tensor")
    if not t.is_contiguous():
        raise OctreeNCAError(f"{name}: must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise OctreeNCAError(f"{name}: expected {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _factors(factors: Sequence[Sequence[int]]):
    flat = [int(v) for f in factors for v in f]
    arr = (_I32 * max(1, len(flat)))(*flat)
    return arr


def _check(status: int, what: str):
    if status != OCTNCA_OK:
        msg = lib().octree_nca_strerror(status).decode()
        raise OctreeNCAError(f"{what} failed: {msg} ({status})", status)


def level_weights_struct(w) -> _LevelWeights:
    """``w`` has device fp32 tensors conv_w [C][taps], conv_b [C], w1 [H][2C],
    b1 [H], w2 [C][H] (attributes or a dict)."""
    get = (lambda k: w[k]) if isinstance(w, dict) else (lambda k: getattr(w, k))
    return _LevelWeights(*(_ptr(get(k), torch.float32, k) for k in
                           ("conv_w", "conv_b", "w1", "b1", "w2")))


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def octree_nca_abi_version() -> int:
    return lib().octree_nca_abi_version()


def octree_nca_strerror(status: int) -> str:
    return lib().octree_nca_strerror(status).decode()


def octree_nca_build_pyramid(model: Model, image: torch.Tensor, factors, level_images,
                             stream=None) -> None:
    levels = len(level_images) + 1
    d, h, w = image.shape[:3]
    imgs = (_P * max(1, levels - 1))(*[_ptr(t, model.torch_dtype, "level image")
                                       for t in level_images])
    st = lib().octree_nca_build_pyramid(ctypes.byref(model.struct()),
                                        _ptr(image, model.torch_dtype, "image"),
                                        _extent((d, h, w)), levels, _factors(factors), imgs,
                                        _stream(stream))
    _check(st, "octree_nca_build_pyramid")


def octree_nca_upsample(model: Model, coarse_state: torch.Tensor, factor, fine_image,
                        fine_state, stream=None) -> None:
    d, h, w = coarse_state.shape[:3]
    st = lib().octree_nca_upsample(ctypes.byref(model.struct()),
                                   _ptr(coarse_state, model.torch_dtype, "coarse_state"),
                                   _extent((d, h, w)), (_I32 * 3)(*[int(v) for v in factor]),
                                   _ptr(fine_image, model.torch_dtype, "fine_image"),
                                   _ptr(fine_state, model.torch_dtype, "fine_state"),
                                   _stream(stream))
    _check(st, "octree_nca_upsample")


def octree_nca_run_level(model: Model, buf0, buf1, weights, level: int, steps: int,
                         fire_rate: float, seed: int, stream=None) -> int:
    """Returns 1 if the final state is in buf1, 0 if in buf0 (steps % 2)."""
    d, h, w = buf0.shape[:3]
    res = _I32(0)
    st = lib().octree_nca_run_level(ctypes.byref(model.struct()),
                                    _ptr(buf0, model.torch_dtype, "buf0"),
                                    _ptr(buf1, model.torch_dtype, "buf1"), _extent((d, h, w)),
                                    ctypes.byref(level_weights_struct(weights)), int(level),
                                    int(steps), float(fire_rate), int(seed), ctypes.byref(res),
                                    _stream(stream))
    _check(st, "octree_nca_run_level")
    return int(res.value)


def octree_nca_readout(model: Model, state, seg, stream=None) -> None:
    d, h, w = state.shape[:3]
    st = lib().octree_nca_readout(ctypes.byref(model.struct()),
                                  _ptr(state, model.torch_dtype, "state"), _extent((d, h, w)),
                                  _ptr(seg, torch.uint8, "seg"), _stream(stream))
    _check(st, "octree_nca_readout")


def octree_nca_readout_classes(model: Model, state, classes: int, seg, stream=None) -> None:
    d, h, w = state.shape[:3]
    st = lib().octree_nca_readout_classes(ctypes.byref(model.struct()),
                                          _ptr(state, model.torch_dtype, "state"),
                                          _extent((d, h, w)), int(classes),
                                          _ptr(seg, torch.uint8, "seg"), _stream(stream))
    _check(st, "octree_nca_readout_classes")


def octree_nca_workspace_bytes(model: Model, finest, factors, with_final_state=True) -> int:
    levels = len(factors) + 1
    n = lib().octree_nca_workspace_bytes(ctypes.byref(model.struct()), _extent(finest), levels,
                                         _factors(factors), 1 if with_final_state else 0)
    if n == 0:
        raise OctreeNCAError("octree_nca_workspace_bytes: invalid arguments", OCTNCA_EINVAL)
    return int(n)


def octree_nca_infer_launches(model: Model, finest, factors, steps) -> list:
    """Step-kernel launches per level (index 0 = finest) that octree_nca_infer
    enqueues with the model's step kernel."""
    levels = len(factors) + 1
    out = (_I32 * levels)()
    st = lib().octree_nca_infer_launches(ctypes.byref(model.struct()), _extent(finest), levels,
                                         _factors(factors), (_I32 * levels)(*steps), out)
    _check(st, "octree_nca_infer_launches")
    return [int(v) for v in out]


def octree_nca_infer(model: Model, image, factors, weights, steps, fire_rate: float, seed: int,
                     workspace, final_state=None, seg=None, level_events=None,
                     stream=None) -> None:
    levels = len(steps)
    d, h, w = image.shape[:3]
    ws = (_LevelWeights * levels)(*[level_weights_struct(x) for x in weights])
    ev = None
    if level_events is not None:
        ev = (_P * (2 * levels))(*[ctypes.c_void_p(int(e)) if e else None
                                   for e in level_events])
    st = lib().octree_nca_infer(ctypes.byref(model.struct()),
                                _ptr(image, model.torch_dtype, "image"), _extent((d, h, w)),
                                levels, _factors(factors), ws,
                                (_I32 * levels)(*[int(s) for s in steps]), float(fire_rate),
                                int(seed), _ptr(workspace, torch.uint8, "workspace"),
                                workspace.numel(),
                                _ptr(final_state, model.torch_dtype, "final_state"),
                                _ptr(seg, torch.uint8, "seg"), ev, _stream(stream))
    _check(st, "octree_nca_infer")


def octree_nca_infer_static(model: Model, image, factors, weights, steps, fire_rate: float,
                            seed: int, final_state, seg=None, stream=None) -> None:
    """octree_nca_infer with the library's static device workspace (no
    allocation in the call); final_state is required.  Calls on one device
    share that workspace and must not overlap."""
    levels = len(steps)
    d, h, w = image.shape[:3]
    ws = (_LevelWeights * levels)(*[level_weights_struct(x) for x in weights])
    st = lib().octree_nca_infer_static(ctypes.byref(model.struct()),
                                       _ptr(image, model.torch_dtype, "image"),
                                       _extent((d, h, w)), levels, _factors(factors), ws,
                                       (_I32 * levels)(*[int(s) for s in steps]),
                                       float(fire_rate), int(seed),
                                       _ptr(final_state, model.torch_dtype, "final_state"),
                                       _ptr(seg, torch.uint8, "seg"), _stream(stream))
    _check(st, "octree_nca_infer_static")


def octree_nca_infer_batch(model: Model, images, factors, weights, steps, fire_rate: float,
                           seed: int, workspace, final_states=None, segs=None,
                           stream=None) -> None:
    """images: [batch][d][h][w][n_in]; final_states [batch][d][h][w][C] or None;
    segs [batch][d][h][w] uint8 or None."""
    levels = len(steps)
    batch, d, h, w = images.shape[:4]
    ws = (_LevelWeights * levels)(*[level_weights_struct(x) for x in weights])
    st = lib().octree_nca_infer_batch(ctypes.byref(model.struct()),
                                      _ptr(images, model.torch_dtype, "images"), int(batch),
                                      _extent((d, h, w)), levels, _factors(factors), ws,
                                      (_I32 * levels)(*[int(s) for s in steps]),
                                      float(fire_rate), int(seed),
                                      _ptr(workspace, torch.uint8, "workspace"),
                                      workspace.numel(),
                                      _ptr(final_states, model.torch_dtype, "final_states"),
                                      _ptr(segs, torch.uint8, "segs"), _stream(stream))
    _check(st, "octree_nca_infer_batch")


def octree_nca_first_level_steps(alpha0: float, coarsest) -> int:
    """Steps of the coarsest level under the alpha0 * max(H, W, D) rule."""
    n = lib().octree_nca_first_level_steps(float(alpha0), _extent(coarsest))
    if n < 0:
        raise OctreeNCAError("octree_nca_first_level_steps: invalid arguments", OCTNCA_EINVAL)
    return int(n)


def octree_nca_fire_mask(seed: int, level: int, step: int, extent, fire_rate: float, mask,
                         stream=None) -> None:
    st = lib().octree_nca_fire_mask(int(seed), int(level), int(step), _extent(extent),
                                    float(fire_rate), _ptr(mask, torch.uint8, "mask"),
                                    _stream(stream))
    _check(st, "octree_nca_fire_mask")


# ---------------------------------------------------------------------------
# training gradients (fp32 states)
# ---------------------------------------------------------------------------

def level_grads_struct(g) -> _LevelGrads:
    """``g`` has device fp32 tensors conv_w, conv_b, w1, b1, w2 shaped like the
    weights (attributes or a dict); the library writes into them."""
    get = (lambda k: g[k]) if isinstance(g, dict) else (lambda k: getattr(g, k))
    return _LevelGrads(*(_ptr(get(k), torch.float32, k) for k in
                         ("conv_w", "conv_b", "w1", "b1", "w2")))


def octree_nca_step_backward_workspace_bytes(model: Model, extent) -> int:
    return int(lib().octree_nca_step_backward_workspace_bytes(ctypes.byref(model.struct()),
                                                              _extent(extent)))


def octree_nca_step_backward(model: Model, state, grad_out, weights, level: int, step: int,
                             fire_rate: float, seed: int, grad_in, grads, workspace,
                             stream=None) -> None:
    """Backward of one step: grad_in <- dL/dS, grads += the weight gradients."""
    d, h, w = state.shape[:3]
    st = lib().octree_nca_step_backward(
        ctypes.byref(model.struct()), _ptr(state, torch.float32, "state"),
        _ptr(grad_out, torch.float32, "grad_out"), _extent((d, h, w)),
        ctypes.byref(level_weights_struct(weights)), int(level), int(step), float(fire_rate),
        int(seed), _ptr(grad_in, torch.float32, "grad_in"), ctypes.byref(level_grads_struct(grads)),
        _ptr(workspace, None, "workspace"), workspace.numel() * workspace.element_size(),
        _stream(stream))
    _check(st, "octree_nca_step_backward")


def octree_nca_upsample_backward(model: Model, grad_fine, factor, grad_coarse,
                                 stream=None) -> None:
    d, h, w = grad_coarse.shape[:3]
    f = (_I32 * 3)(*[int(v) for v in factor])
    st = lib().octree_nca_upsample_backward(ctypes.byref(model.struct()),
                                            _ptr(grad_fine, torch.float32, "grad_fine"),
                                            _extent((d, h, w)), f,
                                            _ptr(grad_coarse, torch.float32, "grad_coarse"),
                                            _stream(stream))
    _check(st, "octree_nca_upsample_backward")


def octree_nca_readout_mse_workspace_bytes(extent) -> int:
    return int(lib().octree_nca_readout_mse_workspace_bytes(_extent(extent)))


def octree_nca_readout_mse(model: Model, state, target, grad, loss, workspace,
                           stream=None) -> None:
    """loss: device float64 tensor of one element."""
    d, h, w = state.shape[:3]
    st = lib().octree_nca_readout_mse(ctypes.byref(model.struct()),
                                      _ptr(state, torch.float32, "state"),
                                      _ptr(target, torch.float32, "target"), _extent((d, h, w)),
                                      _ptr(grad, torch.float32, "grad"),
                                      _ptr(loss, torch.float64, "loss"),
                                      _ptr(workspace, None, "workspace"),
                                      workspace.numel() * workspace.element_size(),
                                      _stream(stream))
    _check(st, "octree_nca_readout_mse")


def octree_nca_train_workspace_bytes(model: Model, finest, factors, steps) -> int:
    levels = len(steps)
    s = (_I32 * levels)(*[int(v) for v in steps])
    return int(lib().octree_nca_train_workspace_bytes(ctypes.byref(model.struct()),
                                                      _extent(finest), levels, _factors(factors),
                                                      s))


def octree_nca_train_step(model: Model, image, factors, weights, steps, fire_rate: float,
                          seed: int, target, workspace, grads, loss, final_state=None,
                          stream=None) -> None:
    """One training step; ``grads`` is a list (index = level) of gradient sets,
    overwritten; ``loss`` a device float64 tensor of one element."""
    levels = len(steps)
    d, h, w = image.shape[:3]
    ws = (_LevelWeights * levels)(*[level_weights_struct(x) for x in weights])
    gs = (_LevelGrads * levels)(*[level_grads_struct(x) for x in grads])
    s = (_I32 * levels)(*[int(v) for v in steps])
    st = lib().octree_nca_train_step(
        ctypes.byref(model.struct()), _ptr(image, torch.float32, "image"), _extent((d, h, w)),
        levels, _factors(factors), ws, s, float(fire_rate), int(seed),
        _ptr(target, torch.float32, "target"), _ptr(workspace, None, "workspace"),
        workspace.numel() * workspace.element_size(), gs, _ptr(loss, torch.float64, "loss"),
        _ptr(final_state, torch.float32, "final_state"), _stream(stream))
    _check(st, "octree_nca_train_step")
